// attn_bwd.hip -- attention backward on token-major tensors, gfx950.
//
// Gradients of L = sum(O * dO) (chain rule through P = softmax(scale Q K^T)
// and O = P V; the paper gives the matrix-product gradients in section 4.1
// and softmax as forward-dependent, consistent-access in the same section):
//   D_i  = sum_k dO_ik O_ik                         (bwd_pre)
//   P    = exp(scale q_i.k_j - LSE_i)               (recomputed, bwd_main)
//   dV  += P^T dO,  dP = dO V^T,  dS = P (dP - D)
//   dK  += scale dS^T Q,  dQ += scale dS K          (bwd_main, dQ via fp32
//                                                    atomics into a workspace)
//   dQ   = storage type of the fp32 accumulator     (bwd_dq)
//
// Key/value-major main pass: one workgroup owns 128 keys of one (batch,
// key/value head); each of its 4 wavefronts owns 32 keys and keeps them (K and
// V rows) in registers, together with its dK and dV accumulators.  It walks
// every query block of every query head of its GQA group, so the reductions
// over queries that build dK/dV (the "reduce along M" direction of section
// 4.2) and the group reduction over the G query heads both stay in registers.
// Q and dO tiles are staged once per block in LDS and serve both reduction
// directions (tile invariance, section 4.2): row reads for S = Q K^T and
// dP = dO V^T (contraction over d), transposed reads (ds_read_b64_tr_b16) for
// dV and dK (contraction over queries).  dS goes through LDS once so the dQ
// product (contraction over keys) can be split over the 4 wavefronts by
// output tile.
#include "cdna4.hpp"
#include "kernels.hpp"
#include "tokmap.hpp"

namespace fbl {

namespace {

constexpr int kBwdWaves = 4;
constexpr int kBwdBN = 32 * kBwdWaves;  // keys per workgroup

template <typename T, int D>
struct BwdTile {
    static constexpr int BQ = 4096 / D;  // queries per block: 128, 64, 32 for D = 32, 64, 128
    static constexpr int NQT = BQ / 32;
    static constexpr int EPC = 16 / (int)sizeof(T);     // elements per 16-byte chunk
    static constexpr int PITCH = D + EPC;               // Q, dO, K tile row pitch (elements)
    static constexpr int SPITCH = BQ + EPC;             // dS^T tile row pitch (elements)
    static constexpr int CPR = D / EPC;                 // 16-byte chunks per row
    static constexpr int OFF_Q = 0;
    static constexpr int OFF_DO = OFF_Q + BQ * PITCH * (int)sizeof(T);
    static constexpr int OFF_K = OFF_DO + BQ * PITCH * (int)sizeof(T);
    static constexpr int OFF_DS = OFF_K + kBwdBN * PITCH * (int)sizeof(T);
    static constexpr int OFF_LSE = OFF_DS + kBwdBN * SPITCH * (int)sizeof(T);
    static constexpr int OFF_DR = OFF_LSE + BQ * 4;
    static constexpr int BYTES = OFF_DR + BQ * 4;
    static_assert(NQT * (D / 32) == kBwdWaves, "one dQ output tile per wavefront");
    static_assert(BYTES <= 160 * 1024, "LDS budget");
};

template <typename T, int D>
__device__ __forceinline__ void stage_tile(T* dst, const T* src, int64_t ss, int row0, int nrows, int nvalid) {
    using TL = BwdTile<T, D>;
    for (int i = threadIdx.x; i < nrows * TL::CPR; i += kBwdWaves * 64) {
        const int r = i / TL::CPR, cc = i % TL::CPR;
        uint4 x = {0u, 0u, 0u, 0u};
        if (r < nvalid) x = load16(src + (int64_t)(row0 + r) * ss + cc * TL::EPC);
        *reinterpret_cast<uint4*>(dst + r * TL::PITCH + cc * TL::EPC) = x;
    }
}

// Register fragment of one row (8 elements at column 16c + 8g).
template <typename T>
__device__ __forceinline__ void global_row_frag(Frag<T>& f, const T* p, bool valid) {
    if (!valid) {
        float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        pack_frag(f, z);
        return;
    }
    if constexpr (sizeof(T) == 2) {
        f.v = __builtin_bit_cast(bf16x8, load16(p));
    } else {
        f32x4 a = __builtin_bit_cast(f32x4, load16(p));
        f32x4 b = __builtin_bit_cast(f32x4, load16(p + 4));
#pragma unroll
        for (int e = 0; e < 4; ++e) { f.v[e] = a[e]; f.v[4 + e] = b[e]; }
    }
}

// D_i = sum_k dO_ik O_ik per (b, h, i) and zeroing of the dQ accumulator.
// Each (b, s, h) row of d elements is read by D*sizeof(T)/16 lanes (one
// 16-byte chunk each); consecutive rows are consecutive heads of one token,
// so a wavefront reads a contiguous run of the token-major tensor.
template <typename T, int D>
__global__ __launch_bounds__(256) void attn_bwd_pre(BwdArgs a) {
    constexpr int EPC = 16 / (int)sizeof(T);
    constexpr int LPR = D / EPC;
    constexpr int RPB = 256 / LPR;
    const int64_t nrows = (int64_t)a.B * a.S * a.Hq;
    const int64_t row = (int64_t)blockIdx.x * RPB + threadIdx.x / LPR;
    const int part = threadIdx.x % LPR;
    float acc = 0.f;
    int b = 0, s = 0, h = 0;
    if (row < nrows) {
        h = (int)(row % a.Hq);
        s = (int)((row / a.Hq) % a.S);
        b = (int)(row / ((int64_t)a.Hq * a.S));
        const T* o = static_cast<const T*>(a.o) + a.mo.offset(b, h, s, part * EPC);
        const T* g = static_cast<const T*>(a.dout) + a.mdo.offset(b, h, s, part * EPC);
        uint4 xo = load16(o), xg = load16(g);
        if constexpr (sizeof(T) == 2) {
            bf16x8 vo = __builtin_bit_cast(bf16x8, xo), vg = __builtin_bit_cast(bf16x8, xg);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc += (float)vo[e] * (float)vg[e];
        } else {
            f32x4 vo = __builtin_bit_cast(f32x4, xo), vg = __builtin_bit_cast(f32x4, xg);
#pragma unroll
            for (int e = 0; e < 4; ++e) acc += vo[e] * vg[e];
        }
        float* z = a.dq_acc + row * D + part * EPC;
#pragma unroll
        for (int e = 0; e < EPC; e += 4) *reinterpret_cast<f32x4*>(z + e) = f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int off = LPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if (row < nrows && part == 0) a.drow[((int64_t)b * a.Hq + h) * a.S + s] = acc;
}

template <typename T, int D>
__global__ __launch_bounds__(256) void attn_bwd_main(BwdArgs a) {
    using TL = BwdTile<T, D>;
    constexpr int NC = D / 16;
    constexpr int ND = D / 32;
    constexpr int BQ = TL::BQ;
    constexpr int NQT = TL::NQT;
    constexpr int PITCH = TL::PITCH;
    constexpr int SPITCH = TL::SPITCH;
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    T* sQ = reinterpret_cast<T*>(smem + TL::OFF_Q);
    T* sdO = reinterpret_cast<T*>(smem + TL::OFF_DO);
    T* sK = reinterpret_cast<T*>(smem + TL::OFF_K);
    T* sdS = reinterpret_cast<T*>(smem + TL::OFF_DS);
    float* sLse = reinterpret_cast<float*>(smem + TL::OFF_LSE);
    float* sDr = reinterpret_cast<float*>(smem + TL::OFF_DR);

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int g = lane >> 5;
    const int c32 = lane & 31;
    const int S = a.S;
    const int k0 = blockIdx.x * kBwdBN;
    const int hk = blockIdx.y;
    const int b = blockIdx.z;
    const int G = a.Hq / a.Hkv;
    int kv_end = S;
    if (a.mask.kv_len) kv_end = min(max(a.mask.kv_len[b], 0), S);
    const int kw0 = k0 + wave * 32;  // first key of this wave
    const int key = kw0 + c32;       // this lane's key (column of S)
    const bool key_ok = key < kv_end;

    const T* kbase = static_cast<const T*>(a.k) + a.mk.head_base(b, hk);
    const T* vbase = static_cast<const T*>(a.v) + a.mv.head_base(b, hk);

    // K_w and V_w rows as B operands: lane <-> key, in-lane d = 16c + 8g + e
    Frag<T> kf[NC], vf[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        global_row_frag(kf[c], kbase + (int64_t)key * a.mk.ss + 16 * c + 8 * g, key < S);
        global_row_frag(vf[c], vbase + (int64_t)key * a.mv.ss + 16 * c + 8 * g, key < S);
    }
    stage_tile<T, D>(sK, kbase, a.mk.ss, k0, kBwdBN, min(kBwdBN, S - k0));

    f32x16 dk[ND], dv[ND];
#pragma unroll
    for (int t = 0; t < ND; ++t) { dk[t] = f32x16{}; dv[t] = f32x16{}; }

    if (k0 < kv_end) {
        const int qb_start = a.mask.causal ? k0 / BQ : 0;
        const int nqb = (S + BQ - 1) / BQ;
        for (int hh = 0; hh < G; ++hh) {
            const int h = hk * G + hh;
            const T* qbase = static_cast<const T*>(a.q) + a.mq.head_base(b, h);
            const T* dobase = static_cast<const T*>(a.dout) + a.mdo.head_base(b, h);
            const float* lse_row = a.lse + ((int64_t)b * a.Hq + h) * S;
            const float* dr_row = a.drow + ((int64_t)b * a.Hq + h) * S;
            for (int qb = qb_start; qb < nqb; ++qb) {
                const int q0 = qb * BQ;
                const int nvalid = min(BQ, S - q0);
                __syncthreads();
                stage_tile<T, D>(sQ, qbase, a.mq.ss, q0, BQ, nvalid);
                stage_tile<T, D>(sdO, dobase, a.mdo.ss, q0, BQ, nvalid);
                for (int i = threadIdx.x; i < BQ; i += kBwdWaves * 64) {
                    float lse = -INFINITY, dr = 0.f;
                    if (i < nvalid) { lse = lse_row[q0 + i]; dr = dr_row[q0 + i]; }
                    sLse[i] = (lse == -INFINITY) ? INFINITY : lse * kLog2e;
                    sDr[i] = dr;
                }
                __syncthreads();

                // S = Q K_w^T and dP = dO V_w^T; accumulators: lane <-> key,
                // in-lane query q0 + 32qt + acc_row(r, g)
                f32x16 s[NQT], dp[NQT];
#pragma unroll
                for (int qt = 0; qt < NQT; ++qt) {
                    s[qt] = f32x16{};
                    dp[qt] = f32x16{};
#pragma unroll
                    for (int c = 0; c < NC; ++c) {
                        Frag<T> fq, fo;
                        lds_row_frag(fq, sQ + (qt * 32 + c32) * PITCH + 16 * c + 8 * g);
                        lds_row_frag(fo, sdO + (qt * 32 + c32) * PITCH + 16 * c + 8 * g);
                        mma(s[qt], fq, kf[c]);
                        mma(dp[qt], fo, vf[c]);
                    }
                }
                // P and dS in place (s <- P, dp <- dS)
#pragma unroll
                for (int qt = 0; qt < NQT; ++qt) {
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr) {
                        const int qloc = qt * 32 + 8 * rr + 4 * g;
                        const f32x4 l4 = *reinterpret_cast<const f32x4*>(sLse + qloc);
                        const f32x4 d4 = *reinterpret_cast<const f32x4*>(sDr + qloc);
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            const int r = 4 * rr + j;
                            const int qi = q0 + qloc + j;
                            const bool ok = key_ok && (!a.mask.causal || key <= qi);
                            const float p = ok ? fast_exp2(s[qt][r] * a.scale_log2 - l4[j]) : 0.f;
                            s[qt][r] = p;
                            dp[qt][r] = p * (dp[qt][r] - d4[j]);
                        }
                    }
                }
                // dV_w += P^T dO and dK_w += dS^T Q, contracting over queries:
                // chunk (qt, cc) covers queries 32qt + 16cc + {4g..4g+3, 8+4g..8+4g+3}
#pragma unroll
                for (int qt = 0; qt < NQT; ++qt) {
#pragma unroll
                    for (int cc = 0; cc < 2; ++cc) {
                        Frag<T> pa, dsa;
                        float pv[8], dsv[8];
#pragma unroll
                        for (int e = 0; e < 8; ++e) { pv[e] = s[qt][8 * cc + e]; dsv[e] = dp[qt][8 * cc + e]; }
                        pack_frag(pa, pv);
                        pack_frag(dsa, dsv);
                        const int row0 = qt * 32 + 16 * cc + 4 * g;
#pragma unroll
                        for (int t = 0; t < ND; ++t) {
                            Frag<T> fdo, fq;
                            lds_tr_frag(fdo, sdO, PITCH, row0, row0 + 8, 32 * t, lane);
                            lds_tr_frag(fq, sQ, PITCH, row0, row0 + 8, 32 * t, lane);
                            mma(dv[t], pa, fdo);
                            mma(dk[t], dsa, fq);
                        }
                    }
                }
                // dS^T (storage type) into LDS: row = key, columns = queries
                T* dsrow = sdS + (wave * 32 + c32) * SPITCH;
#pragma unroll
                for (int qt = 0; qt < NQT; ++qt) {
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr) {
                        store4(dsrow + qt * 32 + 8 * rr + 4 * g, dp[qt][4 * rr], dp[qt][4 * rr + 1],
                               dp[qt][4 * rr + 2], dp[qt][4 * rr + 3]);
                    }
                }
                __syncthreads();
                // dQ tile (qt, t) of this wavefront: dS[q, 0:128] K[0:128, 32t:32t+32]
                {
                    const int qt = wave / ND, t = wave % ND;
                    f32x16 acc = f32x16{};
#pragma unroll
                    for (int ch = 0; ch < kBwdBN / 16; ++ch) {
                        const int row0 = 16 * ch + 8 * g;
                        Frag<T> fa, fb;
                        lds_tr_frag(fa, sdS, SPITCH, row0, row0 + 4, 32 * qt, lane);
                        lds_tr_frag(fb, sK, PITCH, row0, row0 + 4, 32 * t, lane);
                        mma(acc, fa, fb);
                    }
                    float* dq_col = a.dq_acc + (int64_t)h * D + 32 * t + c32;
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int qi = q0 + qt * 32 + acc_row(r, g);
                        if (qi < S) atomicAdd(dq_col + ((int64_t)b * S + qi) * ((int64_t)a.Hq * D), acc[r]);
                    }
                }
            }
        }
    }

    // dK (times scale) and dV rows of this wave's keys; lane <-> d column
    T* dkbase = static_cast<T*>(a.dk) + a.mdk.head_base(b, hk);
    T* dvbase = static_cast<T*>(a.dv) + a.mdv.head_base(b, hk);
#pragma unroll
    for (int t = 0; t < ND; ++t) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int kk = kw0 + acc_row(r, g);
            if (kk < S) {
                store_out<T>(dkbase + (int64_t)kk * a.mdk.ss + 32 * t + c32, dk[t][r] * a.scale);
                store_out<T>(dvbase + (int64_t)kk * a.mdv.ss + 32 * t + c32, dv[t][r]);
            }
        }
    }
}

// dQ = scale * accumulator, converted to the storage type, written through
// dQ's own index map.
template <typename T, int D>
__global__ __launch_bounds__(256) void attn_bwd_dq(BwdArgs a) {
    constexpr int EPC = 16 / (int)sizeof(T);
    constexpr int LPR = D / EPC;
    constexpr int RPB = 256 / LPR;
    const int64_t nrows = (int64_t)a.B * a.S * a.Hq;
    const int64_t row = (int64_t)blockIdx.x * RPB + threadIdx.x / LPR;
    const int part = threadIdx.x % LPR;
    if (row >= nrows) return;
    const int h = (int)(row % a.Hq);
    const int s = (int)((row / a.Hq) % a.S);
    const int b = (int)(row / ((int64_t)a.Hq * a.S));
    const float* src = a.dq_acc + row * D + part * EPC;
    T* dst = static_cast<T*>(a.dq) + a.mdq.offset(b, h, s, part * EPC);
    if constexpr (sizeof(T) == 2) {
        f32x4 x0 = *reinterpret_cast<const f32x4*>(src);
        f32x4 x1 = *reinterpret_cast<const f32x4*>(src + 4);
        bf16x8 y;
#pragma unroll
        for (int e = 0; e < 4; ++e) { y[e] = (bf16)(x0[e] * a.scale); y[4 + e] = (bf16)(x1[e] * a.scale); }
        *reinterpret_cast<bf16x8*>(dst) = y;
    } else {
        f32x4 x = *reinterpret_cast<const f32x4*>(src);
        *reinterpret_cast<f32x4*>(dst) = x * a.scale;
    }
}

template <typename T, int D>
hipError_t set_main_lds() {
    static hipError_t once = hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_bwd_main<T, D>),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize,
                                                 BwdTile<T, D>::BYTES);
    return once;
}

}  // namespace

template <typename T, int D>
hipError_t launch_attn_bwd(const BwdArgs& a, unsigned phases, hipStream_t stream) {
    constexpr int LPR = D / (16 / (int)sizeof(T));
    constexpr int RPB = 256 / LPR;
    const int64_t nrows = (int64_t)a.B * a.S * a.Hq;
    const unsigned rblocks = (unsigned)((nrows + RPB - 1) / RPB);
    hipError_t e = set_main_lds<T, D>();
    if (e != hipSuccess) return e;
    if (phases & 1u) hipLaunchKernelGGL((attn_bwd_pre<T, D>), dim3(rblocks), dim3(256), 0, stream, a);
    if (phases & 2u) {
        dim3 grid((a.S + kBwdBN - 1) / kBwdBN, a.Hkv, a.B);
        constexpr int lds = BwdTile<T, D>::BYTES;
        hipLaunchKernelGGL((attn_bwd_main<T, D>), grid, dim3(256), lds, stream, a);
    }
    if (phases & 4u) hipLaunchKernelGGL((attn_bwd_dq<T, D>), dim3(rblocks), dim3(256), 0, stream, a);
    return hipGetLastError();
}

template hipError_t launch_attn_bwd<float, 32>(const BwdArgs&, unsigned, hipStream_t);
template hipError_t launch_attn_bwd<float, 64>(const BwdArgs&, unsigned, hipStream_t);
template hipError_t launch_attn_bwd<float, 128>(const BwdArgs&, unsigned, hipStream_t);
template hipError_t launch_attn_bwd<bf16, 32>(const BwdArgs&, unsigned, hipStream_t);
template hipError_t launch_attn_bwd<bf16, 64>(const BwdArgs&, unsigned, hipStream_t);
template hipError_t launch_attn_bwd<bf16, 128>(const BwdArgs&, unsigned, hipStream_t);

}  // namespace fbl
