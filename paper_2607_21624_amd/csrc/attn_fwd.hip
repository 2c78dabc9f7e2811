// attn_fwd.hip -- attention forward on token-major Q/K/V, gfx950.
//
// One workgroup = 4 wavefronts = 128 queries of one (batch, query head); each
// wavefront owns 32 queries.  The loop streams key/value tiles of 64 rows
// (the R-Tile, section 4.2) from the token-major tensors straight into LDS:
// row r of the tile is row (k0 + r) of the projection output, read at
// base + b*sb + (k0+r)*ss + hk*sh, so the head split and transpose of the
// multi-head attention chain (section 4.3.1) never materialise.
//
// The products are arranged so that no operand needs a physical transpose
// (the tile invariance of section 4.2: the same staged tile serves both
// reduction directions):
//   S^T = K Q^T   A = K rows (LDS row reads), B = Q rows (registers);
//                 the accumulator puts one query per lane column, so the
//                 softmax row max/sum over keys is an in-lane reduction plus
//                 one exchange between the two 32-lane halves;
//   O^T += V^T P^T  A = V^T via LDS transposed reads (ds_read_b64_tr_b16),
//                 B = P^T taken straight from the S^T accumulator registers.
// QK^T followed by PV is the consecutive matrix-product pair of section 4.4.2;
// here both share one tile configuration inside one kernel.
// Online softmax in base 2 with scale*log2(e) folded into the scores; the
// saved LSE is converted to natural log at the store.
#include "cdna4.hpp"
#include "kernels.hpp"
#include "tokmap.hpp"

namespace fbl {

namespace {

constexpr int kFwdWaves = 4;
constexpr int kFwdBM = 32 * kFwdWaves;  // queries per workgroup
constexpr int kFwdBN = 64;              // keys per tile

template <typename T, int D>
struct FwdTile {
    static constexpr int PITCH = D + 16 / (int)sizeof(T);  // LDS row pitch (elements), 16-byte pad
    static constexpr int CPR = D * (int)sizeof(T) / 16;    // 16-byte chunks per row
};

template <typename T, int D>
__device__ __forceinline__ void stage_rows(T* dst, const T* src, int64_t ss, int row0, int nrows_valid) {
    using TL = FwdTile<T, D>;
    constexpr int NCH = kFwdBN * TL::CPR;
    constexpr int EPC = 16 / (int)sizeof(T);
#pragma unroll
    for (int i = threadIdx.x; i < NCH; i += kFwdWaves * 64) {
        const int r = i / TL::CPR, cc = i % TL::CPR;
        uint4 x = {0u, 0u, 0u, 0u};
        if (r < nrows_valid) x = load16(src + (int64_t)(row0 + r) * ss + cc * EPC);
        *reinterpret_cast<uint4*>(dst + r * TL::PITCH + cc * EPC) = x;
    }
}

template <typename T, int D>
__global__ __launch_bounds__(256) void attn_fwd_kernel(FwdArgs a) {
    using TL = FwdTile<T, D>;
    constexpr int NC = D / 16;  // k-chunks over the head dim
    constexpr int ND = D / 32;  // 32-wide output column blocks
    constexpr int PITCH = TL::PITCH;
    __shared__ __attribute__((aligned(16))) T sK[kFwdBN * PITCH];
    __shared__ __attribute__((aligned(16))) T sV[kFwdBN * PITCH];

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int g = lane >> 5;
    const int c32 = lane & 31;
    const int S = a.S;
    const int nqb = (S + kFwdBM - 1) / kFwdBM;
    // causal: the last query blocks see the most keys; launch them first
    const int qb = a.mask.causal ? (nqb - 1 - (int)blockIdx.x) : (int)blockIdx.x;
    const int h = blockIdx.y;
    const int b = blockIdx.z;
    const int hk = h / (a.Hq / a.Hkv);

    int kv_end = S;
    if (a.mask.kv_len) kv_end = min(max(a.mask.kv_len[b], 0), S);
    const int q0 = qb * kFwdBM;
    const int qw0 = q0 + wave * 32;  // first query of this wave
    const int qi = qw0 + c32;        // this lane's query (column of S^T)
    int k_hi = kv_end;
    if (a.mask.causal) k_hi = min(k_hi, q0 + kFwdBM);
    const int nkb = (k_hi + kFwdBN - 1) / kFwdBN;

    // Q^T as the B operand: lane <-> query, in-lane d = 16c + 8g + e
    Frag<T> qf[NC];
    {
        const T* qrow = static_cast<const T*>(a.q) + a.mq.head_base(b, h) + (int64_t)qi * a.mq.ss;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            if (qi < S) {
                if constexpr (sizeof(T) == 2) {
                    uint4 x = load16(qrow + 16 * c + 8 * g);
                    qf[c].v = __builtin_bit_cast(bf16x8, x);
                } else {
                    uint4 x0 = load16(qrow + 16 * c + 8 * g);
                    uint4 x1 = load16(qrow + 16 * c + 8 * g + 4);
                    f32x4 f0 = __builtin_bit_cast(f32x4, x0), f1 = __builtin_bit_cast(f32x4, x1);
#pragma unroll
                    for (int e = 0; e < 4; ++e) { qf[c].v[e] = f0[e]; qf[c].v[4 + e] = f1[e]; }
                }
            } else {
                float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                pack_frag(qf[c], z);
            }
        }
    }

    f32x16 oacc[ND];
#pragma unroll
    for (int t = 0; t < ND; ++t) oacc[t] = f32x16{};
    float m = -INFINITY, l = 0.f;

    const T* kbase = static_cast<const T*>(a.k) + a.mk.head_base(b, hk);
    const T* vbase = static_cast<const T*>(a.v) + a.mv.head_base(b, hk);

    for (int kb = 0; kb < nkb; ++kb) {
        const int k0 = kb * kFwdBN;
        __syncthreads();
        stage_rows<T, D>(sK, kbase, a.mk.ss, k0, min(kFwdBN, S - k0));
        stage_rows<T, D>(sV, vbase, a.mv.ss, k0, min(kFwdBN, S - k0));
        __syncthreads();

        // a whole tile above this wave's diagonal contributes nothing
        if (a.mask.causal && k0 > qw0 + 31) continue;

        f32x16 s[2];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            s[kt] = f32x16{};
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                Frag<T> kf;
                lds_row_frag(kf, sK + (kt * 32 + c32) * PITCH + 16 * c + 8 * g);
                mma(s[kt], kf, qf[c]);
            }
        }

        const bool need_mask = (k0 + kFwdBN > kv_end) || (a.mask.causal && k0 + kFwdBN - 1 > qw0);
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float x = s[kt][r] * a.scale_log2;
                if (need_mask) {
                    const int key = k0 + kt * 32 + acc_row(r, g);
                    if (key >= kv_end || (a.mask.causal && key > qi)) x = -INFINITY;
                }
                s[kt][r] = x;
                mx = fmaxf(mx, x);
            }
        }
        mx = fmaxf(mx, other_half(mx));
        const float m_new = fmaxf(m, mx);
        const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
        const float alpha = fast_exp2(m - m_use);
        float ls = 0.f;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float p = fast_exp2(s[kt][r] - m_use);
                s[kt][r] = p;
                ls += p;
            }
        }
        ls += other_half(ls);
        l = l * alpha + ls;
        m = m_new;
#pragma unroll
        for (int t = 0; t < ND; ++t) oacc[t] *= alpha;

        // O^T += V^T P^T over the 64 keys: chunk (kt, cc) covers keys
        // kt*32 + 16cc + {4g..4g+3, 8+4g..8+4g+3} in accumulator order
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
            for (int cc = 0; cc < 2; ++cc) {
                Frag<T> pf;
                float pv[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) pv[e] = s[kt][8 * cc + e];
                pack_frag(pf, pv);
                const int row0 = kt * 32 + 16 * cc + 4 * g;
#pragma unroll
                for (int t = 0; t < ND; ++t) {
                    Frag<T> vf;
                    lds_tr_frag(vf, sV, PITCH, row0, row0 + 8, 32 * t, lane);
                    mma(oacc[t], vf, pf);
                }
            }
        }
    }

    if (qi < S) {
        const float inv = (l > 0.f) ? 1.f / l : 0.f;
        T* orow = static_cast<T*>(a.o) + a.mo.head_base(b, h) + (int64_t)qi * a.mo.ss;
#pragma unroll
        for (int t = 0; t < ND; ++t) {
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
                const int dcol = 32 * t + 8 * rr + 4 * g;
                store4(orow + dcol, oacc[t][4 * rr] * inv, oacc[t][4 * rr + 1] * inv, oacc[t][4 * rr + 2] * inv,
                       oacc[t][4 * rr + 3] * inv);
            }
        }
        if (g == 0) {
            a.lse[((int64_t)b * a.Hq + h) * S + qi] = (l > 0.f) ? (m + __log2f(l)) * kLn2 : -INFINITY;
        }
    }
}

}  // namespace

template <typename T, int D>
hipError_t launch_attn_fwd(const FwdArgs& a, hipStream_t stream) {
    const int nqb = (a.S + kFwdBM - 1) / kFwdBM;
    dim3 grid(nqb, a.Hq, a.B);
    hipLaunchKernelGGL((attn_fwd_kernel<T, D>), grid, dim3(256), 0, stream, a);
    return hipGetLastError();
}

template hipError_t launch_attn_fwd<float, 32>(const FwdArgs&, hipStream_t);
template hipError_t launch_attn_fwd<float, 64>(const FwdArgs&, hipStream_t);
template hipError_t launch_attn_fwd<float, 128>(const FwdArgs&, hipStream_t);
template hipError_t launch_attn_fwd<bf16, 32>(const FwdArgs&, hipStream_t);
template hipError_t launch_attn_fwd<bf16, 64>(const FwdArgs&, hipStream_t);
template hipError_t launch_attn_fwd<bf16, 128>(const FwdArgs&, hipStream_t);

}  // namespace fbl
