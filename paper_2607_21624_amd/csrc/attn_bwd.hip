// attn_bwd.hip -- attention backward on token-major tensors, gfx950.
//
// Gradients of L = sum(O * dO) by the chain rule through P = softmax(scale
// Q K^T) and O = P V (the paper states the matrix-product gradients in
// section 4.1, FTD-D, and classes softmax as forward-dependent with
// consistent access, FTD-C):
//   D_i  = sum_k dO_ik O_ik
//   P    = exp(scale q_i.k_j - LSE_i)          (recomputed from the saved LSE)
//   dP   = dO V^T,  dS = P (dP - D)
//   dV   = P^T dO,  dK = scale dS^T Q,  dQ = scale dS K
// Three launches, no atomics, every output written once:
//   attn_bwd_stats  per query row: LSE*log2(e) (+inf for an empty row) and D.
//   attn_bwd_kv     key/value-major.  A workgroup owns 128 keys of one
//                   (batch, kv head); each wavefront keeps its 32 K and V rows
//                   and its dK^T, dV^T accumulators in registers and walks the
//                   query blocks of every query head of its GQA group.  The
//                   reductions over queries that build dK/dV (the "reduce
//                   along M" direction of section 4.2) and the group sum over
//                   the G query heads never leave registers.
//   attn_bwd_q      query-major.  A workgroup owns 128 queries of one
//                   (batch, query head) and walks the key tiles, recomputing S
//                   and dP, and accumulates dQ^T in registers (the "reduce
//                   along N" direction).
// Recomputing S and dP in the query-major pass costs two extra products per
// (query, key) pair; it replaces fp32 atomics, which run at ~1.3 TB/s on this
// part -- far slower than the 3 products they would save at these shapes.
// Q/dO (kv pass) and K/V (q pass) tiles are staged once per block in LDS by
// DMA and serve both reduction directions (tile invariance, section 4.2): row
// reads where the contraction runs along d, transposed reads
// (ds_read_b64_tr_b16) where it runs along tokens.
#include "cdna4.hpp"
#include "kernels.hpp"
#include "stage.hpp"
#include "tokmap.hpp"

namespace fbl {

namespace {

constexpr int kWaves = 4;
constexpr int kKvBN = 32 * kWaves;  // keys per kv-pass workgroup
constexpr int kKvBQ = 64;           // queries per kv-pass block
constexpr int kQBM = 32 * kWaves;   // queries per q-pass workgroup
constexpr int kQBN = 64;            // keys per q-pass tile

// ------------------------------------------------------------------ stats
// Each (b, s, h) row of d elements is read by D*sizeof(T)/16 lanes (one
// 16-byte chunk each); consecutive rows are consecutive heads of one token,
// so a wavefront reads a contiguous run of the token-major tensors.
template <typename T, int D>
__global__ __launch_bounds__(256) void attn_bwd_stats(BwdArgs a) {
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
        const uint4 xo = load16(o), xg = load16(g);
        if constexpr (sizeof(T) == 2) {
            const bf16x8 vo = __builtin_bit_cast(bf16x8, xo), vg = __builtin_bit_cast(bf16x8, xg);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc += (float)vo[e] * (float)vg[e];
        } else {
            const f32x4 vo = __builtin_bit_cast(f32x4, xo), vg = __builtin_bit_cast(f32x4, xg);
#pragma unroll
            for (int e = 0; e < 4; ++e) acc += vo[e] * vg[e];
        }
    }
#pragma unroll
    for (int off = LPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if (row < nrows && part == 0) {
        const int64_t i = ((int64_t)b * a.Hq + h) * a.S + s;
        const float lse = a.lse[i];
        a.stats[i] = f32x2{lse == -INFINITY ? INFINITY : lse * kLog2e, acc};
    }
}

// ------------------------------------------------------------- kv pass
template <typename T, int D>
struct KvSmem {
    static constexpr int TILE = kKvBQ * D;  // elements of one Q or dO tile
    // [Q0 Q1 dO0 dO1] tiles, then two 1 KB stats buffers (64 (lse2, D) pairs
    // plus room for the full 64-lane DMA of one instruction)
    static constexpr int BYTES = 4 * TILE * (int)sizeof(T) + 2 * 1024;
};

template <typename T, int D>
__global__ __launch_bounds__(256, 1) void attn_bwd_kv(BwdArgs a) {
    using SM = KvSmem<T, D>;
    constexpr int NC = D / 16;
    constexpr int ND = D / 32;
    constexpr int TILE = SM::TILE;
    constexpr int NQT = kKvBQ / 32;
    extern __shared__ __attribute__((aligned(1024))) unsigned char kv_smem[];
    T* tiles = reinterpret_cast<T*>(kv_smem);
    float* stat_buf = reinterpret_cast<float*>(kv_smem + 4 * TILE * sizeof(T));

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int g = lane >> 5;
    const int c32 = lane & 31;
    const int S = a.S;
    const int nkb = (S + kKvBN - 1) / kKvBN;
    const int logical = xcd_logical_id(blockIdx.x, nkb * a.Hkv * a.B, gridDim.x);
    if (logical < 0) return;
    const int kblk = logical % nkb;
    const int hk = (logical / nkb) % a.Hkv;
    const int b = logical / (nkb * a.Hkv);
    const int G_ = a.Hq / a.Hkv;
    int kv_end = S;
    if (a.mask.kv_len) kv_end = min(max(a.mask.kv_len[b], 0), S);
    const int k0 = kblk * kKvBN;
    const int kw0 = k0 + wave * 32;  // first key of this wave
    const int key = kw0 + c32;       // this lane's key (column of S)
    const bool key_ok = key < kv_end;

    const uint32_t es = sizeof(T);
    const T* kbase = static_cast<const T*>(a.k) + a.mk.head_base(b, hk);
    const T* vbase = static_cast<const T*>(a.v) + a.mv.head_base(b, hk);

    // K_w and V_w rows as B operands: lane <-> key, in-lane d = 16c + 8g + e
    Frag<T> kf[NC], vf[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        pack_frag(kf[c], z);
        pack_frag(vf[c], z);
        if (key < S) {
            const T* kp = kbase + (int64_t)key * a.mk.ss + 16 * c + 8 * g;
            const T* vp = vbase + (int64_t)key * a.mv.ss + 16 * c + 8 * g;
            if constexpr (sizeof(T) == 2) {
                kf[c].v = __builtin_bit_cast(bf16x8, load16(kp));
                vf[c].v = __builtin_bit_cast(bf16x8, load16(vp));
            } else {
                const f32x4 k0v = __builtin_bit_cast(f32x4, load16(kp)), k1v = __builtin_bit_cast(f32x4, load16(kp + 4));
                const f32x4 v0v = __builtin_bit_cast(f32x4, load16(vp)), v1v = __builtin_bit_cast(f32x4, load16(vp + 4));
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    kf[c].v[e] = k0v[e];
                    kf[c].v[4 + e] = k1v[e];
                    vf[c].v[e] = v0v[e];
                    vf[c].v[4 + e] = v1v[e];
                }
            }
        }
    }

    // dK^T and dV^T: accumulator rows = d (32t + acc_row), columns = keys (lane)
    f32x16 dk[ND], dv[ND];
#pragma unroll
    for (int t = 0; t < ND; ++t) {
        dk[t] = f32x16{};
        dv[t] = f32x16{};
    }

    const int qb_start = a.mask.causal ? (k0 / kKvBQ) : 0;
    const int nqb = (S + kKvBQ - 1) / kKvBQ;
    const int per_head = nqb - qb_start;
    const int n_iter = (k0 < kv_end) ? G_ * per_head : 0;

    auto issue = [&](int it, int buf) {
        const int h = hk * G_ + it / per_head;
        const int q0 = (qb_start + it % per_head) * kKvBQ;
        const Rsrc rq = make_rsrc(static_cast<const T*>(a.q) + a.mq.head_base(b, h),
                                  (uint32_t)((int64_t)(S - 1) * a.mq.ss * es + D * es));
        const Rsrc ro = make_rsrc(static_cast<const T*>(a.dout) + a.mdo.head_base(b, h),
                                  (uint32_t)((int64_t)(S - 1) * a.mdo.ss * es + D * es));
        dma_tile<T, D, kKvBQ, kWaves>(tiles + buf * TILE, rq, q0, (uint32_t)(a.mq.ss * es), wave, lane);
        dma_tile<T, D, kKvBQ, kWaves>(tiles + (2 + buf) * TILE, ro, q0, (uint32_t)(a.mdo.ss * es), wave, lane);
        if (wave == 0) {
            // 64 (lse2, D) pairs = 512 bytes; lanes 32..63 fetch the following
            // rows (zeros past the end) into the spare half of the buffer
            const Rsrc rs = make_rsrc(a.stats + ((int64_t)b * a.Hq + h) * S, (uint32_t)(S * 8));
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (FBL_LDS void*)(stat_buf + buf * 256), 16,
                                                     (uint32_t)(q0 * 8 + lane * 16), 0, 0, 0);
        }
    };

    if (n_iter > 0) issue(0, 0);
    for (int it = 0; it < n_iter; ++it) {
        const int buf = it & 1;
        wait_vmcnt<0>();
        __syncthreads();  // block `it` landed; block it-1's buffers are free
        if (it + 1 < n_iter) issue(it + 1, buf ^ 1);
        const int q0 = (qb_start + it % per_head) * kKvBQ;
        // nothing to do for a wave whose keys are all padding, or all after
        // every query of the block
        if (kw0 >= kv_end) continue;
        if (a.mask.causal && q0 + kKvBQ - 1 < kw0) continue;
        const T* sQ = tiles + buf * TILE;
        const T* sdO = tiles + (2 + buf) * TILE;
        const f32x2* st = reinterpret_cast<const f32x2*>(stat_buf + buf * 256);

        // S = Q K_w^T and dP = dO V_w^T: lane <-> key, in-lane query 32qt + acc_row
        f32x16 s[NQT], dp[NQT];
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt) {
            s[qt] = f32x16{};
            dp[qt] = f32x16{};
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                Frag<T> fq, fo;
                tile_row_frag<D>(fq, sQ, qt * 32 + c32, 16 * c + 8 * g);
                tile_row_frag<D>(fo, sdO, qt * 32 + c32, 16 * c + 8 * g);
                mma(s[qt], fq, kf[c]);
                mma(dp[qt], fo, vf[c]);
            }
        }
        const bool diag = a.mask.causal && q0 < kw0 + 31;
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int ql = qt * 32 + acc_row(r, g);
                const f32x2 sd = st[ql];
                float p = fast_exp2(__builtin_fmaf(s[qt][r], a.scale_log2, -sd[0]));
                if (!key_ok || (diag && key > q0 + ql)) p = 0.f;
                s[qt][r] = p;
                dp[qt][r] = p * (dp[qt][r] - sd[1]);
            }
        }
        // dV^T += dO^T P and dK^T += Q^T dS, contracting over the 64 queries:
        // chunk (qt, cc) covers queries 32qt + 16cc + {4g..4g+3, 8+4g..8+4g+3}
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt) {
#pragma unroll
            for (int cc = 0; cc < 2; ++cc) {
                Frag<T> pb, dsb;
                float pv[8], dsv[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    pv[e] = s[qt][8 * cc + e];
                    dsv[e] = dp[qt][8 * cc + e];
                }
                pack_frag(pb, pv);
                pack_frag(dsb, dsv);
                const int row0 = qt * 32 + 16 * cc + 4 * g;
#pragma unroll
                for (int t = 0; t < ND; ++t) {
                    Frag<T> fdo, fq;
                    tile_tr_frag<D>(fdo, sdO, row0, row0 + 8, 32 * t, lane);
                    tile_tr_frag<D>(fq, sQ, row0, row0 + 8, 32 * t, lane);
                    mma(dv[t], fdo, pb);
                    mma(dk[t], fq, dsb);
                }
            }
        }
    }

    // dK (times scale) and dV rows of this wave's keys: lane <-> key, 4 consecutive d per store
    if (key < S) {
        T* dkrow = static_cast<T*>(a.dk) + a.mdk.head_base(b, hk) + (int64_t)key * a.mdk.ss;
        T* dvrow = static_cast<T*>(a.dv) + a.mdv.head_base(b, hk) + (int64_t)key * a.mdv.ss;
#pragma unroll
        for (int t = 0; t < ND; ++t) {
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
                const int dcol = 32 * t + 8 * rr + 4 * g;
                store4(dkrow + dcol, dk[t][4 * rr] * a.scale, dk[t][4 * rr + 1] * a.scale, dk[t][4 * rr + 2] * a.scale,
                       dk[t][4 * rr + 3] * a.scale);
                store4(dvrow + dcol, dv[t][4 * rr], dv[t][4 * rr + 1], dv[t][4 * rr + 2], dv[t][4 * rr + 3]);
            }
        }
    }
}

// --------------------------------------------------------------- q pass
template <typename T, int D>
struct QSmem {
    static constexpr int TILE = kQBN * D;
    static constexpr int BYTES = 4 * TILE * (int)sizeof(T);  // K0 K1 V0 V1
};

template <typename T, int D>
__global__ __launch_bounds__(256, sizeof(T) == 2 ? 2 : 1) void attn_bwd_q(BwdArgs a) {
    constexpr int NC = D / 16;
    constexpr int ND = D / 32;
    constexpr int TILE = QSmem<T, D>::TILE;
    extern __shared__ __attribute__((aligned(1024))) unsigned char q_smem[];
    T* smem = reinterpret_cast<T*>(q_smem);

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int g = lane >> 5;
    const int c32 = lane & 31;
    const int S = a.S;
    const int nqb = (S + kQBM - 1) / kQBM;
    const int logical = xcd_logical_id(blockIdx.x, nqb * a.Hq * a.B, gridDim.x);
    if (logical < 0) return;
    const int rank = logical % nqb;
    const int h = (logical / nqb) % a.Hq;
    const int b = logical / (nqb * a.Hq);
    const int qb = a.mask.causal ? (nqb - 1 - rank) : rank;
    const int hk = h / (a.Hq / a.Hkv);
    int kv_end = S;
    if (a.mask.kv_len) kv_end = min(max(a.mask.kv_len[b], 0), S);
    const int q0 = qb * kQBM;
    const int qw0 = q0 + wave * 32;
    const int qi = qw0 + c32;  // this lane's query (column of S^T)
    int k_hi = kv_end;
    if (a.mask.causal) k_hi = min(k_hi, q0 + kQBM);
    const int nkb = (k_hi + kQBN - 1) / kQBN;

    // Q^T and dO^T as B operands: lane <-> query, in-lane d = 16c + 8g + e
    Frag<T> qf[NC], of[NC];
    {
        const T* qrow = static_cast<const T*>(a.q) + a.mq.head_base(b, h) + (int64_t)qi * a.mq.ss;
        const T* orow = static_cast<const T*>(a.dout) + a.mdo.head_base(b, h) + (int64_t)qi * a.mdo.ss;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
            pack_frag(qf[c], z);
            pack_frag(of[c], z);
            if (qi < S) {
                if constexpr (sizeof(T) == 2) {
                    qf[c].v = __builtin_bit_cast(bf16x8, load16(qrow + 16 * c + 8 * g));
                    of[c].v = __builtin_bit_cast(bf16x8, load16(orow + 16 * c + 8 * g));
                } else {
                    const f32x4 q0v = __builtin_bit_cast(f32x4, load16(qrow + 16 * c + 8 * g));
                    const f32x4 q1v = __builtin_bit_cast(f32x4, load16(qrow + 16 * c + 8 * g + 4));
                    const f32x4 o0v = __builtin_bit_cast(f32x4, load16(orow + 16 * c + 8 * g));
                    const f32x4 o1v = __builtin_bit_cast(f32x4, load16(orow + 16 * c + 8 * g + 4));
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        qf[c].v[e] = q0v[e];
                        qf[c].v[4 + e] = q1v[e];
                        of[c].v[e] = o0v[e];
                        of[c].v[4 + e] = o1v[e];
                    }
                }
            }
        }
    }
    f32x2 sd = f32x2{INFINITY, 0.f};  // (lse2, D) of this lane's query
    if (qi < S) sd = a.stats[((int64_t)b * a.Hq + h) * S + qi];

    f32x16 dq[ND];  // dQ^T: rows = d (32t + acc_row), columns = queries (lane)
#pragma unroll
    for (int t = 0; t < ND; ++t) dq[t] = f32x16{};

    const uint32_t es = sizeof(T);
    const Rsrc rk = make_rsrc(static_cast<const T*>(a.k) + a.mk.head_base(b, hk),
                              (uint32_t)((int64_t)(S - 1) * a.mk.ss * es + D * es));
    const Rsrc rv = make_rsrc(static_cast<const T*>(a.v) + a.mv.head_base(b, hk),
                              (uint32_t)((int64_t)(S - 1) * a.mv.ss * es + D * es));
    const uint32_t kbytes = (uint32_t)(a.mk.ss * es), vbytes = (uint32_t)(a.mv.ss * es);

    if (nkb > 0) {
        dma_tile<T, D, kQBN, kWaves>(smem, rk, 0, kbytes, wave, lane);
        dma_tile<T, D, kQBN, kWaves>(smem + 2 * TILE, rv, 0, vbytes, wave, lane);
    }
    for (int kb = 0; kb < nkb; ++kb) {
        const int k0 = kb * kQBN;
        wait_vmcnt<0>();
        __syncthreads();
        if (kb + 1 < nkb) {
            const int nb = (kb + 1) & 1;
            dma_tile<T, D, kQBN, kWaves>(smem + nb * TILE, rk, k0 + kQBN, kbytes, wave, lane);
            dma_tile<T, D, kQBN, kWaves>(smem + (2 + nb) * TILE, rv, k0 + kQBN, vbytes, wave, lane);
        }
        if (a.mask.causal && k0 > qw0 + 31) continue;
        const T* sK = smem + (kb & 1) * TILE;
        const T* sV = smem + (2 + (kb & 1)) * TILE;

        // S^T = K Q^T and dP^T = V dO^T: lane <-> query, in-lane key kt*32 + acc_row
        f32x16 s[2], dp[2];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            s[kt] = f32x16{};
            dp[kt] = f32x16{};
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                Frag<T> fk, fv;
                tile_row_frag<D>(fk, sK, kt * 32 + c32, 16 * c + 8 * g);
                tile_row_frag<D>(fv, sV, kt * 32 + c32, 16 * c + 8 * g);
                mma(s[kt], fk, qf[c]);
                mma(dp[kt], fv, of[c]);
            }
        }
        const bool boundary = (k0 + kQBN > kv_end) || (a.mask.causal && k0 + kQBN - 1 > qw0);
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float p = fast_exp2(__builtin_fmaf(s[kt][r], a.scale_log2, -sd[0]));
                if (boundary) {
                    const int kk = k0 + kt * 32 + acc_row(r, g);
                    if (kk >= kv_end || (a.mask.causal && kk > qi)) p = 0.f;
                }
                dp[kt][r] = p * (dp[kt][r] - sd[1]);
            }
        }
        // dQ^T += K^T dS^T over the 64 keys: chunk (kt, cc) covers keys
        // kt*32 + 16cc + {4g..4g+3, 8+4g..8+4g+3} in accumulator order
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
            for (int cc = 0; cc < 2; ++cc) {
                Frag<T> dsb;
                float dsv[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) dsv[e] = dp[kt][8 * cc + e];
                pack_frag(dsb, dsv);
                const int row0 = kt * 32 + 16 * cc + 4 * g;
#pragma unroll
                for (int t = 0; t < ND; ++t) {
                    Frag<T> fk;
                    tile_tr_frag<D>(fk, sK, row0, row0 + 8, 32 * t, lane);
                    mma(dq[t], fk, dsb);
                }
            }
        }
    }

    if (qi < S) {
        T* dqrow = static_cast<T*>(a.dq) + a.mdq.head_base(b, h) + (int64_t)qi * a.mdq.ss;
#pragma unroll
        for (int t = 0; t < ND; ++t) {
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
                const int dcol = 32 * t + 8 * rr + 4 * g;
                store4(dqrow + dcol, dq[t][4 * rr] * a.scale, dq[t][4 * rr + 1] * a.scale, dq[t][4 * rr + 2] * a.scale,
                       dq[t][4 * rr + 3] * a.scale);
            }
        }
    }
}

template <typename K>
hipError_t set_lds(K kernel, int bytes) {
    return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                               bytes);
}

template <typename T, int D>
hipError_t set_bwd_lds() {
    static hipError_t once = [] {
        const hipError_t e = set_lds(&attn_bwd_kv<T, D>, KvSmem<T, D>::BYTES);
        if (e != hipSuccess) return e;
        return set_lds(&attn_bwd_q<T, D>, QSmem<T, D>::BYTES);
    }();
    return once;
}

int padded8(int n) { return (n + 7) / 8 * 8; }

}  // namespace

template <typename T, int D>
hipError_t launch_attn_bwd(const BwdArgs& a, unsigned phases, hipStream_t stream) {
    constexpr int LPR = D / (16 / (int)sizeof(T));
    constexpr int RPB = 256 / LPR;
    const hipError_t e = set_bwd_lds<T, D>();
    if (e != hipSuccess) return e;
    if (phases & 1u) {
        const int64_t nrows = (int64_t)a.B * a.S * a.Hq;
        hipLaunchKernelGGL((attn_bwd_stats<T, D>), dim3((unsigned)((nrows + RPB - 1) / RPB)), dim3(256), 0, stream, a);
    }
    if (phases & 2u) {
        const int n = (a.S + kKvBN - 1) / kKvBN * a.Hkv * a.B;
        constexpr int lds = KvSmem<T, D>::BYTES;
        hipLaunchKernelGGL((attn_bwd_kv<T, D>), dim3(padded8(n)), dim3(256), lds, stream, a);
    }
    if (phases & 4u) {
        const int n = (a.S + kQBM - 1) / kQBM * a.Hq * a.B;
        constexpr int lds = QSmem<T, D>::BYTES;
        hipLaunchKernelGGL((attn_bwd_q<T, D>), dim3(padded8(n)), dim3(256), lds, stream, a);
    }
    return hipGetLastError();
}

template hipError_t launch_attn_bwd<float, 32>(const BwdArgs&, unsigned, hipStream_t);
template hipError_t launch_attn_bwd<float, 64>(const BwdArgs&, unsigned, hipStream_t);
template hipError_t launch_attn_bwd<float, 128>(const BwdArgs&, unsigned, hipStream_t);
template hipError_t launch_attn_bwd<bf16, 32>(const BwdArgs&, unsigned, hipStream_t);
template hipError_t launch_attn_bwd<bf16, 64>(const BwdArgs&, unsigned, hipStream_t);
template hipError_t launch_attn_bwd<bf16, 128>(const BwdArgs&, unsigned, hipStream_t);

}  // namespace fbl
