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
//                   reductions over queries that build dK/dV (the M direction
//                   of section 4.2's naming) and the group sum over
//                   the G query heads never leave registers.
//   attn_bwd_q      query-major.  A workgroup owns 128 queries of one
//                   (batch, query head) and walks the key tiles, recomputing S
//                   and dP, and accumulates dQ^T in registers (the N
//                   direction).
// Recomputing S and dP in the query-major pass costs two extra products per
// (query, key) pair; it replaces fp32 atomics, which run at ~1.3 TB/s on this
// part -- far slower than the 3 products they would save at these shapes.
// Q/dO (kv pass) and K/V (q pass) tiles are staged once per block in LDS by
// DMA and serve both reduction directions (tile invariance, section 4.2): row
// reads where the contraction runs along d, transposed reads
// (ds_read_b64_tr_b16) where it runs along tokens.
#include <type_traits>

#include "cdna4.hpp"
#include "kernels.hpp"
#include "stage.hpp"
#include "tokmap.hpp"

namespace fbl {

namespace {

constexpr int kWaves = 4;
constexpr int kKvBN = 32 * kWaves;  // keys per kv-pass workgroup
constexpr int kQBM = 32 * kWaves;   // queries per q-pass workgroup
constexpr int kQBN = 64;            // keys per q-pass tile

// ------------------------------------------------------------------ stats
// A workgroup covers kStatRows consecutive query tokens of one (batch, query
// head): every row of d elements is read by D*sizeof(T)/16 lanes (one 16-byte
// chunk each, a whole row per lane group), all of a thread's rows are in
// flight at once, and the two statistics of the block's rows are written as
// contiguous runs (the statistics rows are [B, Hq, 2, S]).
constexpr int kStatRows = 64;

template <typename T, int D>
__global__ __launch_bounds__(256) void attn_bwd_stats(BwdArgs a) {
    constexpr int EPC = 16 / (int)sizeof(T);
    constexpr int LPR = D / EPC;        // lanes per row
    constexpr int RPP = 256 / LPR;      // rows per pass of the workgroup
    constexpr int NP = kStatRows / RPP;  // passes (rows per thread)
    __shared__ float dsum[kStatRows];
    const int nsb = (a.S + kStatRows - 1) / kStatRows;
    const int bhi = (int)(blockIdx.x / nsb);
    const int h = bhi % a.Hq, b = bhi / a.Hq;
    const int s0 = (int)(blockIdx.x % nsb) * kStatRows;
    const int part = threadIdx.x % LPR;
    const T* o = static_cast<const T*>(a.o) + a.mo.head_base(b, h) + part * EPC;
    const T* g = static_cast<const T*>(a.dout) + a.mdo.head_base(b, h) + part * EPC;
    uint4 xo[NP], xg[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        const int s = s0 + p * RPP + (int)threadIdx.x / LPR;
        xo[p] = xg[p] = uint4{0u, 0u, 0u, 0u};
        if (s < a.S) {
            xo[p] = load16(o + (int64_t)s * a.mo.ss);
            xg[p] = load16(g + (int64_t)s * a.mdo.ss);
        }
    }
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        float acc = 0.f;
        if constexpr (sizeof(T) == 2) {
            const bf16x8 vo = __builtin_bit_cast(bf16x8, xo[p]), vg = __builtin_bit_cast(bf16x8, xg[p]);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc += (float)vo[e] * (float)vg[e];
        } else {
            const f32x4 vo = __builtin_bit_cast(f32x4, xo[p]), vg = __builtin_bit_cast(f32x4, xg[p]);
#pragma unroll
            for (int e = 0; e < 4; ++e) acc += vo[e] * vg[e];
        }
#pragma unroll
        for (int off = LPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
        if (part == 0) dsum[p * RPP + threadIdx.x / LPR] = acc;
    }
    __syncthreads();
    const int64_t bh = (int64_t)b * a.Hq + h;
    if (threadIdx.x < kStatRows) {
        const int s = s0 + (int)threadIdx.x;
        if (s < a.S) {
            const float lse = a.lse[bh * a.S + s];
            a.stats[2 * bh * a.S + s] = lse == -INFINITY ? INFINITY : lse * kLog2e;
            a.stats[(2 * bh + 1) * a.S + s] = dsum[threadIdx.x];
        }
    }
}

// ------------------------------------------------------------- kv pass
// FUSED: the whole backward in this one pass, for key/value sequences of at
// most one key block (kKvBN keys): every workgroup then holds all the keys of
// its (batch, kv head), so it also forms each query block's row statistics
// (D from O and dO, LSE from the forward's output) and its dQ = scale dS K
// completely -- no statistics pass, no stored dS, no dQ pass.
template <typename T, int D, bool FUSED>
struct KvCfg {
    static constexpr int BQ = D == 128 ? 32 : 64;  // queries per block (register budget)
    static constexpr int NQT = BQ / 32;
    static constexpr int TILE = BQ * D;             // elements of one Q or dO tile
    static constexpr int TB = TILE * (int)sizeof(T);
    // LDS: Q0 Q1 dO0 dO1 tiles, then lse2 0/1 and D 0/1 (256 bytes each: one
    // 64-lane dword DMA; the first BQ floats are used)
    static constexpr int OFF_STATS = 4 * TB;
    // FUSED: the block of kKvBN K rows (the dQ product's operand, staged once)
    // and one block of dS, [BQ queries][DS_PITCH] of T (rows padded by 8
    // elements: 16-byte aligned, and consecutive rows on other LDS banks)
    static constexpr int OFF_K = OFF_STATS + 4 * 256;
    static constexpr int KT_BYTES = kKvBN * D * (int)sizeof(T);
    static constexpr int DS_PITCH = kKvBN + 8;
    static constexpr int OFF_DS = OFF_K + KT_BYTES;
    // FUSED with bf16 storage: the block's O rows too (staged with Q and dO, two
    // buffers), so that D is formed from LDS; fp32 forms it from global memory
    static constexpr bool O_TILE = FUSED && sizeof(T) == 2;
    static constexpr int OFF_O = (OFF_DS + BQ * DS_PITCH * (int)sizeof(T) + 1023) / 1024 * 1024;
    static constexpr int BYTES = !FUSED ? OFF_STATS + 4 * 256
                                 : O_TILE ? OFF_O + 2 * TB
                                          : OFF_DS + BQ * DS_PITCH * (int)sizeof(T);
    static_assert(BYTES <= 160 * 1024, "LDS of one workgroup");
    static_assert(OFF_K % 1024 == 0, "the K block starts on a 1 KB boundary");
    static_assert(OFF_O % 1024 == 0 && TB % 1024 == 0, "the O tiles start on 1 KB boundaries");
};

template <typename T, int D, bool FUSED>
__device__ __forceinline__ void kv_pass(const BwdArgs& a) {
    using C = KvCfg<T, D, FUSED>;
    constexpr int NC = D / 16;
    constexpr int ND = D / 32;
    constexpr int BQ = C::BQ;
    constexpr int NQT = C::NQT;
    constexpr int TB = C::TB;
    constexpr bool kBf16 = sizeof(T) == 2;
    extern __shared__ __attribute__((aligned(1024))) unsigned char kv_smem[];
    const uint32_t lds = lds_addr(kv_smem);  // LDS byte address of the tiles

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = lane >> 5;
    const int c32 = lane & 31;
    const int S = a.S, Skv = a.Skv;  // query tokens, key tokens
    const int nkb = (Skv + kKvBN - 1) / kKvBN;
    const int logical = xcd_logical_id(blockIdx.x, nkb * a.Hkv * a.B, gridDim.x);
    if (logical < 0) return;
    const int kblk = logical % nkb;
    const int hk = (logical / nkb) % a.Hkv;
    const int b = logical / (nkb * a.Hkv);
    const int G_ = a.Hq / a.Hkv;
    int kv_end = Skv;
    if (a.mask.kv_len) kv_end = min(max(a.mask.kv_len[b], 0), Skv);
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
        if (key < Skv) {
            const T* kp = kbase + (int64_t)key * a.mk.ss + 16 * c + 8 * g;
            const T* vp = vbase + (int64_t)key * a.mv.ss + 16 * c + 8 * g;
            if constexpr (kBf16) {
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

    const int qb_start = a.mask.causal ? (k0 / BQ) : 0;
    const int nqb = (S + BQ - 1) / BQ;
    const int per_head = nqb - qb_start;
    const int n_iter = (k0 < kv_end) ? G_ * per_head : 0;
    // blocks needing a mask: all of them when this block's keys run past
    // kv_end; else (causal) those holding a query before one of the keys
    int n_mask = 0;
    if (k0 + kKvBN > kv_end) n_mask = per_head;
    else if (a.mask.causal) n_mask = min(per_head, (k0 + kKvBN - 2) / BQ - qb_start + 1);

    DmaPlan<T, D, BQ, kWaves> pq, po;
    pq.init((uint32_t)(a.mq.ss * es), wave, lane);
    po.init((uint32_t)(a.mdo.ss * es), wave, lane);
    const uint32_t qbytes = (uint32_t)(a.mq.ss * es), obytes = (uint32_t)(a.mdo.ss * es);
    const uint32_t qspan = (uint32_t)((int64_t)(S - 1) * a.mq.ss * es + D * es);
    const uint32_t ospan = (uint32_t)((int64_t)(S - 1) * a.mdo.ss * es + D * es);
    DmaPlan<T, D, BQ, kWaves> pof;  // O rows (FUSED, bf16)
    const uint32_t ofbytes = (uint32_t)(a.mo.ss * es);
    const uint32_t ofspan = (uint32_t)((int64_t)(S - 1) * a.mo.ss * es + D * es);
    if constexpr (C::O_TILE) pof.init(ofbytes, wave, lane);

    auto issue = [&](int it) {
        const int buf = it & 1;
        const int h = hk * G_ + it / per_head;
        const int q0 = (qb_start + it % per_head) * BQ;
        const Rsrc rq = make_rsrc(static_cast<const T*>(a.q) + a.mq.head_base(b, h), qspan);
        const Rsrc ro = make_rsrc(static_cast<const T*>(a.dout) + a.mdo.head_base(b, h), ospan);
        pq.issue(lds + buf * TB, rq, (uint32_t)q0 * qbytes, wave);
        po.issue(lds + (2 + buf) * TB, ro, (uint32_t)q0 * obytes, wave);
        if constexpr (C::O_TILE) {
            const Rsrc rof = make_rsrc(static_cast<const T*>(a.o) + a.mo.head_base(b, h), ofspan);
            pof.issue(lds + C::OFF_O + buf * TB, rof, (uint32_t)q0 * ofbytes, wave);
        }
        if constexpr (FUSED) {  // wave 0: the forward's LSE of the block's queries (D is formed in the step)
            if (wave == 0) {
                const float* row = a.lse + ((int64_t)b * a.Hq + h) * S;
                dma4(make_rsrc(row, (uint32_t)(S * 4)), lds + C::OFF_STATS + buf * 256, (uint32_t)lane * 4u,
                     (uint32_t)q0 * 4u);
            }
        } else if (wave < 2) {  // wave 0: lse2 of the block's queries, wave 1: D
            const float* row = a.stats + (2 * ((int64_t)b * a.Hq + h) + wave) * S;
            dma4(make_rsrc(row, (uint32_t)(S * 4)), lds + C::OFF_STATS + (2 * wave + buf) * 256, (uint32_t)lane * 4u, (uint32_t)q0 * 4u);
        }
    };
    // FUSED: D_i = sum_k dO_ik O_ik of the block's BQ rows of query head h,
    // TPR threads per row, into the block's D slot
    auto form_d = [&](int buf, int h, int q0) {
        constexpr int EPC = 16 / (int)sizeof(T);
        constexpr int TPR = 256 / BQ;           // threads per row
        constexpr int CPT = D / (TPR * EPC);    // 16-byte chunks per thread
        static_assert(CPT >= 1 && D % (TPR * EPC) == 0, "whole chunks per thread");
        const int r = (int)threadIdx.x / TPR, part = (int)threadIdx.x % TPR;
        const int sq = q0 + r;
        float acc = 0.f;
        if constexpr (C::O_TILE) {  // both rows from the staged tiles (rows past S are zeros)
            using G = TileGeom<T, D>;
#pragma unroll
            for (int c = 0; c < CPT; ++c) {
                const uint32_t eo = 2u * (uint32_t)G::off(r, (part * CPT + c) * EPC);
                const bf16x8 vo = lds_b128(lds + C::OFF_O + buf * TB + eo, 0u);
                const bf16x8 vg = lds_b128(lds + (2 + buf) * TB + eo, 0u);
#pragma unroll
                for (int e = 0; e < 8; ++e) acc += (float)vo[e] * (float)vg[e];
            }
        } else if (sq < S) {
            const T* orow = static_cast<const T*>(a.o) + a.mo.head_base(b, h) + (int64_t)sq * a.mo.ss;
            const T* grow = static_cast<const T*>(a.dout) + a.mdo.head_base(b, h) + (int64_t)sq * a.mdo.ss;
#pragma unroll
            for (int c = 0; c < CPT; ++c) {
                const int col = (part * CPT + c) * EPC;
                const uint4 xo = load16(orow + col), xg = load16(grow + col);
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
        }
#pragma unroll
        for (int off = TPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
        if (part == 0) reinterpret_cast<float*>(kv_smem + C::OFF_STATS + (2 + buf) * 256)[r] = acc;
    };

    // per-lane LDS addresses into buffer 0; `flip` moves them to the other buffer
    LaneOffsets<D> lo;
    if constexpr (kBf16) lo.init(lds_addr(kv_smem), lane);
    uint32_t st_addr = lds_addr(kv_smem) + C::OFF_STATS + 16u * g;  // lse2 of queries 4g.. of buffer 0
    int32_t flip = TB;

    auto compute = [&](auto mask_c, int buf, int q0) {
        constexpr bool MASK = decltype(mask_c)::value;
        const T* sQ = reinterpret_cast<const T*>(kv_smem) + buf * C::TILE;
        const T* sdO = reinterpret_cast<const T*>(kv_smem) + (2 + buf) * C::TILE;
        // S = Q K_w^T and dP = dO V_w^T: lane <-> key, in-lane query 32qt + acc_row
        f32x16 s[NQT], dp[NQT];
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt) {
            s[qt] = f32x16{};
            dp[qt] = f32x16{};
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                Frag<T> fq, fo;
                if constexpr (kBf16) {
                    fq.v = lds_b128(lo.row[c], qt * 32 * D * 2);
                    fo.v = lds_b128(lo.row[c], 2 * TB + qt * 32 * D * 2);
                } else {
                    tile_row_frag<D>(fq, sQ, qt * 32 + c32, 16 * c + 8 * g);
                    tile_row_frag<D>(fo, sdO, qt * 32 + c32, 16 * c + 8 * g);
                }
                mma(s[qt], fq, kf[c]);
                mma(dp[qt], fo, vf[c]);
            }
        }
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt) {
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
                f32x4 l4 = *(const FBL_LDS f32x4*)(uintptr_t)(st_addr + (qt * 32 + 8 * rr) * 4);
                if constexpr (FUSED) {  // the forward's natural-log LSE: to log2 units, +inf for an empty row
#pragma unroll
                    for (int j = 0; j < 4; ++j) l4[j] = l4[j] == -INFINITY ? INFINITY : l4[j] * kLog2e;
                }
                const f32x4 d4 = *(const FBL_LDS f32x4*)(uintptr_t)(st_addr + 512 + (qt * 32 + 8 * rr) * 4);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int r = 4 * rr + j;
                    float p = fast_exp2(__builtin_fmaf(s[qt][r], a.scale_log2, -l4[j]));
                    if constexpr (MASK) {
                        if (!key_ok || (a.mask.causal && key > q0 + qt * 32 + acc_row(r, g))) p = 0.f;
                    }
                    s[qt][r] = p;
                    dp[qt][r] = p * (dp[qt][r] - d4[j]);
                }
            }
        }
        // dV^T += dO^T P and dK^T += Q^T dS, contracting over the block's queries:
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
#pragma unroll
                for (int t = 0; t < ND; ++t) {
                    Frag<T> fdo, fq;
                    if constexpr (kBf16) {
                        const uint32_t rb = (qt * 32 + 16 * cc) * D * 2;
                        const bf16x4 o0 = lds_tr(lo.tr[t][0], 2 * TB + rb), o1 = lds_tr(lo.tr[t][1], 2 * TB + rb);
                        const bf16x4 x0 = lds_tr(lo.tr[t][0], rb), x1 = lds_tr(lo.tr[t][1], rb);
                        fdo.v = bf16x8{o0[0], o0[1], o0[2], o0[3], o1[0], o1[1], o1[2], o1[3]};
                        fq.v = bf16x8{x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
                    } else {
                        const int row0 = qt * 32 + 16 * cc + 4 * g;
                        tile_tr_frag<D>(fdo, sdO, row0, row0 + 8, 32 * t, lane);
                        tile_tr_frag<D>(fq, sQ, row0, row0 + 8, 32 * t, lane);
                    }
                    mma(dv[t], fdo, pb);
                    mma(dk[t], fq, dsb);
                }
            }
        }
        if constexpr (FUSED) {  // dS of the wave's 32 keys into the block's dS rows: [query][key]
            T* sds = reinterpret_cast<T*>(kv_smem + C::OFF_DS);
#pragma unroll
            for (int qt = 0; qt < NQT; ++qt)
#pragma unroll
                for (int r = 0; r < 16; ++r) store_out(sds + (qt * 32 + acc_row(r, g)) * C::DS_PITCH + key - k0, dp[qt][r]);
        }
    };
    // FUSED: dQ of the block, dQ^T(d x queries) = scale K^T dS^T over the
    // workgroup's kKvBN keys -- A = K^T from the K block (transposed reads),
    // B = dS^T from the dS rows (row reads); NQT x ND output tiles spread over
    // the four wavefronts; query row q of head h at q0 + 32qt + lane % 32
    // FUSED: dQ of a block is computed after its dS and (bf16) stored at the
    // start of the next step, after that step's wait: its stores then have a
    // whole step to retire before the next wait (which covers every
    // outstanding memory operation of the wavefront).  One output tile per
    // wavefront.
    static_assert(!FUSED || NQT * ND <= kWaves, "at most one dQ tile per wavefront");
    f32x16 dq_acc = f32x16{};
    int dq_h = -1, dq_q0 = 0;  // the block whose dQ tile is held (dq_h < 0: none)
    auto dq_flush_now = [&]() {
        if (dq_h >= 0) {
            const int qt = wave / ND, t = wave % ND;
            const int qi = dq_q0 + qt * 32 + c32;
            if (qi < S) {
                T* dqrow = static_cast<T*>(a.dq) + a.mdq.head_base(b, dq_h) + (int64_t)qi * a.mdq.ss;
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) {
                    const int dcol = 32 * t + 8 * rr + 4 * g;
                    store4(dqrow + dcol, dq_acc[4 * rr] * a.scale, dq_acc[4 * rr + 1] * a.scale,
                           dq_acc[4 * rr + 2] * a.scale, dq_acc[4 * rr + 3] * a.scale);
                }
            }
            dq_h = -1;
        }
    };

    auto dq_block = [&](int h, int q0) {
        const T* sk = reinterpret_cast<const T*>(kv_smem + C::OFF_K);
        const T* sds = reinterpret_cast<const T*>(kv_smem + C::OFF_DS);
        if (wave < NQT * ND) {
            const int qt = wave / ND, t = wave % ND;
            f32x16 acc = f32x16{};
#pragma unroll
            for (int kc = 0; kc < kKvBN / 16; ++kc) {
                Frag<T> fk, fs;
                tile_tr_frag<D>(fk, sk, 16 * kc + 8 * g, 16 * kc + 8 * g + 4, 32 * t, lane);
                lds_row_frag(fs, sds + (qt * 32 + c32) * C::DS_PITCH + 16 * kc + 8 * g);
                mma(acc, fk, fs);
            }
            if constexpr (kBf16) {
                dq_acc = acc;
                dq_h = h;
                dq_q0 = q0;
            } else {  // fp32: no registers to spare for holding it
                const int qi = q0 + qt * 32 + c32;
                if (qi < S) {
                    T* dqrow = static_cast<T*>(a.dq) + a.mdq.head_base(b, h) + (int64_t)qi * a.mdq.ss;
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr) {
                        const int dcol = 32 * t + 8 * rr + 4 * g;
                        store4(dqrow + dcol, acc[4 * rr] * a.scale, acc[4 * rr + 1] * a.scale,
                               acc[4 * rr + 2] * a.scale, acc[4 * rr + 3] * a.scale);
                    }
                }
            }
        }
    };
    auto step = [&](auto mask_c, int it) {
        const int buf = it & 1;
        wait_vmcnt<0>();
        __syncthreads();  // block `it` landed; block it-1's buffers are free
        if (it + 1 < n_iter) issue(it + 1);
        const int q0 = (qb_start + it % per_head) * BQ;
        const int h = hk * G_ + it / per_head;
        if constexpr (FUSED) {
            if constexpr (kBf16) dq_flush_now();  // the previous block's dQ tile
            form_d(buf, h, q0);
            __syncthreads();  // the block's D row is in LDS
        }
        // a wave whose keys all follow every query of the block has nothing to add
        if (!(a.mask.causal && q0 + BQ - 1 < kw0) && kw0 < kv_end) {
            compute(mask_c, buf, q0);
        } else if constexpr (FUSED) {  // its dS columns are zero
            T* sds = reinterpret_cast<T*>(kv_smem + C::OFF_DS);
#pragma unroll
            for (int qt = 0; qt < NQT; ++qt)
#pragma unroll
                for (int r = 0; r < 16; ++r) store_out(sds + (qt * 32 + acc_row(r, g)) * C::DS_PITCH + key - k0, 0.f);
        }
        if constexpr (FUSED) {
            __syncthreads();  // every wavefront's dS columns are in LDS
            dq_block(h, q0);
        }
        if constexpr (kBf16) {
#pragma unroll
            for (int c = 0; c < NC; ++c) lo.row[c] += flip;
#pragma unroll
            for (int t = 0; t < ND; ++t) {
                lo.tr[t][0] += flip;
                lo.tr[t][1] += flip;
            }
        }
        st_addr += flip / TB * 256;
        flip = -flip;
    };

    if constexpr (FUSED) {  // the workgroup's K rows for the dQ products (rows past S_kv read as zeros)
        DmaPlan<T, D, kKvBN, kWaves> pk;
        pk.init((uint32_t)(a.mk.ss * es), wave, lane);
        pk.issue(lds + C::OFF_K, make_rsrc(kbase, (uint32_t)((int64_t)(Skv - 1) * a.mk.ss * es + D * es)), 0u, wave);
    }
    if constexpr (FUSED) {  // no allowed key (kv_len = 0): dQ of the whole group is zero
        if (n_iter == 0) {
            for (int64_t i = threadIdx.x; i < (int64_t)G_ * S * (D / 4); i += 256) {
                const int c4 = (int)(i % (D / 4));
                const int sq = (int)((i / (D / 4)) % S);
                const int h = hk * G_ + (int)(i / ((int64_t)S * (D / 4)));
                store4(static_cast<T*>(a.dq) + a.mdq.head_base(b, h) + (int64_t)sq * a.mdq.ss + 4 * c4, 0.f, 0.f, 0.f,
                       0.f);
            }
        }
    }
    if (n_iter > 0) issue(0);
    int it = 0;
    for (int hh = 0; hh < G_ && n_iter > 0; ++hh) {
        for (int j = 0; j < n_mask; ++j, ++it) step(std::true_type{}, it);
        for (int j = n_mask; j < per_head; ++j, ++it) step(std::false_type{}, it);
    }
    if constexpr (FUSED && kBf16) dq_flush_now();

    // dK (times scale) and dV rows of this wave's keys: lane <-> key, 4 consecutive d per store
    if (key < Skv) {
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

template <typename T, int D>
__global__ __launch_bounds__(256, 1) void attn_bwd_kv(BwdArgs a) {
    kv_pass<T, D, false>(a);
}

// the one-launch backward (keys within one block of kKvBN)
template <typename T, int D>
__global__ __launch_bounds__(256, 1) void attn_bwd_fused(BwdArgs a) {
    kv_pass<T, D, true>(a);
}

// --------------------------------------------------------------- q pass
template <typename T, int D>
struct QSmem {
    static constexpr int TILE = kQBN * D;
    static constexpr int TB = TILE * (int)sizeof(T);
    static constexpr int BYTES = 4 * TB;  // K0 K1 V0 V1
};

template <typename T, int D>
__global__ __launch_bounds__(256, sizeof(T) == 2 ? 2 : 1) void attn_bwd_q(BwdArgs a) {
    constexpr int NC = D / 16;
    constexpr int ND = D / 32;
    constexpr int TILE = QSmem<T, D>::TILE;
    constexpr int TB = QSmem<T, D>::TB;
    constexpr bool kBf16 = sizeof(T) == 2;
    extern __shared__ __attribute__((aligned(1024))) unsigned char q_smem[];
    T* smem = reinterpret_cast<T*>(q_smem);
    const uint32_t lds = lds_addr(q_smem);  // LDS byte address of the tiles

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
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
    const int Skv = a.Skv;  // key tokens
    int kv_end = Skv;
    if (a.mask.kv_len) kv_end = min(max(a.mask.kv_len[b], 0), Skv);
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
                if constexpr (kBf16) {
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
    float lse2 = INFINITY, drow = 0.f;  // this lane's query row statistics
    if (qi < S) {
        const int64_t bh = (int64_t)b * a.Hq + h;
        lse2 = a.stats[2 * bh * S + qi];
        drow = a.stats[(2 * bh + 1) * S + qi];
    }

    f32x16 dq[ND];  // dQ^T: rows = d (32t + acc_row), columns = queries (lane)
#pragma unroll
    for (int t = 0; t < ND; ++t) dq[t] = f32x16{};

    const uint32_t es = sizeof(T);
    const Rsrc rk = make_rsrc(static_cast<const T*>(a.k) + a.mk.head_base(b, hk),
                              (uint32_t)((int64_t)(Skv - 1) * a.mk.ss * es + D * es));
    const Rsrc rv = make_rsrc(static_cast<const T*>(a.v) + a.mv.head_base(b, hk),
                              (uint32_t)((int64_t)(Skv - 1) * a.mv.ss * es + D * es));
    const uint32_t kbytes = (uint32_t)(a.mk.ss * es), vbytes = (uint32_t)(a.mv.ss * es);
    DmaPlan<T, D, kQBN, kWaves> pk, pv;
    pk.init(kbytes, wave, lane);
    pv.init(vbytes, wave, lane);
    LaneOffsets<D> lo;
    if constexpr (kBf16) lo.init(lds_addr(q_smem), lane);
    int32_t flip = TB;

    auto tile = [&](auto mask_c, int k0) {
        constexpr bool MASK = decltype(mask_c)::value;
        const int BUF = (k0 / kQBN) & 1;
        // S^T = K Q^T and dP^T = V dO^T: lane <-> query, in-lane key kt*32 + acc_row
        f32x16 s[2], dp[2];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            s[kt] = f32x16{};
            dp[kt] = f32x16{};
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                Frag<T> fk, fv;
                if constexpr (kBf16) {
                    fk.v = lds_b128(lo.row[c], kt * 32 * D * 2);
                    fv.v = lds_b128(lo.row[c], 2 * TB + kt * 32 * D * 2);
                } else {
                    tile_row_frag<D>(fk, smem + BUF * TILE, kt * 32 + c32, 16 * c + 8 * g);
                    tile_row_frag<D>(fv, smem + (2 + BUF) * TILE, kt * 32 + c32, 16 * c + 8 * g);
                }
                mma(s[kt], fk, qf[c]);
                mma(dp[kt], fv, of[c]);
            }
        }
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float p = fast_exp2(__builtin_fmaf(s[kt][r], a.scale_log2, -lse2));
                if constexpr (MASK) {
                    const int kk = k0 + kt * 32 + acc_row(r, g);
                    if (kk >= kv_end || (a.mask.causal && kk > qi)) p = 0.f;
                }
                dp[kt][r] = p * (dp[kt][r] - drow);
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
#pragma unroll
                for (int t = 0; t < ND; ++t) {
                    Frag<T> fk;
                    if constexpr (kBf16) {
                        const uint32_t rb = (kt * 32 + 16 * cc) * D * 2;
                        const bf16x4 x0 = lds_tr(lo.tr[t][0], rb), x1 = lds_tr(lo.tr[t][1], rb);
                        fk.v = bf16x8{x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
                    } else {
                        const int row0 = kt * 32 + 16 * cc + 4 * g;
                        tile_tr_frag<D>(fk, smem + BUF * TILE, row0, row0 + 8, 32 * t, lane);
                    }
                    mma(dq[t], fk, dsb);
                }
            }
        }
    };

    auto step = [&](auto mask_c, int kb) {
        const int k0 = kb * kQBN;
        wait_vmcnt<0>();
        __syncthreads();
        if (kb + 1 < nkb) {
            const uint32_t nb = (uint32_t)((kb + 1) & 1);
            pk.issue(lds + nb * TB, rk, (uint32_t)(k0 + kQBN) * kbytes, wave);
            pv.issue(lds + (2 + nb) * TB, rv, (uint32_t)(k0 + kQBN) * vbytes, wave);
        }
        tile(mask_c, k0);
        if constexpr (kBf16) {
#pragma unroll
            for (int c = 0; c < NC; ++c) lo.row[c] += flip;
#pragma unroll
            for (int t = 0; t < ND; ++t) {
                lo.tr[t][0] += flip;
                lo.tr[t][1] += flip;
            }
        }
        flip = -flip;
    };

    if (nkb > 0) {
        pk.issue(lds, rk, 0u, wave);
        pv.issue(lds + 2 * TB, rv, 0u, wave);
    }
    const int n_full = min(nkb, min(kv_end, a.mask.causal ? q0 + 1 : Skv) / kQBN);
    for (int kb = 0; kb < n_full; ++kb) step(std::false_type{}, kb);
    for (int kb = n_full; kb < nkb; ++kb) step(std::true_type{}, kb);

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

// Explicit instantiations: the host-side launch stubs of every kernel used
// below.  bf16 storage runs the software-pipelined passes of attn_bwd_kv.hip,
// attn_bwd_dq.hip and attn_bwd_q.hip; the two passes here serve fp32.
#define FBL_BWD_KERNELS_F32(D)                                     \
    template __global__ void attn_bwd_stats<float, D>(BwdArgs);   \
    template __global__ void attn_bwd_kv<float, D>(BwdArgs);        \
    template __global__ void attn_bwd_q<float, D>(BwdArgs);
FBL_BWD_KERNELS_F32(32)
FBL_BWD_KERNELS_F32(64)
FBL_BWD_KERNELS_F32(128)
#undef FBL_BWD_KERNELS_F32
template __global__ void attn_bwd_stats<bf16, 32>(BwdArgs);
template __global__ void attn_bwd_stats<bf16, 64>(BwdArgs);
template __global__ void attn_bwd_stats<bf16, 128>(BwdArgs);

template <int D>
hipError_t set_bwd_lds_f32() {
    const hipError_t e = ensure_dynamic_lds<&attn_bwd_kv<float, D>>(KvCfg<float, D, false>::BYTES);
    if (e != hipSuccess) return e;
    return ensure_dynamic_lds<&attn_bwd_q<float, D>>(QSmem<float, D>::BYTES);
}

int padded8(int n) { return (n + 7) / 8 * 8; }

}  // namespace

template <typename T, int D>
hipError_t launch_attn_bwd_fused(const BwdArgs& a, hipStream_t stream) {
    constexpr int lds = KvCfg<T, D, true>::BYTES;
    const hipError_t e = ensure_dynamic_lds<&attn_bwd_fused<T, D>>(lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((attn_bwd_fused<T, D>), dim3(padded8(a.Hkv * a.B)), dim3(256), lds, stream, a);
    return hipGetLastError();
}

template hipError_t launch_attn_bwd_fused<float, 32>(const BwdArgs&, hipStream_t);
template hipError_t launch_attn_bwd_fused<float, 64>(const BwdArgs&, hipStream_t);
template hipError_t launch_attn_bwd_fused<bf16, 32>(const BwdArgs&, hipStream_t);
template hipError_t launch_attn_bwd_fused<bf16, 64>(const BwdArgs&, hipStream_t);
template hipError_t launch_attn_bwd_fused<bf16, 128>(const BwdArgs&, hipStream_t);

template <typename T, int D>
hipError_t launch_attn_bwd(const BwdArgs& a, unsigned phases, hipStream_t stream) {
    if constexpr (sizeof(T) == 4) {
        const hipError_t e = set_bwd_lds_f32<D>();
        if (e != hipSuccess) return e;
    }
    if (phases & 1u) {
        const int64_t nblk = (int64_t)((a.S + kStatRows - 1) / kStatRows) * a.B * a.Hq;
        hipLaunchKernelGGL((attn_bwd_stats<T, D>), dim3((unsigned)nblk), dim3(256), 0, stream, a);
    }
    if (phases & 2u) {
        if constexpr (sizeof(T) == 2) {
            const hipError_t ek = launch_attn_bwd_kv_bf16<D>(a, a.kv_tile, stream);
            if (ek != hipSuccess) return ek;
        } else {
            const int n = (a.Skv + kKvBN - 1) / kKvBN * a.Hkv * a.B;
            constexpr int lds = KvCfg<T, D, false>::BYTES;
            hipLaunchKernelGGL((attn_bwd_kv<T, D>), dim3(padded8(n)), dim3(256), lds, stream, a);
        }
    }
    if (phases & 4u) {
        if constexpr (sizeof(T) == 2) {
            const hipError_t eq =
                a.ds ? launch_attn_bwd_dq_bf16<D>(a, a.dq_tile, stream) : launch_attn_bwd_q_bf16<D>(a, stream);
            if (eq != hipSuccess) return eq;
        } else {
            const int n = (a.S + kQBM - 1) / kQBM * a.Hq * a.B;
            constexpr int lds = QSmem<T, D>::BYTES;
            hipLaunchKernelGGL((attn_bwd_q<T, D>), dim3(padded8(n)), dim3(256), lds, stream, a);
        }
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
