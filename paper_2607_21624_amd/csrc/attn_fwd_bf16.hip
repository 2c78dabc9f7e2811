// attn_fwd_bf16.hip -- attention forward for bf16 storage, gfx950, templated
// on its tile (attn_tiles.hpp).
//
// A workgroup of NW wavefronts covers 32*QT*NW queries of one (batch, query
// head); each wavefront owns 32*QT queries, whose Q rows it holds as MFMA
// operands for the whole pass.  Key/value tiles of 32*KT rows (the R-Tile,
// paper section 4.2) stream from the token-major tensors into LDS: row r of a
// tile is token k0 + r of kv head hk, at base + b*sb + (k0 + r)*ss + hk*sh,
// so the head split and transpose of the multi-head attention chain (section
// 4.3.1) are a change of base address, never a copy.  Tiles are double
// buffered and filled by LDS DMA; one barrier per tile.
//
// No operand needs a physical transpose (section 4.2's tile invariance: one
// staged tile serves both reduction directions):
//   S^T = K Q^T     A = K rows (LDS row reads), B = Q rows (registers); the
//                   accumulator holds one query per lane column, so the
//                   softmax row max and sum over keys are in-lane plus one
//                   exchange between the two 32-lane halves;
//   O^T += V^T P^T  A = V^T by LDS transposed reads (ds_read_b64_tr_b16),
//                   B = P^T straight from the S^T accumulator registers.
// With QT = 2 every K and V fragment read from LDS feeds two products (one
// per query tile), which halves the LDS traffic per product.  QK^T followed
// by PV is the consecutive matrix-product pair of section 4.4.2, fused here
// under one tile configuration.
//
// Online softmax in base 2 with scale*log2(e) folded into one FMA per score.
// The running maximum is raised only when a tile exceeds it by more than 2^8
// (a stale maximum leaves every probability <= 256 and cancels in O / l), so
// almost no tile rescales the O accumulator.  The saved LSE is converted to
// natural log at the store.
//
// Software pipeline over key tiles j: while the softmax of tile j runs on the
// vector ALUs, the scores of tile j+1 are already in the matrix cores.  K
// tiles are fetched two ahead, V tiles one ahead:
//   iteration j: wait for K_{j+1}, V_j; barrier; DMA K_{j+2} -> Kbuf[j%2],
//                V_{j+1} -> Vbuf[(j+1)%2]; S_{j+1} = K_{j+1} Q^T interleaved
//                with softmax(S_j); O^T += V_j^T P_j^T.
// The loop runs in pairs so buffer and score-array parities are compile-time.
#include <type_traits>

#include "attn_tiles.hpp"
#include "cdna4.hpp"
#include "kernels.hpp"
#include "stage.hpp"
#include "tokmap.hpp"

namespace fbl {

namespace {

constexpr float kRescaleSlack = 8.0f;  // log2 of the largest unnormalised probability

// (the second launch bound is the wavefronts per SIMD that OCC workgroups
// per CU give: a tile built for one wavefront per SIMD gets the whole
// register file)
template <int D, int QT, int KT, int NW, int OCC>
__global__ __launch_bounds__(64 * NW, (NW * OCC + 3) / 4) void attn_fwd_bf16(FwdArgs a) {
    constexpr int NC = D / 16;      // k-chunks over the head dim
    constexpr int ND = D / 32;      // 32-wide output column blocks
    constexpr int BM = 32 * QT * NW;  // queries per workgroup
    constexpr int BN = 32 * KT;       // keys per tile
    constexpr uint32_t TB = BN * D * 2;
    static_assert(3 * TB + (32 * (KT - 1) + 16) * D * 2 < 65536, "LDS offsets fit the 16-bit immediate");
    extern __shared__ __attribute__((aligned(1024))) unsigned char fwdb_smem[];  // K0 K1 V0 V1
    const uint32_t lds = lds_addr(fwdb_smem);

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = lane >> 5;
    const int c32 = lane & 31;
    const int S = a.S;
    const int nqb = (S + BM - 1) / BM;
    int rank, bh;
    if (!rank_major_item(blockIdx.x, nqb, a.Hq * a.B, rank, bh)) return;
    const int h = bh % a.Hq;
    const int b = bh / a.Hq;
    // causal: the last query blocks see the most keys; start them first
    const int qb = a.mask.causal ? (nqb - 1 - rank) : rank;
    const int hk = h / (a.Hq / a.Hkv);

    const int Skv = a.Skv;
    int kv_end = Skv;
    if (a.mask.kv_len) kv_end = min(max(a.mask.kv_len[b], 0), Skv);
    const int q0 = qb * BM;
    const int qw0 = q0 + wave * 32 * QT;  // first query of this wave; query tile qt starts at qw0 + 32 qt
    int k_hi = kv_end;
    if (a.mask.causal) k_hi = min(k_hi, q0 + BM);
    const int nkb = (k_hi + BN - 1) / BN;

    // the softmax FMA below needs a non-negative scale: fold the sign into Q
    const bool neg = a.scale_log2 < 0.f;
    const float c = neg ? -a.scale_log2 : a.scale_log2;

    // Q^T as the B operand: lane <-> query, in-lane d = 16c + 8g + e
    Frag<bf16> qf[QT][NC];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        const int qi = qw0 + 32 * qt + c32;
        const bf16* qrow = static_cast<const bf16*>(a.q) + a.mq.head_base(b, h) + (int64_t)qi * a.mq.ss;
#pragma unroll
        for (int cc = 0; cc < NC; ++cc) {
            uint4 x = uint4{0u, 0u, 0u, 0u};
            if (qi < S) x = load16(qrow + 16 * cc + 8 * g);
            if (neg) { x.x ^= 0x80008000u; x.y ^= 0x80008000u; x.z ^= 0x80008000u; x.w ^= 0x80008000u; }
            qf[qt][cc].v = __builtin_bit_cast(bf16x8, x);
        }
    }

    f32x16 oacc[QT][ND];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt)
#pragma unroll
        for (int t = 0; t < ND; ++t) oacc[qt][t] = f32x16{};
    float m[QT], l[QT];  // running maximum (log2 units, equal in both lane halves); this half's running sum
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        m[qt] = -INFINITY;
        l[qt] = 0.f;
    }

    const Rsrc rk = make_rsrc(static_cast<const bf16*>(a.k) + a.mk.head_base(b, hk),
                              (uint32_t)((int64_t)(Skv - 1) * a.mk.ss * 2 + D * 2));
    const Rsrc rv = make_rsrc(static_cast<const bf16*>(a.v) + a.mv.head_base(b, hk),
                              (uint32_t)((int64_t)(Skv - 1) * a.mv.ss * 2 + D * 2));
    const uint32_t kbytes = (uint32_t)(a.mk.ss * 2), vbytes = (uint32_t)(a.mv.ss * 2);
    DmaPlan<bf16, D, BN, NW> dk, dv;
    dk.init(kbytes, wave, lane);
    dv.init(vbytes, wave, lane);
    LaneOffsets<D> lo;
    lo.init(lds, lane);

    f32x16 sc[2][KT][QT];  // scores of two tiles: [parity][32-key half][query tile]

    // K fragment k of a tile: 32-key half k / NC, d-chunk k % NC
    constexpr int NQK = KT * NC;
    constexpr int LEAD = NQK < 4 ? NQK : 4;  // fragment reads ahead of their products
    Frag<bf16> fk[NQK];
    auto read_k = [&](int kbuf, int k) __attribute__((always_inline)) {
        fk[k].v = lds_b128(lo.row[k % NC], kbuf * TB + (k / NC) * 32 * D * 2);
    };
    // V^T fragment n of a tile: d-block n % ND, 16-key chunk (n / ND) % 2 of half n / (2 ND)
    constexpr int NPV = KT * 2 * ND;
    constexpr int VLEAD = NPV < 4 ? NPV : 4;
    bf16x4 vv[2 * NPV];
    auto read_v = [&](int vbuf, int n) __attribute__((always_inline)) {
        const int t = n % ND, cc = (n / ND) % 2, kt = n / (2 * ND);
        const uint32_t off = (2 + vbuf) * TB + (kt * 32 + 16 * cc) * D * 2;
        vv[2 * n] = lds_tr(lo.tr[t][0], off);
        vv[2 * n + 1] = lds_tr(lo.tr[t][1], off);
    };
    // the S^T products of key fragment k into parity PP, one per query tile
    auto qk_slot = [&](auto pp_c, int k) __attribute__((always_inline)) {
        constexpr int PP = decltype(pp_c)::value;
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
            if (k % NC == 0) sc[PP][k / NC][qt] = f32x16{};
            mma(sc[PP][k / NC][qt], fk[k], qf[qt][k % NC]);
        }
    };

    // Elements of one tile's scores per lane: e -> (half kt, query tile qt, register r)
    constexpr int NE = KT * QT * 16;
    constexpr int NMAX = NQK / 2;  // slots that take the row maximum; the rest take exp2, sum, packing
    constexpr int NEXP = NQK - NMAX;
    static_assert(NMAX >= 1 && NEXP >= 1, "at least one maximum and one exponent slot");

    // iteration j (parity P = j % 2)
    auto step = [&](auto par_c, auto mask_c, int j) __attribute__((always_inline)) {
        constexpr int P = decltype(par_c)::value;
        constexpr int NP = 1 - P;
        constexpr bool MASK = decltype(mask_c)::value;
        using NPc = std::integral_constant<int, NP>;
        wait_vmcnt<0>();
        __syncthreads();  // K_{j+1} and V_j landed; iteration j-1 is done everywhere
        if (j + 2 < nkb) dk.issue(lds + P * TB, rk, (uint32_t)((j + 2) * BN) * kbytes, wave);
        if (j + 1 < nkb) dv.issue(lds + (2 + NP) * TB, rv, (uint32_t)((j + 1) * BN) * vbytes, wave);
        const int k0 = j * BN;
        if constexpr (MASK) {
#pragma unroll
            for (int kt = 0; kt < KT; ++kt)
#pragma unroll
                for (int qt = 0; qt < QT; ++qt) {
                    const int qi = qw0 + 32 * qt + c32;
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int key = k0 + kt * 32 + acc_row(r, g);
                        if (key >= kv_end || (a.mask.causal && key > qi)) sc[P][kt][qt][r] = -INFINITY;
                    }
                }
        }
#pragma unroll
        for (int k = 0; k < LEAD; ++k) read_k(NP, k);
        __builtin_amdgcn_sched_barrier(0);
        // slots 0..NMAX-1: products of S_{j+1} with the row maxima of tile j
        float mx[QT];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) mx[qt] = -INFINITY;
#pragma unroll
        for (int k = 0; k < NMAX; ++k) {
            qk_slot(NPc{}, k);
            if (k + LEAD < NQK) read_k(NP, k + LEAD);
#pragma unroll
            for (int e = k * NE / NMAX; e < (k + 1) * NE / NMAX; ++e) {
                const int qt = (e / 16) % QT, kt = e / (16 * QT);
                mx[qt] = fmaxf(mx[qt], sc[P][kt][qt][e % 16]);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        float nm[QT];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
            const float x = fmaxf(mx[qt], other_half(mx[qt])) * c;
            if (__any(x > m[qt] + kRescaleSlack)) {
                const float m_new = fmaxf(m[qt], x);
                const float alpha = (m_new == -INFINITY) ? 1.f : fast_exp2(m[qt] - m_new);  // 0 when m was -inf
                l[qt] *= alpha;
#pragma unroll
                for (int t = 0; t < ND; ++t) oacc[qt][t] *= alpha;
                m[qt] = m_new;
            }
            nm[qt] = (m[qt] == -INFINITY) ? 0.f : -m[qt];
        }
        __builtin_amdgcn_sched_barrier(0);
        // slots NMAX..NQK-1: the remaining products with exp2, row sums and packing
        float pv[NE];
        Frag<bf16> pf[KT][QT][2];
#pragma unroll
        for (int k = NMAX; k < NQK; ++k) {
            qk_slot(NPc{}, k);
            if (k + LEAD < NQK) read_k(NP, k + LEAD);
#pragma unroll
            for (int e = (k - NMAX) * NE / NEXP; e < (k - NMAX + 1) * NE / NEXP; ++e) {
                const int qt = (e / 16) % QT, kt = e / (16 * QT), r = e % 16;
                const float x = sc[P][kt][qt][r];
                float p = fast_exp2(__builtin_fmaf(x, c, nm[qt]));
                if constexpr (MASK) p = x == -INFINITY ? 0.f : p;
                asm volatile("" : "+v"(p));
                pv[e] = p;
                l[qt] += p;
                if (e % 8 == 7) pack_frag(pf[kt][qt][r / 8], pv + e - 7);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        // O^T += V^T P^T over the tile's keys; chunk (kt, cc) covers keys
        // kt*32 + 16cc + {4g..4g+3, 8+4g..8+4g+3} in accumulator order
#pragma unroll
        for (int n = 0; n < VLEAD; ++n) read_v(P, n);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int n = 0; n < NPV; ++n) {
            const int t = n % ND, cc = (n / ND) % 2, kt = n / (2 * ND);
            Frag<bf16> vf;
            vf.v = bf16x8{vv[2 * n][0], vv[2 * n][1], vv[2 * n][2], vv[2 * n][3],
                          vv[2 * n + 1][0], vv[2 * n + 1][1], vv[2 * n + 1][2], vv[2 * n + 1][3]};
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) mma(oacc[qt][t], vf, pf[kt][qt][cc]);
            if (n + VLEAD < NPV) read_v(P, n + VLEAD);
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    using P0 = std::integral_constant<int, 0>;
    using P1 = std::integral_constant<int, 1>;
    if (nkb > 0) {
        dk.issue(lds, rk, 0u, wave);
        dv.issue(lds + 2 * TB, rv, 0u, wave);
        if (nkb > 1) dk.issue(lds + TB, rk, (uint32_t)BN * kbytes, wave);
        wait_vmcnt<0>();
        __syncthreads();
#pragma unroll
        for (int k = 0; k < NQK; ++k) {
            read_k(0, k);
            qk_slot(P0{}, k);
        }
    }
    // Tiles inside kv_end and (causal) at or below the block's first query need
    // no mask for any wave; rounded down to an even count so the masked loop
    // also starts on parity 0.
    const int n_full = min(nkb, min(kv_end, a.mask.causal ? q0 + 1 : Skv) / BN) & ~1;
    for (int j = 0; j < n_full; j += 2) {
        step(P0{}, std::false_type{}, j);
        step(P1{}, std::false_type{}, j + 1);
    }
    for (int j = n_full; j < nkb; j += 2) {
        step(P0{}, std::true_type{}, j);
        if (j + 1 < nkb) step(P1{}, std::true_type{}, j + 1);
    }

#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        const float lt = l[qt] + other_half(l[qt]);
        const int qi = qw0 + 32 * qt + c32;
        if (qi < S) {
            const float inv = (lt > 0.f) ? 1.f / lt : 0.f;
            bf16* orow = static_cast<bf16*>(a.o) + a.mo.head_base(b, h) + (int64_t)qi * a.mo.ss;
#pragma unroll
            for (int t = 0; t < ND; ++t) {
#pragma unroll
                for (int rr = 0; rr < 4; ++rr) {
                    const int dcol = 32 * t + 8 * rr + 4 * g;
                    store4(orow + dcol, oacc[qt][t][4 * rr] * inv, oacc[qt][t][4 * rr + 1] * inv,
                           oacc[qt][t][4 * rr + 2] * inv, oacc[qt][t][4 * rr + 3] * inv);
                }
            }
            if (g == 0) a.lse[((int64_t)b * a.Hq + h) * S + qi] = (lt > 0.f) ? (m[qt] + __log2f(lt)) * kLn2 : -INFINITY;
        }
    }
}

template <int D, int TILE>
hipError_t launch_tile(const FwdArgs& a, hipStream_t stream) {
    constexpr AttnTile t = kAttnTiles[TILE];
    static_assert(t.pass == kAttnFwd, "a forward tile");
    constexpr int QT = t.per_wave / 32, KT = t.cols / 32, NW = t.waves, OCC = t.occ;
    constexpr int lds = attn_lds_bytes(t, D);
    static_assert(attn_c1(t, D) && attn_c2(t, D), "tiles in the table pass C1 and C2");
    const hipError_t e = ensure_dynamic_lds<&attn_fwd_bf16<D, QT, KT, NW, OCC>>(lds);
    if (e != hipSuccess) return e;
    constexpr int BM = 32 * QT * NW;
    const int nqb = (a.S + BM - 1) / BM;
    hipLaunchKernelGGL((attn_fwd_bf16<D, QT, KT, NW, OCC>), dim3(rank_major_grid(nqb, a.Hq * a.B)), dim3(64 * NW),
                       lds, stream, a);
    return hipGetLastError();
}

}  // namespace

template <int D>
hipError_t launch_attn_fwd_bf16(const FwdArgs& a, int tile, hipStream_t stream) {
    switch (tile) {
        case 0: return launch_tile<D, 0>(a, stream);
        case 1: return launch_tile<D, 1>(a, stream);
        case 2: return launch_tile<D, 2>(a, stream);
        case 3: return launch_tile<D, 3>(a, stream);
        case 4: return launch_tile<D, 4>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

template hipError_t launch_attn_fwd_bf16<32>(const FwdArgs&, int, hipStream_t);
template hipError_t launch_attn_fwd_bf16<64>(const FwdArgs&, int, hipStream_t);
template hipError_t launch_attn_fwd_bf16<128>(const FwdArgs&, int, hipStream_t);

}  // namespace fbl
