// attn_fwd.hip -- attention forward for fp32 storage on token-major Q/K/V,
// gfx950.  (bf16 storage: attn_fwd_bf16.hip, templated on its tile.)
//
// One workgroup = 4 wavefronts = 128 queries of one (batch, query head); each
// wavefront owns 32 queries.  Key/value tiles of 64 rows (the R-Tile, paper
// section 4.2) stream from the token-major tensors into LDS: row r of a tile
// is token (k0 + r) of head hk, read at base + b*sb + (k0+r)*ss + hk*sh, so
// the head split and transpose of the multi-head attention chain (section
// 4.3.1) are a change of base address, never a copy.  Tiles are double
// buffered and filled by LDS DMA, so tile j+1 is in flight while tile j is
// consumed; one barrier per tile.
//
// The products are arranged so that no operand needs a physical transpose
// (the tile invariance of section 4.2: one staged tile serves both reduction
// directions):
//   S^T = K Q^T     A = K rows (LDS row reads), B = Q rows (registers); the
//                   accumulator holds one query per lane column, so the
//                   softmax row max/sum over keys is an in-lane reduction
//                   plus one exchange between the two 32-lane halves;
//   O^T += V^T P^T  A = V^T from LDS column reads, B = P^T straight from the
//                   S^T accumulator registers.
// fp32 MFMAs (v_mfma_f32_32x32x2_f32, eight per 16-deep chunk).  Online
// softmax in base 2 with scale*log2(e) folded into one FMA per score; the
// running maximum is raised only when a tile exceeds it by more than 2^8 (a
// stale maximum leaves every probability <= 256 and cancels in O/l).  The
// saved LSE is converted to natural log at the store.
#include <type_traits>

#include "cdna4.hpp"
#include "kernels.hpp"
#include "stage.hpp"
#include "tokmap.hpp"

namespace fbl {

namespace {

constexpr int kFwdWaves = 4;
constexpr int kFwdBM = 32 * kFwdWaves;  // queries per workgroup
constexpr int kFwdBN = 64;              // keys per tile
constexpr float kRescaleSlack = 8.0f;   // log2 of the largest unnormalised probability

template <int D>
__global__ __launch_bounds__(256, 1) void attn_fwd_f32(FwdArgs a) {
    using T = float;
    constexpr int NC = D / 16;  // k-chunks over the head dim
    constexpr int ND = D / 32;  // 32-wide output column blocks
    constexpr int TILE = kFwdBN * D;
    constexpr uint32_t TB = TILE * sizeof(T);  // tile bytes
    extern __shared__ __attribute__((aligned(1024))) unsigned char fwd_smem[];
    T* smem = reinterpret_cast<T*>(fwd_smem);  // K0 K1 V0 V1, TILE elements each
    const uint32_t lds = lds_addr(fwd_smem);  // LDS byte address of the tiles

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = lane >> 5;
    const int c32 = lane & 31;
    const int S = a.S;
    const int nqb = (S + kFwdBM - 1) / kFwdBM;
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
    const int q0 = qb * kFwdBM;
    const int qw0 = q0 + wave * 32;  // first query of this wave
    const int qi = qw0 + c32;        // this lane's query (column of S^T)
    int k_hi = kv_end;
    if (a.mask.causal) k_hi = min(k_hi, q0 + kFwdBM);
    const int nkb = (k_hi + kFwdBN - 1) / kFwdBN;

    // the softmax FMA below needs a non-negative scale: fold the sign into Q
    const bool neg = a.scale_log2 < 0.f;
    const float c = neg ? -a.scale_log2 : a.scale_log2;

    // Q^T as the B operand: lane <-> query, in-lane d = 16c + 8g + e
    Frag<T> qf[NC];
    {
        const T* qrow = static_cast<const T*>(a.q) + a.mq.head_base(b, h) + (int64_t)qi * a.mq.ss;
#pragma unroll
        for (int cc = 0; cc < NC; ++cc) {
            float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
            if (qi < S) {
                const f32x4 x0 = __builtin_bit_cast(f32x4, load16(qrow + 16 * cc + 8 * g));
                const f32x4 x1 = __builtin_bit_cast(f32x4, load16(qrow + 16 * cc + 8 * g + 4));
#pragma unroll
                for (int e = 0; e < 4; ++e) { z[e] = neg ? -x0[e] : x0[e]; z[4 + e] = neg ? -x1[e] : x1[e]; }
            }
            pack_frag(qf[cc], z);
        }
    }

    f32x16 oacc[ND];
#pragma unroll
    for (int t = 0; t < ND; ++t) oacc[t] = f32x16{};
    float m = -INFINITY;  // running maximum (log2 units), equal in both lane halves
    float l = 0.f;        // this lane half's share of the running sum

    const uint32_t es = sizeof(T);
    const Rsrc rk = make_rsrc(static_cast<const T*>(a.k) + a.mk.head_base(b, hk),
                              (uint32_t)((int64_t)(Skv - 1) * a.mk.ss * es + D * es));
    const Rsrc rv = make_rsrc(static_cast<const T*>(a.v) + a.mv.head_base(b, hk),
                              (uint32_t)((int64_t)(Skv - 1) * a.mv.ss * es + D * es));
    const uint32_t kbytes = (uint32_t)(a.mk.ss * es), vbytes = (uint32_t)(a.mv.ss * es);
    DmaPlan<T, D, kFwdBN, kFwdWaves> dk, dv;
    dk.init(kbytes, wave, lane);
    dv.init(vbytes, wave, lane);

    // Software pipeline over key tiles j: while the softmax of tile j runs on
    // the vector ALUs, the scores of tile j+1 are already in the matrix
    // cores.  K tiles are fetched two ahead, V tiles one ahead:
    //   iteration j: wait for K_{j+1}, V_j; barrier; DMA K_{j+2} -> Kbuf[j%2],
    //                V_{j+1} -> Vbuf[(j+1)%2]; S_{j+1} = Q K_{j+1}^T;
    //                P_j = softmax(S_j); O += P_j V_j.
    // The loop runs in pairs so buffer and score-array parities are
    // compile-time.
    f32x16 sc[2][2];  // scores of two tiles: [parity][32-key half]

    auto qk = [&](auto par_c, int kbuf) {
        constexpr int P = decltype(par_c)::value;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            sc[P][kt] = f32x16{};
#pragma unroll
            for (int cc = 0; cc < NC; ++cc) {
                Frag<T> kf;
                tile_row_frag<D>(kf, smem + kbuf * TILE, kt * 32 + c32, 16 * cc + 8 * g);
                mma(sc[P][kt], kf, qf[cc]);
            }
        }
    };

    // softmax of the tile in sc[P] (keys k0..k0+63) and O += P V from V buffer P
    auto softmax_pv = [&](auto par_c, auto mask_c, int k0) {
        constexpr int P = decltype(par_c)::value;
        constexpr bool MASK = decltype(mask_c)::value;
        f32x16* s = sc[P];
        if constexpr (MASK) {
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = k0 + kt * 32 + acc_row(r, g);
                    if (key >= kv_end || (a.mask.causal && key > qi)) s[kt][r] = -INFINITY;
                }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kt][r]);
        mx = fmaxf(mx, other_half(mx)) * c;
        if (__any(mx > m + kRescaleSlack)) {
            const float m_new = fmaxf(m, mx);
            const float alpha = (m_new == -INFINITY) ? 1.f : fast_exp2(m - m_new);  // 0 when m was -inf
            l *= alpha;
#pragma unroll
            for (int t = 0; t < ND; ++t) oacc[t] *= alpha;
            m = m_new;
        }
        const float nm = (m == -INFINITY) ? 0.f : -m;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float p = fast_exp2(__builtin_fmaf(s[kt][r], c, nm));
                if constexpr (MASK) {
                    if (s[kt][r] == -INFINITY) p = 0.f;
                }
                s[kt][r] = p;
                l += p;
            }
        // O^T += V^T P^T over the 64 keys: chunk (kt, cc) covers keys
        // kt*32 + 16cc + {4g..4g+3, 8+4g..8+4g+3} in accumulator order
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int cc = 0; cc < 2; ++cc) {
                Frag<T> pf;
                float pv[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) pv[e] = s[kt][8 * cc + e];
                pack_frag(pf, pv);
#pragma unroll
                for (int t = 0; t < ND; ++t) {
                    Frag<T> vf;
                    const int row0 = kt * 32 + 16 * cc + 4 * g;
                    tile_tr_frag<D>(vf, smem + (2 + P) * TILE, row0, row0 + 8, 32 * t, lane);
                    mma(oacc[t], vf, pf);
                }
            }
    };

    // iteration j (parity P = j % 2)
    auto step = [&](auto par_c, auto mask_c, int j) {
        constexpr int P = decltype(par_c)::value;
        constexpr int NP = 1 - P;
        wait_vmcnt<0>();
        __syncthreads();  // K_{j+1} and V_j landed; iteration j-1 is done everywhere
        if (j + 2 < nkb) dk.issue(lds + P * TB, rk, (uint32_t)((j + 2) * kFwdBN) * kbytes, wave);
        if (j + 1 < nkb) {
            dv.issue(lds + (2 + NP) * TB, rv, (uint32_t)((j + 1) * kFwdBN) * vbytes, wave);
            qk(std::integral_constant<int, NP>{}, NP);
        }
        softmax_pv(par_c, mask_c, j * kFwdBN);
    };

    if (nkb > 0) {
        dk.issue(lds, rk, 0u, wave);
        dv.issue(lds + 2 * TB, rv, 0u, wave);
        if (nkb > 1) dk.issue(lds + TB, rk, (uint32_t)kFwdBN * kbytes, wave);
        wait_vmcnt<0>();
        __syncthreads();
        qk(std::integral_constant<int, 0>{}, 0);
    }
    // Tiles inside kv_end and (causal) at or below the block's first query need
    // no mask for any wave; rounded down to an even count so the masked loop
    // also starts on parity 0.
    const int n_full = min(nkb, min(kv_end, a.mask.causal ? q0 + 1 : Skv) / kFwdBN) & ~1;
    using P0 = std::integral_constant<int, 0>;
    using P1 = std::integral_constant<int, 1>;
    for (int j = 0; j < n_full; j += 2) {
        step(P0{}, std::false_type{}, j);
        step(P1{}, std::false_type{}, j + 1);
    }
    for (int j = n_full; j < nkb; j += 2) {
        step(P0{}, std::true_type{}, j);
        if (j + 1 < nkb) step(P1{}, std::true_type{}, j + 1);
    }

    l += other_half(l);
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

template <int D>
constexpr int fwd_lds_bytes() {
    return 4 * kFwdBN * D * (int)sizeof(float);
}

}  // namespace

template <int D>
hipError_t launch_attn_fwd_f32(const FwdArgs& a, hipStream_t stream) {
    const hipError_t e = ensure_dynamic_lds<&attn_fwd_f32<D>>(fwd_lds_bytes<D>());
    if (e != hipSuccess) return e;
    const int nqb = (a.S + kFwdBM - 1) / kFwdBM;
    hipLaunchKernelGGL((attn_fwd_f32<D>), dim3(rank_major_grid(nqb, a.Hq * a.B)), dim3(256), fwd_lds_bytes<D>(),
                       stream, a);
    return hipGetLastError();
}

template hipError_t launch_attn_fwd_f32<32>(const FwdArgs&, hipStream_t);
template hipError_t launch_attn_fwd_f32<64>(const FwdArgs&, hipStream_t);
template hipError_t launch_attn_fwd_f32<128>(const FwdArgs&, hipStream_t);

}  // namespace fbl
