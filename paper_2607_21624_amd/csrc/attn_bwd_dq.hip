// attn_bwd_dq.hip -- dQ from the stored dS, bf16 storage, gfx950.
//
// dQ = scale dS K (section 4.1, the reduction over keys: the N direction of
// section 4.2) as a plain contraction: the key/value-major pass has already
// produced every block of dS (bf16, the values its own dK product used) and
// stored it in the workspace, so this pass only streams dS and K:
//   dQ^T(32 queries) += K_kb^T dS_kb^T       for the key blocks kb of the row
// It is bound by HBM (2 bytes of dS per allowed pair against 2*d MFMA flops),
// so the design goal is a full memory pipe, not MFMA issue: a workgroup of
// NW wavefronts covers blocks of 32*NW queries of one (batch, query head), one
// 32-query tile per wavefront; per 32-key step it brings the K tile (shared)
// and each wavefront's dS block into LDS by DMA, with NBUF - 1 steps in
// flight.  Under a causal mask block q reads NW(q+1) key blocks, so a
// workgroup takes the pair (nqb-1-r, r): every workgroup streams the same
// number of steps.
//
// dS block layout (written by the key/value-major pass): block (qb32, kb32)
// of query head h is 1024 bf16 at ((b*Hq + h)*nk32 + kb32)*nq32*1024 +
// qb32*1024 -- key-block major, so the blocks one step reads (consecutive
// query tiles at one key block) are contiguous; element cc*512 + l*8 + e
// holds dS[query acc_row(8cc + e, l/32)]
// [key l % 32] -- keys across lanes, queries inside a lane.  The dQ product
// contracts over keys, so both operands come from transposed LDS reads
// (ds_read_b64_tr_b16): A = K^T (lane <-> d) from the staged K tile, and
// B = dS^T (lane <-> query) from the staged block, with the per-lane read
// addresses arranged so that fragment element e of lane group g is key
// 8*(e/4) + 4g + e%4 of a 16-key chunk on both sides.  Keys at or past kv_end
// in the last key block are masked here (the key/value pass stores them
// unmasked, and they may be non-finite).
#include <type_traits>

#include "attn_tiles.hpp"
#include "cdna4.hpp"
#include "kernels.hpp"
#include "stage.hpp"
#include "tokmap.hpp"

namespace fbl {

namespace {

constexpr int kDqTiles = 1;  // 32-query tiles per wavefront

// NW wavefronts, NBUF LDS buffers (NBUF - 1 steps in flight)
template <int D, int NW, int NBUF_>
struct DqPipe {
    static constexpr int NBUF = NBUF_;
    static constexpr int ROWS = 32 * kDqTiles * NW;       // queries per block
    static constexpr int TPB = ROWS / 32;                 // 32-query tiles per block
    static constexpr int KT = 32 * D * 2;                 // bytes of a 32-key K tile
    static constexpr int KINST = KT / 1024;               // 1 KB DMA loads per K tile
    static constexpr int KPW = KINST >= NW ? KINST / NW : 1;  // per wavefront
    static constexpr int DSW = kDqTiles * 2048;           // one wavefront's dS blocks per step
    static constexpr int DSBUF = NW * DSW;
    static constexpr int OFF_K = NBUF * DSBUF;
    static constexpr int SPARE = OFF_K + NBUF * KT;       // sink of the K loads of idle wavefronts
    static constexpr int BYTES = SPARE + (KINST < NW ? 1024 : 0);
    static constexpr int LOADS = 2 * kDqTiles + KPW;      // DMA loads per wavefront per step
    static constexpr int OCC = 2 * BYTES <= 160 * 1024 && NW == 4 ? 2 : 1;  // workgroups per CU
    static_assert(KINST % NW == 0 || KINST < NW, "K tile loads spread evenly");
    static_assert(NBUF >= 3 && NBUF <= 6 && (NBUF - 1) * LOADS < 64, "pipeline depth, vmcnt range");
    // dS buffers are read from two bases (buffers 0-2 and 3-5), K from one
    static_assert(2 * DSBUF + (kDqTiles - 1) * 2048 + 384 < 65536 && (NBUF - 1) * KT + KT < 65536,
                  "buffer offsets fit the 16-bit LDS immediate");
    static_assert(BYTES <= 160 * 1024, "LDS of one workgroup");
};

template <int D, int NW, int NBUF>
__global__ __launch_bounds__(64 * NW, (DqPipe<D, NW, NBUF>::OCC)) void attn_bwd_dq_bf16(BwdArgs a) {
    using P = DqPipe<D, NW, NBUF>;
    constexpr int kDqWaves = NW;
    constexpr int kDqRows = P::ROWS;
    constexpr int kDqTilesPerBlock = P::TPB;
    using u32x4 = uint32_t __attribute__((ext_vector_type(4)));
    constexpr int ND = D / 32;
    constexpr int NT = kDqTiles;
    extern __shared__ __attribute__((aligned(1024))) unsigned char dqs_smem[];
    const uint32_t lds = lds_addr(dqs_smem);

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = lane >> 5;
    const int c32 = lane & 31;
    const int S = a.S, Skv = a.Skv;  // query tokens, key tokens
    const int nq32 = a.nq32;
    const bool causal = a.mask.causal != 0;
    const int nqb = (S + kDqRows - 1) / kDqRows;
    const int per_bh = causal ? (nqb + 1) / 2 : nqb;  // workgroups per (batch, query head)
    const int logical = xcd_logical_id(blockIdx.x, per_bh * a.Hq * a.B, gridDim.x);
    if (logical < 0) return;
    const int r = logical % per_bh;
    const int h = (logical / per_bh) % a.Hq;
    const int b = logical / (per_bh * a.Hq);
    const int hk = h / (a.Hq / a.Hkv);
    int kv_end = Skv;
    if (a.mask.kv_len) kv_end = min(max(a.mask.kv_len[b], 0), Skv);
    const int nkv = (kv_end + 31) / 32;  // key blocks holding an allowed key
    // Query blocks of this workgroup and the key blocks each reads.
    const int qa = causal ? nqb - 1 - r : r;
    const int qz = causal && r != qa ? r : -1;
    auto n_kb = [&](int qb) __attribute__((always_inline)) { return causal ? min(nkv, (qb + 1) * kDqTilesPerBlock) : nkv; };
    const int n_a = n_kb(qa);
    const int n = n_a + (qz >= 0 ? n_kb(qz) : 0);
    // step s -> (first 32-query tile of this wavefront, key block)
    auto tile0_of = [&](int s) __attribute__((always_inline)) { return (s < n_a ? qa : qz) * kDqTilesPerBlock + wave * NT; };
    auto kb_of = [&](int s) __attribute__((always_inline)) { return s < n_a ? s : s - n_a; };
    auto tile_ok = [&](int tile, int kb) __attribute__((always_inline)) { return tile < nq32 && (!causal || kb <= tile); };

    // ---- DMA.  K rows past S and dS blocks outside the head's range read as
    // zeros; blocks above the causal diagonal are not fetched (their loads
    // point past the range) and not used.
    const uint32_t kbytes = (uint32_t)(a.mk.ss * 2);
    const bool k_loader = wave < P::KINST;
    const Rsrc rk = make_rsrc(static_cast<const bf16*>(a.k) + a.mk.head_base(b, hk),
                              k_loader ? (uint32_t)((int64_t)(Skv - 1) * a.mk.ss * 2 + D * 2) : 0u);
    DmaPlan<bf16, D, 32, kDqWaves> pk;
    pk.init(kbytes, wave, lane);
    const uint32_t ds_head_elems = (uint32_t)nq32 * (uint32_t)a.nk32 * 1024u;
    const Rsrc rds = make_rsrc(static_cast<const bf16*>(a.ds) + ((int64_t)b * a.Hq + h) * ds_head_elems,
                               ds_head_elems * 2u);
    constexpr uint32_t kNoRecord = 0x80000000u;  // past every head's dS range (< 2 GiB)
    // (resources and scalar offsets pass through readfirstlane: the DMA takes
    // them as SGPR operands, and the compiler cannot always prove them uniform)
    auto uniform = [](Rsrc x) __attribute__((always_inline)) {
        return Rsrc{__builtin_amdgcn_readfirstlane(x[0]), __builtin_amdgcn_readfirstlane(x[1]),
                    __builtin_amdgcn_readfirstlane(x[2]), __builtin_amdgcn_readfirstlane(x[3])};
    };
    auto issue = [&](int s, int buf) __attribute__((always_inline)) {
        const int tile0 = tile0_of(s), kb = kb_of(s);
        const Rsrc rk_s = uniform(rk), rds_s = uniform(rds);
        const uint32_t kl = k_loader ? lds + P::OFF_K + buf * P::KT : lds + P::SPARE;
#pragma unroll
        for (int j = 0; j < P::KPW; ++j)
            dma16(rk_s, kl + (uint32_t)((j * kDqWaves + wave) % P::KINST) * 1024u * (k_loader ? 1u : 0u),
                  pk.voff[j], __builtin_amdgcn_readfirstlane((uint32_t)(kb * 32) * kbytes));
#pragma unroll
        for (int qt = 0; qt < NT; ++qt) {
            const uint32_t soff =
                tile_ok(tile0 + qt, kb) ? ((uint32_t)kb * (uint32_t)nq32 + (uint32_t)(tile0 + qt)) * 2048u : kNoRecord;
            const uint32_t dl = lds + buf * P::DSBUF + wave * P::DSW + qt * 2048;
            dma16_stream(rds_s, dl, (uint32_t)lane * 16u, __builtin_amdgcn_readfirstlane(soff));
            dma16_stream(rds_s, dl + 1024, (uint32_t)lane * 16u + 1024u, __builtin_amdgcn_readfirstlane(soff));
        }
    };

    // ---- per-lane LDS read addresses of buffer 0
    LaneOffsets<D> lo;  // tr[t][h]: K^T fragment, column (d) 32t + lane % 32, keys 8h + 4g + [0..3]
    lo.init(lds + P::OFF_K, lane);
    // dS^T fragment: lane <-> query lane % 32, keys 8h + 4g + [0..3] of a
    // 16-key chunk; source lane s = 4j + m of its 16-lane group fetches the
    // four queries 16*(grp&1) + 4m + [0..3] at key 4*(grp>>1) + j.
    uint32_t ds_lane[2];  // buffers 0-2, buffers 3-5
    {
        const int grp = lane >> 4, s = lane & 15, j = s >> 2, m = s & 3;
        ds_lane[0] = lds + wave * P::DSW + (grp & 1) * 1024 + (32 * (m & 1) + 4 * (grp >> 1) + j) * 16 + (m >> 1) * 8;
        ds_lane[1] = ds_lane[0] + 3 * P::DSBUF;
    }
    // Mask of the last key block when kv_end is not a multiple of 32: fragment
    // element e of chunk kc is key 16kc + 8(e/4) + 4g + e%4 of the block.
    const int kb_tail = kv_end % 32 ? nkv - 1 : -1;
    u32x4 tail_mask[2];
#pragma unroll
    for (int kc = 0; kc < 2; ++kc)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int e0 = 2 * u, e1 = 2 * u + 1;
            const int k0 = 16 * kc + 8 * (e0 / 4) + 4 * g + e0 % 4, k1 = 16 * kc + 8 * (e1 / 4) + 4 * g + e1 % 4;
            const int rem = kv_end % 32;
            tail_mask[kc][u] = (k0 < rem ? 0x0000ffffu : 0u) | (k1 < rem ? 0xffff0000u : 0u);
        }

    // dQ^T accumulators: rows = d (32t + acc_row), columns = queries (lane)
    f32x16 acc[NT][ND];
    auto reset = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int qt = 0; qt < NT; ++qt)
#pragma unroll
            for (int t = 0; t < ND; ++t) acc[qt][t] = f32x16{};
    };
    reset();
    auto store_block = [&](int tile0) __attribute__((always_inline)) {
#pragma unroll
        for (int qt = 0; qt < NT; ++qt) {
            const int qi = (tile0 + qt) * 32 + c32;
            if (qi < S) {
                bf16* dqrow = static_cast<bf16*>(a.dq) + a.mdq.head_base(b, h) + (int64_t)qi * a.mdq.ss;
#pragma unroll
                for (int t = 0; t < ND; ++t)
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr) {
                        const int dcol = 32 * t + 8 * rr + 4 * g;
                        store4(dqrow + dcol, acc[qt][t][4 * rr] * a.scale, acc[qt][t][4 * rr + 1] * a.scale,
                               acc[qt][t][4 * rr + 2] * a.scale, acc[qt][t][4 * rr + 3] * a.scale);
                    }
            }
        }
    };

    auto compute = [&](auto buf_c, int s) __attribute__((always_inline)) {
        constexpr int B = decltype(buf_c)::value;
        const int tile0 = tile0_of(s), kb = kb_of(s);
        Frag<bf16> kt[2][ND];
#pragma unroll
        for (int kc = 0; kc < 2; ++kc)
#pragma unroll
            for (int t = 0; t < ND; ++t) {
                const uint32_t off = B * P::KT + kc * 16 * D * 2;
                const bf16x4 x = lds_tr(lo.tr[t][0], off), y = lds_tr(lo.tr[t][1], off);
                kt[kc][t].v = bf16x8{x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
            }
        const bool tail = kb == kb_tail;
#pragma unroll
        for (int qt = 0; qt < NT; ++qt) {
            if (!tile_ok(tile0 + qt, kb)) continue;
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const uint32_t off = (B % 3) * P::DSBUF + qt * 2048 + kc * 256;
                const bf16x4 x = lds_tr(ds_lane[B / 3], off), y = lds_tr(ds_lane[B / 3], off + 128);
                Frag<bf16> f;
                f.v = bf16x8{x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
                if (tail) f.v = __builtin_bit_cast(bf16x8, __builtin_bit_cast(u32x4, f.v) & tail_mask[kc]);
#pragma unroll
                for (int t = 0; t < ND; ++t) mma(acc[qt][t], kt[kc][t], f);
            }
        }
        if (s == n_a - 1 || s == n - 1) {  // last key block of a query block
            store_block(tile0);
            reset();
        }
    };
    // One step s, held in buffer B: its loads landed in every wavefront (the
    // NBUF - 2 later steps may still be in flight), then the buffer of step
    // s-1 takes step s + NBUF - 1.
    auto step = [&](auto buf_c, int s) __attribute__((always_inline)) {
        constexpr int B = decltype(buf_c)::value;
        const int later = min(NBUF - 2, n - 1 - s);  // steps issued after step s
        if (later >= 4) wait_vmcnt<(NBUF >= 6 ? 4 : 0) * P::LOADS>();
        else if (later == 3) wait_vmcnt<(NBUF >= 5 ? 3 : 0) * P::LOADS>();
        else if (later == 2) wait_vmcnt<2 * P::LOADS>();
        else if (later == 1) wait_vmcnt<P::LOADS>();
        else wait_vmcnt<0>();
        __syncthreads();
        if (s + NBUF - 1 < n) issue(s + NBUF - 1, (B + NBUF - 1) % NBUF);
        compute(buf_c, s);
    };

    for (int s = 0; s < NBUF - 1 && s < n; ++s) issue(s, s);
    // steps in order, NBUF per trip (one per LDS buffer, so every LDS address
    // is a per-lane base plus an immediate)
    for (int s = 0; s < n; s += NBUF)
        unroll_steps(std::make_integer_sequence<int, NBUF>{}, [&](auto buf_c) __attribute__((always_inline)) {
            if (s + decltype(buf_c)::value < n) step(buf_c, s + decltype(buf_c)::value);
        });
    if (n == 0) {  // no allowed key at all: dQ = 0
        store_block(qa * kDqTilesPerBlock + wave * NT);
        if (qz >= 0) store_block(qz * kDqTilesPerBlock + wave * NT);
    }
}

template <int D, int NW, int NBUF>
hipError_t launch_dq(const BwdArgs& a, hipStream_t stream) {
    using P = DqPipe<D, NW, NBUF>;
    const hipError_t once = ensure_dynamic_lds<&attn_bwd_dq_bf16<D, NW, NBUF>>(P::BYTES);
    if (once != hipSuccess) return once;
    const int nqb = (a.S + P::ROWS - 1) / P::ROWS;
    const int n = (a.mask.causal ? (nqb + 1) / 2 : nqb) * a.Hq * a.B;
    hipLaunchKernelGGL((attn_bwd_dq_bf16<D, NW, NBUF>), dim3((n + 7) / 8 * 8), dim3(64 * NW), P::BYTES, stream, a);
    return hipGetLastError();
}

template <int D, int TILE>
hipError_t launch_dq_tile(const BwdArgs& a, hipStream_t stream) {
    constexpr AttnTile t = kAttnTiles[TILE];
    static_assert(t.pass == kAttnDq && t.per_wave == 32 * kDqTiles && t.cols == 32, "a dQ-pass tile");
    using P = DqPipe<D, t.waves, t.bufs>;
    static_assert(P::BYTES == attn_lds_bytes(t, D) && P::OCC == attn_occ(t, D),
                  "the kernel's LDS layout and occupancy are the tile table's");
    return launch_dq<D, t.waves, t.bufs>(a, stream);
}

}  // namespace

template <int D>
hipError_t launch_attn_bwd_dq_bf16(const BwdArgs& a, int tile, hipStream_t stream) {
    switch (tile) {
        case 7: return launch_dq_tile<D, 7>(a, stream);
        case 8: return launch_dq_tile<D, 8>(a, stream);
        case 9: return launch_dq_tile<D, 9>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

template hipError_t launch_attn_bwd_dq_bf16<32>(const BwdArgs&, int, hipStream_t);
template hipError_t launch_attn_bwd_dq_bf16<64>(const BwdArgs&, int, hipStream_t);
template hipError_t launch_attn_bwd_dq_bf16<128>(const BwdArgs&, int, hipStream_t);

}  // namespace fbl
