// api.cpp -- the C ABI: layout descriptors, validation and kernel dispatch.
//
// Every check runs on the host before the first launch; an error return
// means nothing was enqueued.  Mutable global state is limited to the
// per-kernel LDS attribute flags (set once per device, thread-safely) and the
// per-process tables of measured tile choices (mutex-guarded), which only the
// tuning calls write.  The library never allocates, frees or synchronises,
// except that the tuning calls wait for their own timing events.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <map>
#include <mutex>
#include <tuple>
#include <vector>

#include "../../include/fbl.h"
#include "attn_tiles.hpp"
#include "kernels.hpp"

using fbl::bf16;

namespace {

int64_t elem_size(int32_t dt) { return dt == FBL_BF16 ? 2 : (dt == FBL_F32 ? 4 : 0); }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Tile-legality of one descriptor (paper section 4.3.1 checks): intra-tile
// continuity (sd == 1), tile boundary preservation (tile_d divides D), rows
// that hold whole heads, and 16-byte aligned rows.
fbl_status check_layout(const fbl_layout* l) {
    if (!l) return FBL_ERR_NULL;
    const int64_t es = elem_size(l->dtype);
    if (es == 0) return FBL_ERR_DTYPE;
    if (l->B <= 0 || l->S <= 0 || l->H <= 0 || l->D <= 0) return FBL_ERR_SHAPE;
    if (l->B > INT32_MAX || l->S > (1 << 30) || l->H > 65535) return FBL_ERR_SHAPE;
    if (l->sd != 1) return FBL_ERR_LAYOUT;
    if (l->tile_d <= 0 || l->D % l->tile_d != 0 || (l->tile_d * es) % 16 != 0) return FBL_ERR_LAYOUT;
    if (l->sh < l->D) return FBL_ERR_LAYOUT;
    if (l->ss < (l->H - 1) * l->sh + l->D) return FBL_ERR_LAYOUT;
    if (l->B > 1 && l->sb < (l->S - 1) * l->ss + (l->H - 1) * l->sh + l->D) return FBL_ERR_LAYOUT;
    if (l->sb < 0) return FBL_ERR_LAYOUT;
    if ((l->ss * es) % 16 != 0 || (l->sh * es) % 16 != 0 || (l->sb * es) % 16 != 0) return FBL_ERR_ALIGN;
    return FBL_OK;
}

bool same_extents(const fbl_layout* a, const fbl_layout* b) {
    return a->B == b->B && a->S == b->S && a->H == b->H && a->D == b->D && a->dtype == b->dtype;
}

// Bytes spanned by a tensor from its base pointer (last element + 1).
int64_t span_bytes(const fbl_layout* l) {
    const int64_t last = (l->B - 1) * l->sb + (l->S - 1) * l->ss + (l->H - 1) * l->sh + (l->D - 1);
    return (last + 1) * elem_size(l->dtype);
}

// The attention kernels address a tensor from each (batch, head) base with
// 32-bit byte offsets, and their tiles run up to 128 rows past the last token
// (those rows read as zeros and are never stored): every such offset must stay
// below 2^31, the largest range of a buffer resource.
constexpr int64_t kTileRowPad = 128;
bool rows_fit(const fbl_layout* l) {
    return (l->S + kTileRowPad) * l->ss * elem_size(l->dtype) <= ((int64_t)1 << 31);
}

bool overlaps(const void* a, int64_t na, const void* b, int64_t nb) {
    const uintptr_t pa = reinterpret_cast<uintptr_t>(a), pb = reinterpret_cast<uintptr_t>(b);
    return pa < pb + (uintptr_t)nb && pb < pa + (uintptr_t)na;
}

// Whether two described tensors share any byte.  Exact for the common case of
// column views into one packed projection output (same row and batch strides,
// rows of one view falling between the columns of the other); otherwise the
// byte ranges decide (conservative).
bool views_overlap(const void* pa, const fbl_layout* la, const void* pb, const fbl_layout* lb) {
    const int64_t na = span_bytes(la), nb = span_bytes(lb);
    if (!overlaps(pa, na, pb, nb)) return false;
    const int64_t es = elem_size(la->dtype);
    if (es != elem_size(lb->dtype) || la->ss != lb->ss || la->B != lb->B || la->S != lb->S) return true;
    if (la->B > 1 && (la->sb != lb->sb || la->sb % la->ss != 0)) return true;
    const int64_t dbytes = (int64_t)(reinterpret_cast<uintptr_t>(pb) - reinterpret_cast<uintptr_t>(pa));
    if (dbytes % es != 0) return true;
    const int64_t delta = dbytes / es;
    const int64_t wa = (la->H - 1) * la->sh + la->D;  // columns a row of each view covers
    const int64_t wb = (lb->H - 1) * lb->sh + lb->D;
    if (delta >= 0) return !(delta >= wa && delta + wb <= la->ss);
    return !(-delta >= wb && -delta + wa <= la->ss);
}

fbl::TokMap tokmap(const fbl_layout* l) { return fbl::TokMap{l->sb, l->ss, l->sh}; }

fbl::MaskArgs mask_args(const fbl_mask& m) {
    return fbl::MaskArgs{(m.kind & FBL_MASK_CAUSAL) ? 1 : 0,
                         (m.kind & FBL_MASK_KEY_PADDING) ? m.kv_len : nullptr};
}

// Checks shared by forward and backward: q/k/v consistency, mask, scale.
fbl_status check_qkv(const fbl_layout* lq, const void* q, const fbl_layout* lk, const void* k, const fbl_layout* lv,
                     const void* v, float scale, const fbl_mask& mask) {
    if (!lq || !lk || !lv || !q || !k || !v) return FBL_ERR_NULL;
    fbl_status st;
    if ((st = check_layout(lq)) != FBL_OK) return st;
    if ((st = check_layout(lk)) != FBL_OK) return st;
    if ((st = check_layout(lv)) != FBL_OK) return st;
    if (lq->dtype != lk->dtype || lq->dtype != lv->dtype) return FBL_ERR_DTYPE;
    if (lq->B != lk->B || lq->B != lv->B) return FBL_ERR_SHAPE;
    if (!same_extents(lk, lv)) return FBL_ERR_SHAPE;  // K and V: the same S_kv tokens
    if (lq->D != lk->D) return FBL_ERR_SHAPE;
    if (lq->H % lk->H != 0) return FBL_ERR_SHAPE;
    if (lq->D != 32 && lq->D != 64 && lq->D != 128) return FBL_ERR_UNSUPPORTED;
    for (const fbl_layout* l : {lq, lk, lv})
        if (!rows_fit(l)) return FBL_ERR_UNSUPPORTED;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v)) return FBL_ERR_ALIGN;
    if (mask.kind & ~(FBL_MASK_CAUSAL | FBL_MASK_KEY_PADDING)) return FBL_ERR_ARG;
    if ((mask.kind & FBL_MASK_KEY_PADDING) && !mask.kv_len) return FBL_ERR_NULL;
    // cross-attention (S_q != S_kv) takes no causal mask: its alignment is not defined here
    if ((mask.kind & FBL_MASK_CAUSAL) && lq->S != lk->S) return FBL_ERR_UNSUPPORTED;
    if (!std::isfinite(scale)) return FBL_ERR_ARG;
    // launch grids count 32-row blocks of every (batch, head): keep them in range
    for (const fbl_layout* l : {lq, lk})
        if (l->B * l->H * ((l->S + 31) / 32) > INT32_MAX) return FBL_ERR_UNSUPPORTED;
    return FBL_OK;
}

hipError_t dispatch_fwd(int32_t dtype, int D, int tile, const fbl::FwdArgs& a, hipStream_t s) {
    if (dtype == FBL_BF16) {
        switch (D) {
            case 32: return fbl::launch_attn_fwd_bf16<32>(a, tile, s);
            case 64: return fbl::launch_attn_fwd_bf16<64>(a, tile, s);
            default: return fbl::launch_attn_fwd_bf16<128>(a, tile, s);
        }
    }
    switch (D) {
        case 32: return fbl::launch_attn_fwd_f32<32>(a, s);
        case 64: return fbl::launch_attn_fwd_f32<64>(a, s);
        default: return fbl::launch_attn_fwd_f32<128>(a, s);
    }
}

hipError_t dispatch_bwd_fused(int32_t dtype, int D, const fbl::BwdArgs& a, hipStream_t s) {
    if (dtype == FBL_F32) return D == 32 ? fbl::launch_attn_bwd_fused<float, 32>(a, s)
                                         : fbl::launch_attn_bwd_fused<float, 64>(a, s);
    switch (D) {
        case 32: return fbl::launch_attn_bwd_fused<bf16, 32>(a, s);
        case 64: return fbl::launch_attn_bwd_fused<bf16, 64>(a, s);
        default: return fbl::launch_attn_bwd_fused<bf16, 128>(a, s);
    }
}

// Key/value sequences up to this length fit one kv workgroup (four
// wavefronts of 32 keys), and the backward runs as one fused pass (fp32
// storage up to d = 64: at d = 128 its fused state exceeds the registers).
// The fused pass has one workgroup per (batch, kv head), each walking every
// query block of its group; with few such workgroups and long query
// sequences the three-launch path (its key/value pass split over up to four
// workgroups, its dQ pass over query blocks) spreads the work wider, so the
// fused pass is taken only when its grid holds at least 128 workgroups or
// each workgroup has at most 64 query blocks.
constexpr int64_t kFusedBwdMaxKeys = 128;
bool bwd_fuses(const fbl_layout* lq, const fbl_layout* lk) {
    if (lk->S > kFusedBwdMaxKeys || (lq->dtype != FBL_BF16 && lq->D > 64)) return false;
    const int64_t bq = lq->D == 128 ? 32 : 64;  // query rows per block of the fused pass
    const int64_t blocks = lq->H / lk->H * ((lq->S + bq - 1) / bq);
    return lq->B * lk->H >= 128 || blocks <= 64;
}

template <typename T>
hipError_t dispatch_bwd(int D, const fbl::BwdArgs& a, unsigned phases, hipStream_t s) {
    switch (D) {
        case 32: return fbl::launch_attn_bwd<T, 32>(a, phases, s);
        case 64: return fbl::launch_attn_bwd<T, 64>(a, phases, s);
        default: return fbl::launch_attn_bwd<T, 128>(a, phases, s);
    }
}

// ---------------------------------------------------------- attention tiles
// Candidate tiles of one pass at one shape (C1, C2, C3 of attn_tiles.hpp) as
// a bit set over the ids: when no tile keeps the padding within 10%, the
// C1/C2 survivors of least padded volume.
uint64_t attn_candidate_set(uint32_t pass, int64_t D, int64_t Sq, int64_t Skv) {
    static_assert(fbl::kAttnTileCount <= 64, "tile ids fit the bit set");
    uint64_t c12 = 0, all = 0;
    for (int i = 0; i < fbl::kAttnTileCount; ++i) {
        const fbl::AttnTile& t = fbl::kAttnTiles[i];
        if ((uint32_t)t.pass != pass || !fbl::attn_c1(t, (int)D) || !fbl::attn_c2(t, (int)D)) continue;
        c12 |= uint64_t(1) << i;
        if (fbl::attn_c3(t, Sq, Skv)) all |= uint64_t(1) << i;
    }
    if (all || !c12) return all;
    double best = 0;
    for (int i = 0; i < fbl::kAttnTileCount; ++i)
        if (c12 >> i & 1) {
            const double v = fbl::attn_padded_volume(fbl::kAttnTiles[i], Sq, Skv);
            if (!all || v < best) all = uint64_t(1) << i, best = v;
            else if (v == best) all |= uint64_t(1) << i;
        }
    return all;
}

bool attn_tile_legal(uint32_t pass, int32_t tile, int64_t D) {
    if (tile < 0 || tile >= fbl::kAttnTileCount) return false;
    const fbl::AttnTile& t = fbl::kAttnTiles[tile];
    return (uint32_t)t.pass == pass && fbl::attn_c1(t, (int)D) && fbl::attn_c2(t, (int)D);
}

// Per-shape table of measured choices (fbl_attn_tune), keyed by the pass and
// everything that sets its work: storage type, extents, heads, head dim and
// mask kind.
struct AttnKey {
    uint32_t pass;
    int32_t dtype;
    int64_t B, Sq, Skv, Hq, Hkv, D;
    uint32_t mask;
    bool operator<(const AttnKey& o) const {
        return std::tie(pass, dtype, B, Sq, Skv, Hq, Hkv, D, mask) <
               std::tie(o.pass, o.dtype, o.B, o.Sq, o.Skv, o.Hq, o.Hkv, o.D, o.mask);
    }
};
std::mutex g_attn_mu;
std::map<AttnKey, int32_t> g_attn_tuned;

AttnKey attn_key(uint32_t pass, const fbl_layout* lq, const fbl_layout* lk, uint32_t mask_kind) {
    return AttnKey{pass, lq->dtype, lq->B, lq->S, lk->S, lq->H, lk->H, lq->D, mask_kind};
}

// Untuned choice: the first candidate in a preference order per pass, else
// the first legal tile of the pass.  The orders are the measured ones (tuned
// at steady clocks on the Llama-7B-like, Llama-3.2-1B-like GQA, GPT-2-medium-
// like and S = 512 shapes):
//   forward  128 queries in 64-key tiles first, the 64-queries-per-wavefront
//            tiles last (the same at d = 128 and 64);
//   kv pass  at d = 64, the 32-query tiles with two workgroups per CU while
//            the grid has at least 512 key blocks of 128 (two per CU), else
//            the 64-query tiles, which halve the iterations of each of the
//            fewer workgroups (GQA 2048: 120 -> 110 us; S = 512: -7..-25%;
//            GPT-2-like 1024 with 512 blocks: +5%);
//   dQ pass  the 8-wavefront tile (256 queries per workgroup) when it still
//            gives 512 workgroups (Llama-7B-like -2%, GQA 2048 -10%), else
//            the 4-wavefront one (GPT-2-like with 256: +30% for the wide tile).
int32_t attn_default_tile(uint32_t pass, const fbl_layout* lq, const fbl_layout* lk) {
    const int64_t D = lq->D, Sq = lq->S, Skv = lk->S;
    static const int fwd[] = {0, 2, 3, 4, 1};
    static const int kv_many[] = {5, 6, 10}, kv_few[] = {6, 5, 10};
    static const int dq_narrow[] = {7, 8, 9}, dq_wide[] = {8, 7, 9};
    const int* order;
    int n = 3;
    if (pass == FBL_ATTN_FWD) {
        order = fwd, n = 5;
    } else if (pass == FBL_ATTN_BWD_KV) {
        const int64_t blocks = lk->B * lk->H * ((Skv + 127) / 128);
        order = (D == 64 && blocks < 512) ? kv_few : kv_many;
    } else {
        const int64_t wgs = lq->B * lq->H * ((Sq + 255) / 256);
        order = wgs >= 512 ? dq_wide : dq_narrow;
    }
    const uint64_t cand = attn_candidate_set(pass, D, Sq, Skv);
    for (int i = 0; i < n; ++i)
        if (cand >> order[i] & 1) return order[i];
    for (int i = 0; i < n; ++i)
        if (attn_tile_legal(pass, order[i], D)) return order[i];
    return -1;
}

// The tile a launch runs: an explicit id (legal for the pass at this head
// dim), else the measured choice for the shape, else the untuned default.
fbl_status attn_resolve(uint32_t pass, const fbl_layout* lq, const fbl_layout* lk, uint32_t mask_kind,
                        int32_t requested, int32_t* out) {
    if (requested != FBL_ATTN_TILE_AUTO) {
        if (requested < 0 || requested >= fbl::kAttnTileCount || (uint32_t)fbl::kAttnTiles[requested].pass != pass)
            return FBL_ERR_ARG;
        if (!attn_tile_legal(pass, requested, lq->D)) return FBL_ERR_UNSUPPORTED;
        *out = requested;
        return FBL_OK;
    }
    {
        std::lock_guard<std::mutex> lock(g_attn_mu);
        const auto it = g_attn_tuned.find(attn_key(pass, lq, lk, mask_kind));
        if (it != g_attn_tuned.end()) {
            *out = it->second;
            return FBL_OK;
        }
    }
    *out = attn_default_tile(pass, lq, lk);
    return *out >= 0 ? FBL_OK : FBL_ERR_UNSUPPORTED;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Workspace, part 1: the per-query-row statistics, [B, Hq, 2, S] floats (a
// row of LSE * log2(e), then a row of D, for each (batch, query head)).
size_t ws_stats_bytes(const fbl_layout* lq) {
    return align256((size_t)lq->B * lq->H * lq->S * 2 * sizeof(float));
}

// Workspace, part 2 (bf16 only): dS in 32x32-element blocks, [B, Hq, nk32,
// nq32] x 2 KB with nq32 = ceil(S_q / 32), nk32 = ceil(S_kv / 32), so that the
// dQ pass contracts the stored dS with K instead of recomputing S and dP.  0
// when the storage type is fp32 or one head's blocks would reach 2 GiB (the dQ
// pass addresses a head with a 32-bit buffer offset); the backward then
// recomputes.
size_t ws_ds_bytes(const fbl_layout* lq, const fbl_layout* lk) {
    if (lq->dtype != FBL_BF16) return 0;
    const uint64_t per_head = (uint64_t)((lq->S + 31) / 32) * (uint64_t)((lk->S + 31) / 32) * 2048u;
    if (per_head >= (uint64_t(1) << 31)) return 0;
    const uint64_t heads = (uint64_t)lq->B * (uint64_t)lq->H;
    if (heads > (uint64_t(1) << 46) / per_head) return 0;  // keep the total far from overflow
    return (size_t)(heads * per_head);
}

// Split of the key/value pass (bf16 with stored dS).  Its work items are the
// kv tile's key blocks (`rows` keys) per (batch, kv head).  Under a causal
// mask the first key blocks carry the most queries, and with few items (less
// than 512 items of 128 keys: two per CU) the pass waits on those few large
// items while other CUs idle; without a mask the items are equal and only a
// grid of fewer items than half the resident workgroup slots (256 CUs times
// the tile's workgroups per CU) leaves CUs idle.  Sharing each key block's
// query iterations among 2 (or 4) workgroups gives the scheduler items of
// half (a quarter) the size; each writes fp32 partial dK and dV and a
// reduction adds them in a fixed order.  Only where the first key block has
// at least 16 iterations per share.  (Measured with 128-key blocks: splitting
// the 512 items of the GPT-2-medium-like causal shape, or the Llama-3.2-1B-like
// GQA shape four ways, is slower.)
int kv_split_for(const fbl_layout* lq, const fbl_layout* lk, bool causal, int tile) {
    if (lq->dtype != FBL_BF16 || lk->H <= 0 || lq->D <= 0) return 1;
    const fbl::AttnTile& t = fbl::kAttnTiles[tile];
    const int64_t rows = fbl::attn_rows(t);
    const int64_t items = (lk->S + rows - 1) / rows * lk->H * lk->B;
    const int64_t slots = 256 * (int64_t)fbl::attn_occ(t, (int)lq->D);
    const int64_t iters = lq->H / lk->H * ((lq->S + t.cols - 1) / t.cols);
    int split = 1;
    while (split < 4 && (causal ? items * split * rows < 512 * 128 : items * split * 2 <= slots) &&
           iters >= 16 * split)
        split *= 2;
    return split;
}

// Workspace, part 3 (with part 2 only): the split key/value pass's fp32
// partial dK and dV, [2][kv_split][B, S_kv, Hkv, D]; 0 without a split.
// Sized for the largest split any kv tile that runs at this head dim takes,
// with or without a causal mask.
size_t ws_part_bytes(const fbl_layout* lq, const fbl_layout* lk) {
    int split = 1;
    for (int i = 0; i < fbl::kAttnTileCount; ++i)
        if (attn_tile_legal(FBL_ATTN_BWD_KV, i, lq->D))
            split = std::max(split, std::max(kv_split_for(lq, lk, true, i), kv_split_for(lq, lk, false, i)));
    if (split == 1 || ws_ds_bytes(lq, lk) == 0) return 0;
    return align256((size_t)2 * split * lk->B * lk->S * lk->H * lk->D * sizeof(float));
}

size_t ws_bytes_for(const fbl_layout* lq, const fbl_layout* lk) {
    return ws_stats_bytes(lq) + ws_ds_bytes(lq, lk) + ws_part_bytes(lq, lk);
}

}  // namespace

extern "C" {

const char* fbl_status_str(fbl_status s) {
    switch (s) {
        case FBL_OK: return "FBL_OK";
        case FBL_ERR_NULL: return "FBL_ERR_NULL: a required pointer is NULL";
        case FBL_ERR_SHAPE: return "FBL_ERR_SHAPE: non-positive or inconsistent extents";
        case FBL_ERR_DTYPE: return "FBL_ERR_DTYPE: unknown or mismatched dtype";
        case FBL_ERR_LAYOUT: return "FBL_ERR_LAYOUT: tile-legality check failed";
        case FBL_ERR_ALIGN: return "FBL_ERR_ALIGN: pointer or stride not 16-byte aligned";
        case FBL_ERR_UNSUPPORTED: return "FBL_ERR_UNSUPPORTED: shape, head dim or mask not implemented";
        case FBL_ERR_WORKSPACE: return "FBL_ERR_WORKSPACE: workspace missing or too small";
        case FBL_ERR_HIP: return "FBL_ERR_HIP: HIP runtime error at launch";
        case FBL_ERR_ARG: return "FBL_ERR_ARG: invalid argument";
    }
    return "FBL_ERR_UNKNOWN";
}

fbl_status fbl_layout_desc(fbl_layout* out, int32_t dtype, int64_t B, int64_t S, int64_t H, int64_t D,
                           int64_t row_stride, int64_t batch_stride, int64_t tile_d) {
    if (!out) return FBL_ERR_NULL;
    std::memset(out, 0, sizeof(*out));
    if (elem_size(dtype) == 0) return FBL_ERR_DTYPE;
    if (B <= 0 || S <= 0 || H <= 0 || D <= 0 || row_stride < 0 || batch_stride < 0 || tile_d < 0) return FBL_ERR_SHAPE;
    fbl_layout l;
    std::memset(&l, 0, sizeof(l));
    l.dtype = dtype;
    l.B = B;
    l.S = S;
    l.H = H;
    l.D = D;
    l.sd = 1;
    l.sh = D;
    l.ss = row_stride ? row_stride : H * D;
    l.sb = batch_stride ? batch_stride : S * l.ss;
    if (tile_d > INT32_MAX) return FBL_ERR_LAYOUT;
    l.tile_d = (int32_t)(tile_d ? tile_d : D);
    const fbl_status st = check_layout(&l);
    if (st != FBL_OK) return st;
    *out = l;
    return FBL_OK;
}

fbl_status fbl_layout_packed_qkv(fbl_layout* lq, fbl_layout* lk, fbl_layout* lv, int64_t* k_off, int64_t* v_off,
                                 int32_t dtype, int64_t B, int64_t S, int64_t Hq, int64_t Hkv, int64_t D,
                                 int64_t batch_stride, int64_t tile_d) {
    if (!lq || !lk || !lv || !k_off || !v_off) return FBL_ERR_NULL;
    std::memset(lq, 0, sizeof(*lq));
    std::memset(lk, 0, sizeof(*lk));
    std::memset(lv, 0, sizeof(*lv));
    *k_off = 0;
    *v_off = 0;
    if (Hq <= 0 || Hkv <= 0 || D <= 0 || Hq > INT32_MAX || Hkv > INT32_MAX) return FBL_ERR_SHAPE;
    const int64_t row = (Hq + 2 * Hkv) * D;  // one token of the packed projection output
    fbl_layout q, k, v;
    fbl_status st;
    if ((st = fbl_layout_desc(&q, dtype, B, S, Hq, D, row, batch_stride, tile_d)) != FBL_OK) return st;
    if ((st = fbl_layout_desc(&k, dtype, B, S, Hkv, D, row, batch_stride, tile_d)) != FBL_OK) return st;
    if ((st = fbl_layout_desc(&v, dtype, B, S, Hkv, D, row, batch_stride, tile_d)) != FBL_OK) return st;
    *lq = q;
    *lk = k;
    *lv = v;
    *k_off = Hq * D;
    *v_off = (Hq + Hkv) * D;
    return FBL_OK;
}

int64_t fbl_layout_offset(const fbl_layout* l, int64_t b, int64_t h, int64_t s, int64_t i) {
    if (!l) return -1;
    if (b < 0 || b >= l->B || h < 0 || h >= l->H || s < 0 || s >= l->S || i < 0 || i >= l->D) return -1;
    return b * l->sb + s * l->ss + h * l->sh + i * l->sd;
}

fbl_status fbl_layout_map_device(const fbl_layout* l, int64_t* out, void* stream) {
    if (!l || !out) return FBL_ERR_NULL;
    const fbl_status st = check_layout(l);
    if (st != FBL_OK) return st;
    const hipError_t e = fbl::launch_layout_map(tokmap(l), (int)l->B, (int)l->H, (int)l->S, (int)l->D, out,
                                                static_cast<hipStream_t>(stream));
    return e == hipSuccess ? FBL_OK : FBL_ERR_HIP;
}

fbl_status fbl_attn_fwd_tiled(const fbl_layout* lq, const void* q, const fbl_layout* lk, const void* k,
                              const fbl_layout* lv, const void* v, const fbl_layout* lo, void* o, float* lse,
                              float scale, fbl_mask mask, int32_t tile, void* stream) {
    fbl_status st = check_qkv(lq, q, lk, k, lv, v, scale, mask);
    if (st != FBL_OK) return st;
    if (!lo || !o || !lse) return FBL_ERR_NULL;
    if ((st = check_layout(lo)) != FBL_OK) return st;
    if (!same_extents(lo, lq)) return lo->dtype != lq->dtype ? FBL_ERR_DTYPE : FBL_ERR_SHAPE;
    if (!rows_fit(lo)) return FBL_ERR_UNSUPPORTED;
    if (!aligned16(o) || !aligned16(lse)) return FBL_ERR_ALIGN;
    const int64_t lse_bytes = lq->B * lq->H * lq->S * 4;
    const void* ins[3] = {q, k, v};
    const fbl_layout* in_l[3] = {lq, lk, lv};
    for (int i = 0; i < 3; ++i) {
        if (views_overlap(o, lo, ins[i], in_l[i])) return FBL_ERR_ARG;
        if (overlaps(lse, lse_bytes, ins[i], span_bytes(in_l[i]))) return FBL_ERR_ARG;
    }
    if (overlaps(o, span_bytes(lo), lse, lse_bytes)) return FBL_ERR_ARG;
    int32_t t = -1;
    if (lq->dtype == FBL_BF16) {
        if ((st = attn_resolve(FBL_ATTN_FWD, lq, lk, mask.kind, tile, &t)) != FBL_OK) return st;
    } else if (tile != FBL_ATTN_TILE_AUTO) {
        return FBL_ERR_ARG;  // fp32 storage has one configuration
    }

    fbl::FwdArgs a;
    a.q = q;
    a.k = k;
    a.v = v;
    a.o = o;
    a.lse = lse;
    a.mq = tokmap(lq);
    a.mk = tokmap(lk);
    a.mv = tokmap(lv);
    a.mo = tokmap(lo);
    a.B = (int)lq->B;
    a.S = (int)lq->S;
    a.Skv = (int)lk->S;
    a.Hq = (int)lq->H;
    a.Hkv = (int)lk->H;
    a.scale_log2 = scale * 1.4426950408889634f;
    a.mask = mask_args(mask);
    const hipError_t e = dispatch_fwd(lq->dtype, (int)lq->D, t, a, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? FBL_OK : FBL_ERR_HIP;
}

fbl_status fbl_attn_fwd(const fbl_layout* lq, const void* q, const fbl_layout* lk, const void* k,
                        const fbl_layout* lv, const void* v, const fbl_layout* lo, void* o, float* lse, float scale,
                        fbl_mask mask, void* stream) {
    return fbl_attn_fwd_tiled(lq, q, lk, k, lv, v, lo, o, lse, scale, mask, FBL_ATTN_TILE_AUTO, stream);
}

fbl_status fbl_attn_bwd_workspace(const fbl_layout* lq, const fbl_layout* lk, size_t* bytes) {
    if (!lq || !lk || !bytes) return FBL_ERR_NULL;
    fbl_status st;
    if ((st = check_layout(lq)) != FBL_OK) return st;
    if ((st = check_layout(lk)) != FBL_OK) return st;
    *bytes = ws_bytes_for(lq, lk);
    return FBL_OK;
}

fbl_status fbl_attn_bwd_workspace_min(const fbl_layout* lq, const fbl_layout* lk, size_t* bytes) {
    if (!lq || !lk || !bytes) return FBL_ERR_NULL;
    fbl_status st;
    if ((st = check_layout(lq)) != FBL_OK) return st;
    if ((st = check_layout(lk)) != FBL_OK) return st;
    *bytes = ws_stats_bytes(lq);
    return FBL_OK;
}

}  // extern "C"

namespace {

// What a backward call runs, from the shapes, the mask, the workspace size
// and the requested tiles alone (no pointer is read).
struct BwdPlan {
    bool fused = false;      // the one-launch backward
    bool stores_ds = false;  // the kv pass stores dS, the dQ pass reads it
    int kv_split = 1;        // key/value pass split (partial sums + reduction)
    int32_t kv_tile = 5, dq_tile = 7;
};

fbl_status bwd_plan(uint32_t phases, const fbl_layout* lq, const fbl_layout* lk, uint32_t mask_kind,
                    size_t ws_bytes, int32_t kv_tile, int32_t dq_tile, BwdPlan* p) {
    fbl_status st;
    // tiles of the bf16 passes (fp32 storage has one configuration per pass)
    if (lq->dtype == FBL_BF16) {
        if ((st = attn_resolve(FBL_ATTN_BWD_KV, lq, lk, mask_kind, kv_tile, &p->kv_tile)) != FBL_OK) return st;
        if ((st = attn_resolve(FBL_ATTN_BWD_DQ, lq, lk, mask_kind, dq_tile, &p->dq_tile)) != FBL_OK) return st;
    } else if (kv_tile != FBL_ATTN_TILE_AUTO || dq_tile != FBL_ATTN_TILE_AUTO) {
        return FBL_ERR_ARG;
    }
    // the whole backward with automatic tiles, keys within one kv workgroup: one fused launch
    p->fused = phases == FBL_BWD_ALL && bwd_fuses(lq, lk) && kv_tile == FBL_ATTN_TILE_AUTO &&
               dq_tile == FBL_ATTN_TILE_AUTO;
    // stored-dS path when the workspace holds the dS blocks, else recompute
    const size_t ds_bytes = ws_ds_bytes(lq, lk);
    p->stores_ds = ds_bytes && ws_bytes >= ws_stats_bytes(lq) + ds_bytes;
    // and the split key/value pass when it also holds the partial sums
    const size_t part_bytes = ws_part_bytes(lq, lk);
    if (p->stores_ds && part_bytes && ws_bytes >= ws_stats_bytes(lq) + ds_bytes + part_bytes)
        p->kv_split = kv_split_for(lq, lk, (mask_kind & FBL_MASK_CAUSAL) != 0, p->kv_tile);
    return FBL_OK;
}

fbl_status bwd_run(uint32_t phases, const fbl_layout* lq, const void* q, const fbl_layout* lk, const void* k,
                   const fbl_layout* lv, const void* v, const fbl_layout* lo, const void* o, const fbl_layout* ldo,
                   const void* dO, const float* lse, float scale, fbl_mask mask, const fbl_layout* ldq, void* dq,
                   const fbl_layout* ldk, void* dk, const fbl_layout* ldv, void* dv, void* ws, size_t ws_bytes,
                   int32_t kv_tile, int32_t dq_tile, void* stream) {
    if (phases == 0 || (phases & ~FBL_BWD_ALL)) return FBL_ERR_ARG;
    fbl_status st = check_qkv(lq, q, lk, k, lv, v, scale, mask);
    if (st != FBL_OK) return st;
    if (!lo || !o || !ldo || !dO || !lse || !ldq || !dq || !ldk || !dk || !ldv || !dv) return FBL_ERR_NULL;
    const fbl_layout* all[5] = {lo, ldo, ldq, ldk, ldv};
    for (const fbl_layout* l : all)
        if ((st = check_layout(l)) != FBL_OK) return st;
    for (const fbl_layout* l : {lo, ldo, ldq})
        if (!same_extents(l, lq)) return l->dtype != lq->dtype ? FBL_ERR_DTYPE : FBL_ERR_SHAPE;
    for (const fbl_layout* l : {ldk, ldv})
        if (!same_extents(l, lk)) return l->dtype != lq->dtype ? FBL_ERR_DTYPE : FBL_ERR_SHAPE;
    for (const fbl_layout* l : all)
        if (!rows_fit(l)) return FBL_ERR_UNSUPPORTED;
    if (!aligned16(o) || !aligned16(dO) || !aligned16(lse) || !aligned16(dq) || !aligned16(dk) || !aligned16(dv))
        return FBL_ERR_ALIGN;
    if (!ws) return FBL_ERR_WORKSPACE;
    if (ws_bytes < ws_stats_bytes(lq)) return FBL_ERR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0) return FBL_ERR_ALIGN;

    const int64_t lse_bytes = lq->B * lq->H * lq->S * 4;
    const void* ins[5] = {q, k, v, o, dO};
    const fbl_layout* in_l[5] = {lq, lk, lv, lo, ldo};
    void* outs[3] = {dq, dk, dv};
    const fbl_layout* out_l[3] = {ldq, ldk, ldv};
    // the workspace is written (statistics, dS, partial sums) while every
    // input is read: it may share no byte with an input or with lse
    for (int j = 0; j < 5; ++j)
        if (overlaps(ws, (int64_t)ws_bytes, ins[j], span_bytes(in_l[j]))) return FBL_ERR_ARG;
    if (overlaps(ws, (int64_t)ws_bytes, lse, lse_bytes)) return FBL_ERR_ARG;
    for (int i = 0; i < 3; ++i) {
        for (int j = 0; j < 5; ++j)
            if (views_overlap(outs[i], out_l[i], ins[j], in_l[j])) return FBL_ERR_ARG;
        if (overlaps(outs[i], span_bytes(out_l[i]), lse, lse_bytes)) return FBL_ERR_ARG;
        if (overlaps(outs[i], span_bytes(out_l[i]), ws, (int64_t)ws_bytes)) return FBL_ERR_ARG;
        for (int j = i + 1; j < 3; ++j)
            if (views_overlap(outs[i], out_l[i], outs[j], out_l[j])) return FBL_ERR_ARG;
    }

    BwdPlan plan;
    if ((st = bwd_plan(phases, lq, lk, mask.kind, ws_bytes, kv_tile, dq_tile, &plan)) != FBL_OK) return st;
    fbl::BwdArgs a;
    a.q = q;
    a.k = k;
    a.v = v;
    a.o = o;
    a.dout = dO;
    a.lse = lse;
    a.dq = dq;
    a.dk = dk;
    a.dv = dv;
    a.stats = static_cast<float*>(ws);
    a.ds = plan.stores_ds ? static_cast<char*>(ws) + ws_stats_bytes(lq) : nullptr;
    a.kv_tile = plan.kv_tile;
    a.dq_tile = plan.dq_tile;
    a.kv_split = plan.kv_split;
    if (plan.kv_split > 1)
        a.dkv_part = reinterpret_cast<float*>(static_cast<char*>(ws) + ws_stats_bytes(lq) + ws_ds_bytes(lq, lk));
    a.nq32 = (int)((lq->S + 31) / 32);
    a.nk32 = (int)((lk->S + 31) / 32);
    a.mq = tokmap(lq);
    a.mk = tokmap(lk);
    a.mv = tokmap(lv);
    a.mo = tokmap(lo);
    a.mdo = tokmap(ldo);
    a.mdq = tokmap(ldq);
    a.mdk = tokmap(ldk);
    a.mdv = tokmap(ldv);
    a.B = (int)lq->B;
    a.S = (int)lq->S;
    a.Skv = (int)lk->S;
    a.Hq = (int)lq->H;
    a.Hkv = (int)lk->H;
    a.scale = scale;
    a.scale_log2 = scale * 1.4426950408889634f;
    a.mask = mask_args(mask);
    const hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e;
    if (plan.fused)
        e = dispatch_bwd_fused(lq->dtype, (int)lq->D, a, s);
    else
        e = lq->dtype == FBL_BF16 ? dispatch_bwd<bf16>((int)lq->D, a, phases, s)
                                  : dispatch_bwd<float>((int)lq->D, a, phases, s);
    return e == hipSuccess ? FBL_OK : FBL_ERR_HIP;
}

}  // namespace

extern "C" {

fbl_status fbl_attn_bwd_phases(uint32_t phases, const fbl_layout* lq, const void* q, const fbl_layout* lk,
                               const void* k, const fbl_layout* lv, const void* v, const fbl_layout* lo,
                               const void* o, const fbl_layout* ldo, const void* dO, const float* lse, float scale,
                               fbl_mask mask, const fbl_layout* ldq, void* dq, const fbl_layout* ldk, void* dk,
                               const fbl_layout* ldv, void* dv, void* ws, size_t ws_bytes, void* stream) {
    return bwd_run(phases, lq, q, lk, k, lv, v, lo, o, ldo, dO, lse, scale, mask, ldq, dq, ldk, dk, ldv, dv, ws,
                   ws_bytes, FBL_ATTN_TILE_AUTO, FBL_ATTN_TILE_AUTO, stream);
}

fbl_status fbl_attn_bwd(const fbl_layout* lq, const void* q, const fbl_layout* lk, const void* k,
                        const fbl_layout* lv, const void* v, const fbl_layout* lo, const void* o,
                        const fbl_layout* ldo, const void* dO, const float* lse, float scale, fbl_mask mask,
                        const fbl_layout* ldq, void* dq, const fbl_layout* ldk, void* dk, const fbl_layout* ldv,
                        void* dv, void* ws, size_t ws_bytes, void* stream) {
    return bwd_run(FBL_BWD_ALL, lq, q, lk, k, lv, v, lo, o, ldo, dO, lse, scale, mask, ldq, dq, ldk, dk, ldv, dv, ws,
                   ws_bytes, FBL_ATTN_TILE_AUTO, FBL_ATTN_TILE_AUTO, stream);
}

fbl_status fbl_attn_bwd_launches(uint32_t phases, const fbl_layout* lq, const fbl_layout* lk, uint32_t mask_kind,
                                size_t ws_bytes, int32_t kv_tile, int32_t dq_tile, int32_t* launches) {
    if (!launches) return FBL_ERR_NULL;
    if (phases == 0 || (phases & ~FBL_BWD_ALL) || (mask_kind & ~(FBL_MASK_CAUSAL | FBL_MASK_KEY_PADDING)))
        return FBL_ERR_ARG;
    fbl_status st;
    if ((st = check_layout(lq)) != FBL_OK || (st = check_layout(lk)) != FBL_OK) return st;
    if (lq->dtype != lk->dtype) return FBL_ERR_DTYPE;
    if (lq->B != lk->B || lq->D != lk->D || lq->H % lk->H != 0) return FBL_ERR_SHAPE;
    if (lq->D != 32 && lq->D != 64 && lq->D != 128) return FBL_ERR_UNSUPPORTED;
    BwdPlan plan;
    if ((st = bwd_plan(phases, lq, lk, mask_kind, ws_bytes, kv_tile, dq_tile, &plan)) != FBL_OK) return st;
    if (plan.fused) {
        *launches = 1;
        return FBL_OK;
    }
    *launches = (int32_t)__builtin_popcount(phases) + ((phases & FBL_BWD_KV) && plan.kv_split > 1 ? 1 : 0);
    return FBL_OK;
}

fbl_status fbl_attn_bwd_tiled(uint32_t phases, const fbl_layout* lq, const void* q, const fbl_layout* lk,
                              const void* k, const fbl_layout* lv, const void* v, const fbl_layout* lo, const void* o,
                              const fbl_layout* ldo, const void* dO, const float* lse, float scale, fbl_mask mask,
                              const fbl_layout* ldq, void* dq, const fbl_layout* ldk, void* dk, const fbl_layout* ldv,
                              void* dv, void* ws, size_t ws_bytes, int32_t kv_tile, int32_t dq_tile, void* stream) {
    return bwd_run(phases, lq, q, lk, k, lv, v, lo, o, ldo, dO, lse, scale, mask, ldq, dq, ldk, dk, ldv, dv, ws,
                   ws_bytes, kv_tile, dq_tile, stream);
}

int32_t fbl_attn_tile_count(void) { return fbl::kAttnTileCount; }

fbl_status fbl_attn_tile_info(int32_t tile, int64_t D, int32_t* info) {
    if (!info) return FBL_ERR_NULL;
    if (tile < 0 || tile >= fbl::kAttnTileCount) return FBL_ERR_ARG;
    if (D != 32 && D != 64 && D != 128) return FBL_ERR_UNSUPPORTED;
    const fbl::AttnTile& t = fbl::kAttnTiles[tile];
    const int32_t v[8] = {t.pass,
                          fbl::attn_rows(t),
                          t.cols,
                          t.waves,
                          t.per_wave,
                          fbl::attn_occ(t, (int)D),
                          fbl::attn_lds_bytes(t, (int)D),
                          (fbl::attn_c1(t, (int)D) && fbl::attn_c2(t, (int)D)) ? 1 : 0};
    std::memcpy(info, v, sizeof(v));
    return FBL_OK;
}

fbl_status fbl_attn_candidates(uint32_t pass, const fbl_layout* lq, const fbl_layout* lk, int32_t* tiles,
                               int32_t cap, int32_t* count) {
    if (!lq || !lk || !count || (cap > 0 && !tiles)) return FBL_ERR_NULL;
    if (pass > FBL_ATTN_BWD_DQ) return FBL_ERR_ARG;
    fbl_status st;
    if ((st = check_layout(lq)) != FBL_OK) return st;
    if ((st = check_layout(lk)) != FBL_OK) return st;
    if (lq->dtype != FBL_BF16) return FBL_ERR_DTYPE;  // fp32 storage: one configuration per pass
    if (lq->D != 32 && lq->D != 64 && lq->D != 128) return FBL_ERR_UNSUPPORTED;
    const uint64_t cand = attn_candidate_set(pass, lq->D, lq->S, lk->S);
    int32_t n = 0;
    for (int t = 0; t < fbl::kAttnTileCount; ++t)
        if (cand >> t & 1) {
            if (n < cap) tiles[n] = t;
            ++n;
        }
    *count = n;
    return FBL_OK;
}

fbl_status fbl_attn_auto_tiles(const fbl_layout* lq, const fbl_layout* lk, uint32_t mask_kind, int32_t* tiles) {
    if (!lq || !lk || !tiles) return FBL_ERR_NULL;
    fbl_status st;
    if ((st = check_layout(lq)) != FBL_OK) return st;
    if ((st = check_layout(lk)) != FBL_OK) return st;
    if (lq->dtype != FBL_BF16) return FBL_ERR_DTYPE;
    if (lq->D != 32 && lq->D != 64 && lq->D != 128) return FBL_ERR_UNSUPPORTED;
    for (uint32_t pass = 0; pass <= FBL_ATTN_BWD_DQ; ++pass)
        if ((st = attn_resolve(pass, lq, lk, mask_kind, FBL_ATTN_TILE_AUTO, &tiles[pass])) != FBL_OK) return st;
    return FBL_OK;
}

fbl_status fbl_attn_tune(const fbl_layout* lq, const void* q, const fbl_layout* lk, const void* k,
                         const fbl_layout* lv, const void* v, const fbl_layout* lo, void* o, float* lse,
                         const fbl_layout* ldo, const void* dO, float scale, fbl_mask mask, const fbl_layout* ldq,
                         void* dq, const fbl_layout* ldk, void* dk, const fbl_layout* ldv, void* dv, void* ws,
                         size_t ws_bytes, uint32_t objective, int32_t reps, float* ms, int32_t* best, void* stream) {
    if (objective > FBL_TUNE_GFLOPS_X_MEMEFF || reps < 1 || reps > 1000) return FBL_ERR_ARG;
    // every argument check, once, before anything is timed
    fbl_status st = fbl_attn_fwd_tiled(lq, q, lk, k, lv, v, lo, o, lse, scale, mask, FBL_ATTN_TILE_AUTO, stream);
    if (st != FBL_OK) return st;
    if (lq->dtype != FBL_BF16) return FBL_ERR_DTYPE;  // fp32 storage: one configuration per pass
    auto bwd = [&](uint32_t phases, int32_t kv_tile, int32_t dq_tile) {
        return bwd_run(phases, lq, q, lk, k, lv, v, lo, o, ldo, dO, lse, scale, mask, ldq, dq, ldk, dk, ldv, dv, ws,
                       ws_bytes, kv_tile, dq_tile, stream);
    };
    if ((st = bwd(FBL_BWD_ALL, FBL_ATTN_TILE_AUTO, FBL_ATTN_TILE_AUTO)) != FBL_OK) return st;
    if (ms)
        for (int t = 0; t < fbl::kAttnTileCount; ++t) ms[t] = -1.0f;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
        if (e0) hipEventDestroy(e0);
        return FBL_ERR_HIP;
    }
    // average milliseconds of `reps` launches after one untimed launch
    auto timed = [&](auto&& launch, float* out) -> fbl_status {
        fbl_status r = launch();
        if (r != FBL_OK) return r;
        if (hipEventRecord(e0, s) != hipSuccess) return FBL_ERR_HIP;
        for (int i = 0; i < reps; ++i)
            if ((r = launch()) != FBL_OK) return r;
        float total = 0;
        if (hipEventRecord(e1, s) != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
            hipEventElapsedTime(&total, e0, e1) != hipSuccess)
            return FBL_ERR_HIP;
        *out = total / (float)reps;
        return FBL_OK;
    };
    // MemEfficiency of a tile (section 4.2): the pass's minimal bytes over the
    // bytes its tile schedule stages.  Per (batch, query head), the forward
    // stages the K and V rows a query block sees once per block of `rows`
    // queries, the dQ pass the K rows once per block; the kv pass stages the
    // same rows whatever its query tile, so its efficiency is 1.
    const bool causal = (mask.kind & FBL_MASK_CAUSAL) != 0;
    const double D = (double)lq->D, Sq = (double)lq->S, Skv = (double)lk->S;
    const double bh = (double)lq->B * (double)lq->H;
    auto keys_staged = [&](int rows) {  // keys read per (batch, query head) over its query blocks
        double n = 0;
        for (int64_t q0 = 0; q0 < lq->S; q0 += rows) n += causal ? std::min(Skv, (double)(q0 + rows)) : Skv;
        return n;
    };
    auto mem_eff = [&](uint32_t pass, int tile) {
        const int rows = fbl::attn_rows(fbl::kAttnTiles[tile]);
        if (pass == FBL_ATTN_FWD) {
            const double qo = 2.0 * bh * Sq * D * 2 + bh * Sq * 4;  // Q read, O written, LSE written
            const double kv_min = 2.0 * (double)lk->B * (double)lk->H * Skv * D * 2;
            return (qo + kv_min) / (qo + 2.0 * bh * keys_staged(rows) * D * 2);
        }
        if (pass == FBL_ATTN_BWD_DQ) {
            const double ds = 2048.0 * bh * std::ceil(Sq / 32) * std::ceil(Skv / 32) * (causal ? 0.5 : 1.0);
            const double fixed = ds + bh * Sq * D * 2;  // dS read, dQ written
            return (fixed + (double)lk->B * (double)lk->H * Skv * D * 2) / (fixed + bh * keys_staged(rows) * D * 2);
        }
        return 1.0;
    };
    int32_t pick[3] = {-1, -1, -1};
    const bool ds_path = ws_ds_bytes(lq, lk) && ws_bytes >= ws_stats_bytes(lq) + ws_ds_bytes(lq, lk);
    for (uint32_t pass = 0; pass <= FBL_ATTN_BWD_DQ && st == FBL_OK; ++pass) {
        if (pass == FBL_ATTN_BWD_DQ && !ds_path) break;  // the recompute pass has one configuration
        const uint64_t cand = attn_candidate_set(pass, lq->D, lq->S, lk->S);
        double pick_score = 0;
        for (int t = 0; t < fbl::kAttnTileCount && st == FBL_OK; ++t) {
            if (!(cand >> t & 1)) continue;
            float avg = 0;
            if (pass == FBL_ATTN_FWD)
                st = timed([&] { return fbl_attn_fwd_tiled(lq, q, lk, k, lv, v, lo, o, lse, scale, mask, t, stream); },
                           &avg);
            else if (pass == FBL_ATTN_BWD_KV)
                st = timed([&] { return bwd(FBL_BWD_KV, t, FBL_ATTN_TILE_AUTO); }, &avg);
            else
                st = timed([&] { return bwd(FBL_BWD_Q, pick[FBL_ATTN_BWD_KV], t); }, &avg);
            if (st != FBL_OK) break;
            if (ms) ms[t] = avg;
            double score = 1.0 / (double)avg;
            if (objective == FBL_TUNE_GFLOPS_X_MEMEFF) score *= mem_eff(pass, t);
            if (pick[pass] < 0 || score > pick_score) pick[pass] = t, pick_score = score;
        }
        if (st == FBL_OK && pick[pass] < 0) st = FBL_ERR_UNSUPPORTED;
    }
    hipEventDestroy(e0);
    hipEventDestroy(e1);
    if (st != FBL_OK) return st;
    {
        std::lock_guard<std::mutex> lock(g_attn_mu);
        for (uint32_t pass = 0; pass <= FBL_ATTN_BWD_DQ; ++pass)
            if (pick[pass] >= 0) g_attn_tuned[attn_key(pass, lq, lk, mask.kind)] = pick[pass];
    }
    if (best) std::memcpy(best, pick, sizeof(pick));
    // leave o, lse, dq, dk and dv holding the results of the chosen tiles
    if ((st = fbl_attn_fwd_tiled(lq, q, lk, k, lv, v, lo, o, lse, scale, mask, pick[0], stream)) != FBL_OK) return st;
    return bwd(FBL_BWD_ALL, pick[1], pick[2] >= 0 ? pick[2] : FBL_ATTN_TILE_AUTO);
}

int32_t fbl_attn_tuned_tile(uint32_t pass, const fbl_layout* lq, const fbl_layout* lk, uint32_t mask_kind) {
    if (!lq || !lk || pass > FBL_ATTN_BWD_DQ) return -1;
    std::lock_guard<std::mutex> lock(g_attn_mu);
    const auto it = g_attn_tuned.find(attn_key(pass, lq, lk, mask_kind));
    return it == g_attn_tuned.end() ? -1 : it->second;
}

void fbl_attn_tune_reset(void) {
    std::lock_guard<std::mutex> lock(g_attn_mu);
    g_attn_tuned.clear();
}

}  // extern "C"

namespace {

// A projection product, validated: kernel arguments, operand orientation,
// the output/contraction extents and the operands' stored row widths.
struct ProjPlan {
    fbl::GemmArgs p;
    int a_kmajor = 0, b_nmajor = 0;
    int64_t orows = 0, ocols = 0, kc = 0;
    int64_t a_width = 0, b_width = 0;
};

// Orientation and extents of a product from (op, M, K, N) alone.
void proj_shape(uint32_t op, int64_t M, int64_t K, int64_t N, ProjPlan& pl) {
    pl.a_kmajor = op == FBL_PROJ_BWD_WEIGHT;
    pl.b_nmajor = op == FBL_PROJ_BWD_DATA;
    pl.orows = op == FBL_PROJ_BWD_WEIGHT ? K : M;
    pl.ocols = op == FBL_PROJ_BWD_DATA ? K : N;
    pl.kc = op == FBL_PROJ_FWD ? K : (op == FBL_PROJ_BWD_DATA ? N : M);
    pl.a_width = op == FBL_PROJ_BWD_DATA ? N : K;  // X [M, K] or dY [M, N]
    pl.b_width = N;                                // W [K, N] or dY [M, N]
}

// es: element size (2: bf16, 4: fp32).  bf16 operands are staged by 16-byte
// DMA loads (16-byte aligned pointers and rows, output widths a multiple of
// 4, contraction a multiple of 8); fp32 operands by bounds-checked element
// loads (natural alignment only).
fbl_status proj_plan(uint32_t op, int64_t M, int64_t K, int64_t N, const void* a, int64_t lda, const void* b,
                     int64_t ldb, void* c, int64_t ldc, ProjPlan& pl, int es = 2) {
    if (op > FBL_PROJ_BWD_WEIGHT) return FBL_ERR_ARG;
    if (!a || !b || !c) return FBL_ERR_NULL;
    if (M <= 0 || K <= 0 || N <= 0 || M > INT32_MAX || K > INT32_MAX || N > INT32_MAX) return FBL_ERR_SHAPE;
    // stored shapes: a [ra, wa], b [rb, wb], c [rc, wc]; the product's output
    // rows/cols and contraction length
    int64_t ra, wa, rb, wb, rc, wc;
    if (op == FBL_PROJ_FWD) {  // Y = X W
        ra = M, wa = K, rb = K, wb = N, rc = M, wc = N, pl.orows = M, pl.ocols = N, pl.kc = K;
    } else if (op == FBL_PROJ_BWD_DATA) {  // dX = dY W^T
        ra = M, wa = N, rb = K, wb = N, rc = M, wc = K, pl.orows = M, pl.ocols = K, pl.kc = N;
        pl.b_nmajor = 1;
    } else {  // dW = X^T dY
        ra = M, wa = K, rb = M, wb = N, rc = K, wc = N, pl.orows = K, pl.ocols = N, pl.kc = M;
        pl.a_kmajor = 1;
    }
    if (lda < wa || ldb < wb || ldc < wc) return FBL_ERR_LAYOUT;
    const auto aligned = [es](const void* x) { return (reinterpret_cast<uintptr_t>(x) & (es == 2 ? 15u : 3u)) == 0; };
    if (!aligned(a) || !aligned(b) || !aligned(c)) return FBL_ERR_ALIGN;
    if (es == 2 && ((lda * 2) % 16 || (ldb * 2) % 16 || (ldc * 2) % 16)) return FBL_ERR_ALIGN;
    pl.a_width = wa;
    pl.b_width = wb;
    if (es == 2 && (pl.ocols % 4 || pl.kc % 8)) return FBL_ERR_UNSUPPORTED;
    const int64_t sa = ((ra - 1) * lda + wa) * es, sb = ((rb - 1) * ldb + wb) * es, sc = ((rc - 1) * ldc + wc) * es;
    if (sa >= ((int64_t)1 << 31) || sb >= ((int64_t)1 << 31) || sc >= ((int64_t)1 << 31)) return FBL_ERR_UNSUPPORTED;
    if (overlaps(c, sc, a, sa) || overlaps(c, sc, b, sb)) return FBL_ERR_ARG;
    fbl::GemmArgs& p = pl.p;
    p.a = a;
    p.b = b;
    p.c = c;
    p.lda = lda;
    p.ldb = ldb;
    p.ldc = ldc;
    p.M = (int)pl.orows;
    p.N = (int)pl.ocols;
    p.K = (int)pl.kc;
    // The loads move 16-byte chunks and the hardware drops every dword that
    // reaches past a resource's range, so a span ending inside a dword (an
    // odd row width) would lose the operand's last element: the load spans
    // end at the 16-byte chunk holding it.  Pointers and row strides are
    // 16-byte aligned, so that chunk is aligned and never crosses a page.
    const auto chunk_end = [](int64_t n) { return (uint32_t)((n + 15) / 16 * 16); };
    p.a_bytes = chunk_end(sa);
    p.b_bytes = chunk_end(sb);
    p.c_bytes = (uint32_t)sc;  // stores are 4 elements wide and output widths a multiple of 4
    return FBL_OK;
}

// Candidate tiles (C1, C2, C3 of gemm_tiles.hpp) as a bit set over the ids:
// when no tile keeps the padding within 10%, the C1/C2 survivors of least
// padded volume.
uint64_t candidate_set(const ProjPlan& pl) {
    static_assert(fbl::kGemmTileCount <= 64, "tile ids fit the bit set");
    uint64_t c12 = 0, all = 0;
    for (int i = 0; i < fbl::kGemmTileCount; ++i) {
        const fbl::GemmTile& t = fbl::kGemmTiles[i];
        if (!fbl::gemm_c1(t) || !fbl::gemm_c2(t, pl.a_kmajor, pl.b_nmajor, pl.a_width, pl.b_width)) continue;
        c12 |= uint64_t(1) << i;
        if (fbl::gemm_c3(t, pl.orows, pl.ocols, pl.kc)) all |= uint64_t(1) << i;
    }
    if (all || !c12) return all;
    double best = 0;
    for (int i = 0; i < fbl::kGemmTileCount; ++i)
        if (c12 >> i & 1) {
            const double v = fbl::gemm_padded_volume(fbl::kGemmTiles[i], pl.orows, pl.ocols, pl.kc);
            if (!all || v < best) all = uint64_t(1) << i, best = v;
            else if (v == best) all |= uint64_t(1) << i;
        }
    return all;
}

// Per-shape table of measured choices (fbl_proj_tune), the run-time analogue
// of a lookup table keyed by input shape.
struct TunedKey {
    uint32_t op;
    int64_t M, K, N;
    bool operator<(const TunedKey& o) const {
        return std::tie(op, M, K, N) < std::tie(o.op, o.M, o.K, o.N);
    }
};
std::mutex g_tuned_mu;
std::map<TunedKey, int32_t> g_tuned;

int32_t tuned_tile(uint32_t op, int64_t M, int64_t K, int64_t N) {
    std::lock_guard<std::mutex> lock(g_tuned_mu);
    const auto it = g_tuned.find(TunedKey{op, M, K, N});
    return it == g_tuned.end() ? -1 : it->second;
}

// Untuned choice among the candidates, by how many 128 x 128 output tiles
// the product has (n128) and how long its contraction is -- measured on the
// 512 x {2048, 4096} x {8192, 12288}, {1024, 2048} x 4096 x 4096 and 4096 x
// 4096 x {4096, 12288} products and their transposes:
//   n128 >= 1024, contraction >= 2048: the 256 x 256 tiles, 8 wavefronts
//     first when A is read along its rows, 4 first for the weight gradient's
//     transposed A;
//   n128 >= 1024, shorter contraction: 4-wavefront 128 x 128 tiles (for the
//     weight gradient 3-4% ahead of the 256 x 256 tiles, timed interleaved);
//   384 <= n128 < 1024: the 8-wavefront 256 x 128 (forward) or 128 x 256
//     (data gradient) tile, even below one workgroup per CU (two waves per
//     SIMD do more for these than a full grid of 4-wavefront tiles); for the
//     weight gradient's transposed A the 4-wavefront 128 x 128 tile, then
//     128 x 256;
//   256 <= n128 < 384: 4-wavefront 64 x 128 and 128 x 64 tiles;
//   below: the 8-wavefront 128 x 64 tile that splits a deep contraction four
//     ways, then the 4-wavefront 64 x 64 one.
// Orders marked `fill` take the first candidate that gives at least one
// workgroup per CU (256), else the first candidate; the others take the
// first candidate.
int32_t default_tile(const ProjPlan& pl) {
    static const int big[] = {19, 18, 20, 17, 11, 12, 8, 4, 0, 6, 5, 2, 1, 10, 9, 7, 3, 13, 15, 14, 16};
    static const int big_t[] = {18, 20, 19, 17, 11, 12, 8, 4, 0, 6, 5, 2, 1, 10, 9, 7, 3, 13, 15, 14, 16};
    static const int many[] = {0, 4, 8, 1, 2, 5, 6, 11, 12, 10, 9, 7, 3, 13, 15, 14, 16, 17, 18, 19, 20};
    static const int wide[] = {11, 12, 8, 4, 0, 5, 6, 2, 1, 10, 9, 7, 3, 13, 15, 14, 16, 17, 18, 19, 20};
    static const int wide_d[] = {12, 11, 8, 4, 0, 5, 6, 2, 1, 10, 9, 7, 3, 13, 15, 14, 16, 17, 18, 19, 20};
    static const int wide_t[] = {0, 12, 8, 11, 4, 5, 6, 2, 1, 10, 9, 7, 3, 13, 15, 14, 16, 17, 18, 19, 20};
    static const int some[] = {6, 5, 8, 4, 11, 12, 0, 2, 1, 10, 9, 7, 3, 13, 15, 14, 16, 17, 18, 19, 20};
    static const int few[] = {10, 9, 7, 6, 5, 8, 4, 3, 2, 1, 0, 11, 12, 14, 13, 15, 16, 17, 18, 19, 20};
    static_assert(sizeof(many) == sizeof(int) * fbl::kGemmTileCount && sizeof(some) == sizeof(many) &&
                      sizeof(few) == sizeof(many) && sizeof(big) == sizeof(many) && sizeof(big_t) == sizeof(many) &&
                      sizeof(wide) == sizeof(many) && sizeof(wide_d) == sizeof(many) && sizeof(wide_t) == sizeof(many),
                  "every tile ranked once");
    const uint64_t cand = candidate_set(pl);
    const int64_t n128 = ((pl.orows + 127) / 128) * ((pl.ocols + 127) / 128);
    const int* order;
    bool fill = true;
    if (n128 >= 1024) {
        order = pl.kc >= 2048 ? (pl.a_kmajor ? big_t : big) : many;
    } else if (n128 >= 384) {
        order = pl.a_kmajor ? wide_t : (pl.b_nmajor ? wide_d : wide);
        fill = false;
    } else {
        order = n128 >= 256 ? some : few;
    }
    int32_t first = -1;
    for (int i = 0; i < fbl::kGemmTileCount; ++i) {
        const int t = order[i];
        if (!(cand >> t & 1)) continue;
        if (!fill) return t;
        const fbl::GemmTile& g = fbl::kGemmTiles[t];
        if (((pl.orows + g.bm - 1) / g.bm) * ((pl.ocols + g.bn - 1) / g.bn) >= 256) return t;
        if (first < 0) first = t;
    }
    return first >= 0 ? first : order[0];
}

}  // namespace

extern "C" {

int32_t fbl_gemm_tile_count(void) { return fbl::kGemmTileCount; }

fbl_status fbl_gemm_tile_info(int32_t tile, int32_t* info) {
    if (!info) return FBL_ERR_NULL;
    if (tile < 0 || tile >= fbl::kGemmTileCount) return FBL_ERR_ARG;
    const fbl::GemmTile& t = fbl::kGemmTiles[tile];
    const int32_t v[8] = {t.bm, t.bn, t.bk, t.ns, t.wm, t.wn, t.wk, fbl::gemm_lds_bytes(t)};
    std::memcpy(info, v, sizeof(v));
    return FBL_OK;
}

fbl_status fbl_proj_candidates(uint32_t op, int64_t M, int64_t K, int64_t N, int32_t* tiles, int32_t cap,
                               int32_t* count) {
    if (!count || (cap > 0 && !tiles)) return FBL_ERR_NULL;
    if (op > FBL_PROJ_BWD_WEIGHT) return FBL_ERR_ARG;
    if (M <= 0 || K <= 0 || N <= 0 || M > INT32_MAX || K > INT32_MAX || N > INT32_MAX) return FBL_ERR_SHAPE;
    ProjPlan pl;
    proj_shape(op, M, K, N, pl);
    const uint64_t cand = candidate_set(pl);
    int32_t n = 0;
    for (int t = 0; t < fbl::kGemmTileCount; ++t)
        if (cand >> t & 1) {
            if (n < cap) tiles[n] = t;
            ++n;
        }
    *count = n;
    return FBL_OK;
}

fbl_status fbl_proj_dt(uint32_t op, int32_t dtype, int64_t M, int64_t K, int64_t N, const void* a, int64_t lda,
                       const void* b, int64_t ldb, void* c, int64_t ldc, int32_t tile, void* stream) {
    if (dtype != FBL_BF16 && dtype != FBL_F32) return FBL_ERR_DTYPE;
    ProjPlan pl;
    const fbl_status st = proj_plan(op, M, K, N, a, lda, b, ldb, c, ldc, pl, dtype == FBL_BF16 ? 2 : 4);
    if (st != FBL_OK) return st;
    if (dtype == FBL_F32) {  // one tile shape (64 x 64 outputs, 16-deep steps)
        if (tile != FBL_GEMM_TILE_AUTO) return FBL_ERR_ARG;
        const hipError_t e = fbl::launch_proj_gemm_f32(pl.a_kmajor, pl.b_nmajor, pl.p, static_cast<hipStream_t>(stream));
        return e == hipSuccess ? FBL_OK : FBL_ERR_HIP;
    }
    if (tile < FBL_GEMM_TILE_AUTO || tile >= fbl::kGemmTileCount) return FBL_ERR_ARG;
    if (tile == FBL_GEMM_TILE_AUTO) {
        tile = tuned_tile(op, M, K, N);
        if (tile < 0) tile = default_tile(pl);
    }
    const hipError_t e = fbl::launch_proj_gemm(pl.a_kmajor, pl.b_nmajor, tile, pl.p, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? FBL_OK : FBL_ERR_HIP;
}

fbl_status fbl_proj_tune(uint32_t op, int64_t M, int64_t K, int64_t N, const void* a, int64_t lda, const void* b,
                         int64_t ldb, void* c, int64_t ldc, uint32_t objective, int32_t reps, float* ms,
                         int32_t* best, void* stream) {
    ProjPlan pl;
    const fbl_status st = proj_plan(op, M, K, N, a, lda, b, ldb, c, ldc, pl);
    if (st != FBL_OK) return st;
    if (objective > FBL_TUNE_GFLOPS_X_MEMEFF || reps < 1 || reps > 1000) return FBL_ERR_ARG;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if (ms)
        for (int t = 0; t < fbl::kGemmTileCount; ++t) ms[t] = -1.0f;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
        if (e0) hipEventDestroy(e0);
        return FBL_ERR_HIP;
    }
    // minimal bytes: every operand read once, the result written once
    const double flops = 2.0 * (double)pl.orows * (double)pl.ocols * (double)pl.kc;
    const double min_bytes = 2.0 * ((double)pl.orows * pl.kc + (double)pl.kc * pl.ocols + (double)pl.orows * pl.ocols);
    int32_t pick = -1;
    double pick_score = 0;
    fbl_status out = FBL_OK;
    const uint64_t cand = candidate_set(pl);
    for (int t = 0; t < fbl::kGemmTileCount && out == FBL_OK; ++t) {
        if (!(cand >> t & 1)) continue;
        hipError_t e = fbl::launch_proj_gemm(pl.a_kmajor, pl.b_nmajor, t, pl.p, s);  // warm-up
        if (e == hipSuccess) e = hipEventRecord(e0, s);
        for (int r = 0; r < reps && e == hipSuccess; ++r) e = fbl::launch_proj_gemm(pl.a_kmajor, pl.b_nmajor, t, pl.p, s);
        if (e == hipSuccess) e = hipEventRecord(e1, s);
        if (e == hipSuccess) e = hipEventSynchronize(e1);
        float total = 0;
        if (e == hipSuccess) e = hipEventElapsedTime(&total, e0, e1);
        if (e != hipSuccess) {
            out = FBL_ERR_HIP;
            break;
        }
        const float avg = total / (float)reps;
        if (ms) ms[t] = avg;
        double score = 1.0 / (double)avg;
        if (objective == FBL_TUNE_GFLOPS_X_MEMEFF) {
            // staged bytes: each row block of A is read once per column block
            // of the output and each column block of B once per row block
            const fbl::GemmTile& g = fbl::kGemmTiles[t];
            const double staged =
                2.0 * ((double)pl.orows * pl.kc * (double)((pl.ocols + g.bn - 1) / g.bn) +
                       (double)pl.kc * pl.ocols * (double)((pl.orows + g.bm - 1) / g.bm) + (double)pl.orows * pl.ocols);
            score = flops / (avg * 1e-3) * (min_bytes / staged);
        }
        if (pick < 0 || score > pick_score) pick = t, pick_score = score;
    }
    hipEventDestroy(e0);
    hipEventDestroy(e1);
    if (out != FBL_OK) return out;
    if (pick < 0) return FBL_ERR_UNSUPPORTED;
    {
        std::lock_guard<std::mutex> lock(g_tuned_mu);
        g_tuned[TunedKey{op, M, K, N}] = pick;
    }
    if (best) *best = pick;
    // leave c holding the product computed with the chosen tile
    const hipError_t e = fbl::launch_proj_gemm(pl.a_kmajor, pl.b_nmajor, pick, pl.p, s);
    return e == hipSuccess ? FBL_OK : FBL_ERR_HIP;
}

fbl_status fbl_proj(uint32_t op, int64_t M, int64_t K, int64_t N, const void* a, int64_t lda, const void* b,
                    int64_t ldb, void* c, int64_t ldc, int32_t tile, void* stream) {
    return fbl_proj_dt(op, FBL_BF16, M, K, N, a, lda, b, ldb, c, ldc, tile, stream);
}

int32_t fbl_proj_tuned_tile(uint32_t op, int64_t M, int64_t K, int64_t N) { return tuned_tile(op, M, K, N); }

fbl_status fbl_proj_auto_tile(uint32_t op, int64_t M, int64_t K, int64_t N, int32_t* tile) {
    if (!tile) return FBL_ERR_NULL;
    if (op > FBL_PROJ_BWD_WEIGHT) return FBL_ERR_ARG;
    if (M <= 0 || K <= 0 || N <= 0 || M > INT32_MAX || K > INT32_MAX || N > INT32_MAX) return FBL_ERR_SHAPE;
    ProjPlan pl;
    proj_shape(op, M, K, N, pl);
    const int32_t t = tuned_tile(op, M, K, N);
    *tile = t >= 0 ? t : default_tile(pl);
    return FBL_OK;
}

void fbl_proj_tune_reset(void) {
    std::lock_guard<std::mutex> lock(g_tuned_mu);
    g_tuned.clear();
}

}  // extern "C"
