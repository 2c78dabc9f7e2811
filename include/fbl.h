/*
 * fbl.h -- C ABI of the layout-copy-free attention forward/backward library
 * for AMD Instinct MI355X (gfx950).
 *
 * What it computes.  Multi-head attention forward and backward of a
 * fine-tuning step, directly on token-major activations [B, S, H*d] as a QKV
 * projection writes them.  The paper's attention module (section 2.2, the
 * LoRA fine-tuning example) forms P = softmax(Q K^T) and multiplies by V; the
 * head split (reshape (B,S,D) -> (B,S,H,HD)) and the transpose to
 * (B,H,S,HD) (section 4.3.1, the multi-head attention chain) are not carried
 * out as copies: they are folded into one affine index map per tensor
 * (section 4.3.2, the composed tile-index function f3 o f2 o f1), which the
 * kernels apply when they stage (rows x d) row tiles -- the R-Tile of
 * section 4.2 -- into LDS.  Which tile each kernel stages is chosen per
 * shape from a filtered candidate set, by measurement (fbl_attn_tune) or a
 * preference order.  No layout-conversion kernel is ever launched.
 * The projection products around attention (fbl_proj: Y = X W and its two
 * gradients, also for LoRA adapters) read the same token-major activations
 * in place, and Q, K, V can be views of one packed projection output
 * (fbl_layout_packed_qkv).
 *
 * Conventions shared by every entry point.
 *  - Element (b, h, s, i) of a tensor described by an fbl_layout L is at
 *    element offset  b*L.sb + s*L.ss + h*L.sh + i*L.sd  from its base pointer.
 *  - Q, O, dO, dQ have Hq heads and S_q tokens; K, V, dK, dV have Hkv heads
 *    and S_kv tokens; query head h reads key/value head h / (Hq/Hkv)
 *    (grouped-query attention with contiguous groups).  All tensors share B.
 *    S_q == S_kv is self-attention; S_q != S_kv is cross-attention (the
 *    encoder-decoder attention section 2.2 lists among the attention variants
 *    whose layouts conflict), which takes no causal mask.
 *  - Scores are  scale * q_i . k_j ; key j is allowed for query i iff
 *    (!causal || j <= i) && (!key_padding || j < kv_len[b]).  Disallowed
 *    scores are -inf.  A query row with no allowed key gets O = 0,
 *    LSE = -inf and contributes no gradient.
 *  - LSE is float32 [B, Hq, S_q], contiguous, natural-log log-sum-exp of the
 *    scaled masked scores.
 *  - Storage type of Q, K, V, O, dO, dQ, dK, dV is one fbl_dtype for the whole
 *    call (fp32 or bf16); accumulation is fp32.
 *  - Ownership: the caller owns every buffer (device memory for tensors,
 *    host memory for descriptors).  The library never allocates or frees
 *    device memory and never synchronises (except fbl_proj_tune, which
 *    waits for its own timing events).  Inputs are read-only; outputs are
 *    fully overwritten
 *    (no accumulate semantics) and must not alias inputs.
 *  - Errors: every check runs on the host before the first launch, so an
 *    error return means nothing was enqueued.  Return codes are the only
 *    error channel; nothing aborts or throws across the ABI.
 *  - Streams: `stream` is a hipStream_t (NULL = the null stream).  On FBL_OK
 *    the work is enqueued on it and the call returns without waiting.
 */
#ifndef FBL_H
#define FBL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    FBL_OK = 0,
    FBL_ERR_NULL = 1,        /* a required pointer is NULL                          */
    FBL_ERR_SHAPE = 2,       /* non-positive or mutually inconsistent extents       */
    FBL_ERR_DTYPE = 3,       /* unknown dtype, or dtypes differ between tensors     */
    FBL_ERR_LAYOUT = 4,      /* a tile-legality check failed (strides, tile shape)  */
    FBL_ERR_ALIGN = 5,       /* base pointer or row stride not 16-byte aligned      */
    FBL_ERR_UNSUPPORTED = 6, /* shape, head dim or mask combination not implemented  */
    FBL_ERR_WORKSPACE = 7,   /* workspace NULL or below fbl_attn_bwd_workspace_min  */
    FBL_ERR_HIP = 8,         /* the HIP runtime reported an error at launch         */
    FBL_ERR_ARG = 9          /* other invalid argument (non-finite scale, aliasing) */
} fbl_status;

typedef enum { FBL_F32 = 0, FBL_BF16 = 1 } fbl_dtype;

/*
 * Layout descriptor of one tensor with logical dims (B, H, S, D) -- the
 * logical shape S(t) and physical layout L(t) of a tensor in the paper's problem
 * statement (section 3.1) -- plus the tile-legality parameter of its R-Tile.
 *
 * Strides are in elements.  Token-major defaults: sd = 1, sh = D,
 * ss = H*D (row stride), sb = S*ss.  A row stride larger than H*D describes a
 * view into a wider packed projection output without copying it.
 * tile_d is the R-Tile width in head-dim elements: it must divide D (tile
 * boundary preservation, section 4.3.1), with sd == 1 (intra-tile
 * continuity, section 4.3.1).  The kernels stage whole head rows; the number
 * of rows per staged tile belongs to the kernel's tile configuration
 * (fbl_attn_tile_info), not to the tensor.
 */
typedef struct {
    int32_t dtype;     /* fbl_dtype                                   */
    int32_t reserved0; /* zero                                        */
    int32_t tile_d;    /* R-Tile columns (head-dim elements)          */
    int32_t reserved1; /* zero                                        */
    int64_t B, S, H, D;
    int64_t sb, ss, sh, sd;
} fbl_layout;

#define FBL_MASK_CAUSAL 1u      /* key j allowed only for queries i >= j        */
#define FBL_MASK_KEY_PADDING 2u /* key j allowed only if j < kv_len[b]           */

typedef struct {
    uint32_t kind;          /* OR of FBL_MASK_* bits                             */
    uint32_t reserved;      /* zero                                              */
    const int32_t* kv_len;  /* device pointer, int32 [B]; required with KEY_PADDING;
                               values are clamped to [0, S_kv]                  */
} fbl_mask;

/*
 * Fill *out with the token-major descriptor of a tensor with B batches, S
 * tokens, H heads of D elements, and run the tile-legality checks of the
 * paper's tile propagation (section 4.3.1): the R-Tile column count tile_d
 * must divide the head dim (tile boundary preservation), the innermost
 * stride is 1 (intra-tile continuity), and rows and heads must not overlap.
 *
 *   dtype        FBL_F32 or FBL_BF16.
 *   row_stride   elements between consecutive tokens; 0 means H*D.
 *                Must be >= H*D.
 *   batch_stride elements between consecutive batches; 0 means S*row_stride.
 *                Must be >= S*row_stride when B > 1.
 *   tile_d       R-Tile width in head-dim elements; 0 means D.  Must divide D
 *                and span a multiple of 16 bytes.
 * Returns FBL_ERR_NULL, FBL_ERR_SHAPE, FBL_ERR_DTYPE or FBL_ERR_LAYOUT on
 * failure (then *out is left zeroed).  Pure host function.
 */
fbl_status fbl_layout_desc(fbl_layout* out, int32_t dtype, int64_t B, int64_t S, int64_t H, int64_t D,
                           int64_t row_stride, int64_t batch_stride, int64_t tile_d);

/*
 * Descriptors of Q, K and V as views into one packed projection output of
 * logical shape [B, S, (Hq + 2*Hkv) * D] -- the fused QKV projection writes
 * each token row as Hq query heads, then Hkv key heads, then Hkv value heads.
 * The reshape/transpose chain of section 4.3.1 then splits the row into three
 * head-split tensors; here each is an index map with row stride
 * (Hq + 2*Hkv) * D and a start offset, so none of them is copied out.
 *   lq, lk, lv      filled with the three descriptors (as fbl_layout_desc
 *                   would for a tensor of Hq, Hkv, Hkv heads with that row
 *                   stride, and the same tile-legality checks).
 *   k_off, v_off    element offsets of K and V from the packed base (Q is at
 *                   offset 0): Hq*D and (Hq + Hkv)*D.
 *   batch_stride    elements between batches; 0 means S * (Hq + 2*Hkv) * D.
 * The same descriptors and offsets describe a packed gradient buffer
 * [B, S, (Hq + 2*Hkv) * D] receiving dQ, dK, dV.  Returns the status of
 * fbl_layout_desc; on failure all outputs are left zeroed.  Pure host function.
 */
fbl_status fbl_layout_packed_qkv(fbl_layout* lq, fbl_layout* lk, fbl_layout* lv, int64_t* k_off, int64_t* v_off,
                                 int32_t dtype, int64_t B, int64_t S, int64_t Hq, int64_t Hkv, int64_t D,
                                 int64_t batch_stride, int64_t tile_d);

/*
 * Host evaluation of the index map: element offset of logical (b, h, s, i),
 * or -1 when the descriptor is NULL or an index is out of range.  This is
 * the composition of the head split and transpose of the multi-head
 * attention chain (section 4.3.1) into one coordinate map (section 4.3.2,
 * f3 o f2 o f1), evaluated for one element.
 */
int64_t fbl_layout_offset(const fbl_layout* l, int64_t b, int64_t h, int64_t s, int64_t i);

/*
 * Diagnostic: evaluate the index map (the tile-based index transformation of
 * section 4.3, device side) on the GPU with the same device code the
 * attention kernels use to address tensors, writing out[((b*H + h)*S + s)*D + i]
 * = offset(b, h, s, i) as int64 into the device buffer `out` of
 * B*H*S*D elements.  Enqueued on `stream`.
 */
fbl_status fbl_layout_map_device(const fbl_layout* l, int64_t* out, void* stream);

/*
 * Attention forward: O = softmax(scale Q K^T) V per query head, the attention
 * module of section 2.2 (the LoRA fine-tuning example), with the masks and
 * grouped-query head map described above, and the row log-sum-exp saved for
 * the backward.  QK^T and the product with V are the consecutive
 * matrix-product pair of section 4.4.2, fused in one kernel.  bf16 storage
 * runs the forward tile FBL_ATTN_TILE_AUTO resolves to (fbl_attn_auto_tiles).
 *   lq/q     queries, Hq heads.       lk/k, lv/v  keys and values, Hkv heads.
 *   lo/o     output, same extents as q.
 *   lse      float32 [B, Hq, S_q] contiguous, written (saved for the backward).
 *   scale    softmax scale (finite), e.g. 1/sqrt(D).
 *   mask     see fbl_mask.
 * Supported: D in {32, 64, 128}; Hq % Hkv == 0; for every tensor
 * (S + 128) * ss * element size at most 2^31 bytes -- rows are addressed
 * from each (batch, head) base with 32-bit offsets, and tiles reach up to
 * 128 rows past the last token; a causal mask needs S_q == S_kv.  Otherwise
 * FBL_ERR_UNSUPPORTED.
 * Checks: non-NULL pointers; one dtype; lq.B == lk.B == lv.B == lo.B;
 * lk and lv extents equal (S_kv = lk.S); lq.D == lk.D;
 * lo extents equal lq's; sd == 1; tile_d divides D; base pointers and
 * row strides 16-byte aligned; kv_len given with KEY_PADDING; o and lse do
 * not overlap any input.
 */
fbl_status fbl_attn_fwd(const fbl_layout* lq, const void* q, const fbl_layout* lk, const void* k,
                        const fbl_layout* lv, const void* v, const fbl_layout* lo, void* o, float* lse,
                        float scale, fbl_mask mask, void* stream);

/*
 * Bytes of device workspace for the fastest backward at these shapes.
 * Part 1, always: one pair of fp32 per query row, [B, Hq, S] x
 * (LSE * log2(e), D_i = sum_k dO_ik O_ik), rounded up to 256 bytes.
 * Part 2, bf16 storage only: the gradient of the scores dS = P o (dP - D)
 * (section 4.1's softmax backward, FTD-C) in bf16,
 * B*Hq*ceil(S_q/32)*ceil(S_kv/32) blocks of 32x32 elements (2 KB each),
 * written by the key/value pass and contracted with K by the dQ pass -- the
 * dQ pass then does not recompute S and dP.  Part 2 is omitted (the size
 * equals fbl_attn_bwd_workspace_min) for fp32 storage and when one head's
 * blocks would reach 2 GiB (S_q = S_kv above 32736).
 * Part 3, with part 2, where the key/value pass has fewer than 512 blocks of
 * 128 keys (B * Hkv * ceil(S_kv/128)) and the first block at least 16 query
 * iterations per share (Hq/Hkv * ceil(S_q/32), ceil(S_q/64) at D = 32): the
 * pass splits each key block's iterations among 2, or 4, workgroups (4 below
 * 128 blocks when the iterations allow), and this part holds their fp32
 * partial dK and dV, 2 * split * B*S_kv*Hkv*D floats, which a reduction adds
 * in a fixed order.  Without a causal mask the split is used only while the
 * split grid fits the resident workgroups (256, or 512 at D = 64).
 */
fbl_status fbl_attn_bwd_workspace(const fbl_layout* lq, const fbl_layout* lk, size_t* bytes);

/*
 * Smallest workspace fbl_attn_bwd accepts (section 4.1's backward with the
 * dQ products recomputed): part 1 above only.  With any
 * workspace smaller than fbl_attn_bwd_workspace the dQ pass recomputes S and
 * dP from Q, K, V, dO and the row statistics instead of reading stored dS
 * (same results up to rounding order).
 */
fbl_status fbl_attn_bwd_workspace_min(const fbl_layout* lq, const fbl_layout* lk, size_t* bytes);

/*
 * Attention backward of L = sum(O * dO): writes dQ (Hq heads), dK and dV
 * (Hkv heads; each the sum over the query heads of its group) -- the chain
 * rule through the matrix-product gradients of section 4.1 (forward-tensor
 * dependent: they read Q, K, V and dO along other axes than the forward,
 * dK and dV reducing over queries, dQ over keys) and the softmax gradient
 * (section 4.1's forward-dependent, consistent-access class).  The softmax
 * probabilities are recomputed from q, k and the saved lse.  No output is
 * accumulated atomically, so the results are bitwise repeatable.  o and lse
 * must be the forward's outputs for q, k, v.
 *   ws/ws_bytes  device workspace of at least fbl_attn_bwd_workspace_min
 *                bytes, 256-byte aligned; its contents on entry do not matter.
 *                With parts 1 and 2 of fbl_attn_bwd_workspace the key/value
 *                pass stores dS there for the dQ pass; with all of it the
 *                key/value pass may also be split (see fbl_attn_bwd_workspace).
 *                Each size gives bitwise repeatable results; sizes that select
 *                different passes may differ in the last bits.
 * Same checks as fbl_attn_fwd for the shared arguments, plus: ldo/ldq
 * extents equal lq's, ldk/ldv extents equal lk's, the row-offset limit of
 * fbl_attn_fwd for every layout, outputs do not overlap inputs, each other or
 * the workspace, and the workspace does not overlap an input or lse (it is
 * written while they are read).  bf16 storage runs the kv and dQ tiles
 * FBL_ATTN_TILE_AUTO resolves to.
 * Up to 128 keys (S_kv <= 128; fp32 storage only at D <= 64), when there are
 * at least 128 (batch, key/value head) pairs or each pair has at most 64
 * query blocks (Hq/Hkv * ceil(S_q / 64), ceil(S_q / 32) at D = 128), the
 * backward is one launch: a workgroup holds all keys of one (batch, key/value head) in
 * LDS and, per block of queries of its group, forms D_i, the dK and dV
 * contributions and the block's dS, and contracts that dS with K into dQ --
 * no workspace is read or written.  Its results agree with the three-launch
 * path of fbl_attn_bwd_phases up to rounding order, not bit for bit.
 */
fbl_status fbl_attn_bwd(const fbl_layout* lq, const void* q, const fbl_layout* lk, const void* k,
                        const fbl_layout* lv, const void* v, const fbl_layout* lo, const void* o,
                        const fbl_layout* ldo, const void* dO, const float* lse, float scale, fbl_mask mask,
                        const fbl_layout* ldq, void* dq, const fbl_layout* ldk, void* dk,
                        const fbl_layout* ldv, void* dv, void* ws, size_t ws_bytes, void* stream);

/*
 * The three launches of fbl_attn_bwd -- the backward's two reduction
 * directions of sections 4.1 and 4.2 (the key/value pass reduces over
 * queries, the dQ pass over keys) after the row statistics -- selectable one
 * by one (same arguments
 * and checks as fbl_attn_bwd; `phases` is an OR of the bits below, enqueued
 * in the order listed).  fbl_attn_bwd(...) equals
 * fbl_attn_bwd_phases(FBL_BWD_ALL, ...), which takes the one-launch backward
 * where fbl_attn_bwd does; the three phases called separately (or
 * fbl_attn_bwd_tiled with an explicit tile) always run the three launches
 * below, and give the same bits on any streams they are ordered on.
 * FBL_BWD_KV and FBL_BWD_Q read what
 * FBL_BWD_PREP left in the workspace, so the same workspace must be passed to
 * all phases.  With the full workspace (fbl_attn_bwd_workspace bytes, bf16)
 * FBL_BWD_Q reads the dS that FBL_BWD_KV stored, so KV must run before Q;
 * with a smaller one KV and Q are independent of each other.
 *   FBL_BWD_PREP  per query row: LSE * log2(e) and D_i = sum_k dO_ik O_ik
 *   FBL_BWD_KV    key/value-major pass: recompute P, write dK and dV (and,
 *                 with the full workspace, dS)
 *   FBL_BWD_Q     dQ: from the stored dS, or query-major with P and dP
 *                 recomputed
 */
#define FBL_BWD_PREP 1u
#define FBL_BWD_KV 2u
#define FBL_BWD_Q 4u
#define FBL_BWD_ALL 7u
fbl_status fbl_attn_bwd_phases(uint32_t phases, const fbl_layout* lq, const void* q, const fbl_layout* lk,
                               const void* k, const fbl_layout* lv, const void* v, const fbl_layout* lo,
                               const void* o, const fbl_layout* ldo, const void* dO, const float* lse, float scale,
                               fbl_mask mask, const fbl_layout* ldq, void* dq, const fbl_layout* ldk, void* dk,
                               const fbl_layout* ldv, void* dv, void* ws, size_t ws_bytes, void* stream);

/*
 * The number of kernel launches fbl_attn_bwd_tiled(phases, ...) enqueues (the
 * passes of section 4.1's backward, or the one-launch form) for
 * query/key descriptors lq and lk, mask bits mask_kind (FBL_MASK_*), a
 * workspace of ws_bytes and the requested tiles: 1 for the one-launch
 * backward (fbl_attn_bwd: FBL_BWD_ALL, automatic tiles, the shapes given at
 * fbl_attn_bwd); else
 * one per phase bit, plus one with FBL_BWD_KV when the key/value pass is
 * split (its partial sums are then added by a reduction launch).  Checks the
 * descriptors as fbl_attn_bwd does (FBL_ERR_* as there) and the tiles as
 * fbl_attn_bwd_tiled.  Host only; reads no data pointer.
 */
fbl_status fbl_attn_bwd_launches(uint32_t phases, const fbl_layout* lq, const fbl_layout* lk, uint32_t mask_kind,
                                 size_t ws_bytes, int32_t kv_tile, int32_t dq_tile, int32_t* launches);

/*
 * Tile configurations of the attention kernels (bf16 storage).  Each pass
 * stages one kind of row tile of a token-major tensor -- the R-Tile of
 * section 4.2, whole head rows -- and gives every wavefront a block of rows
 * it keeps in registers:
 *   FBL_ATTN_FWD     the forward: K/V tiles of `cols` keys; each wavefront
 *                    owns `per_wave` queries of a workgroup's `rows`;
 *   FBL_ATTN_BWD_KV  the backward's key/value pass: Q/dO tiles of `cols`
 *                    queries; each wavefront owns 32 of the workgroup's
 *                    `rows` keys;
 *   FBL_ATTN_BWD_DQ  the backward's dQ pass from stored dS: K tiles of 32
 *                    keys; each wavefront owns 32 of the `rows` queries.
 * fbl_attn_tile_count gives the number of ids; fbl_attn_tile_info writes 8
 * values for one id at head dim D (32, 64 or 128):
 *   info[0] pass   info[1] rows   info[2] cols   info[3] wavefronts
 *   info[4] per_wave   info[5] workgroups per CU   info[6] LDS bytes
 *   info[7] 1 if the tile passes C1 and C2 at this head dim (runs), else 0.
 * FBL_ERR_NULL, FBL_ERR_ARG (id out of range), FBL_ERR_UNSUPPORTED (D).
 */
#define FBL_ATTN_FWD 0u
#define FBL_ATTN_BWD_KV 1u
#define FBL_ATTN_BWD_DQ 2u
#define FBL_ATTN_TILE_AUTO (-1)
int32_t fbl_attn_tile_count(void);
fbl_status fbl_attn_tile_info(int32_t tile, int64_t D, int32_t* info);

/*
 * Candidate tiles of one pass for the shapes lq (queries) and lk (keys):
 * the three progressive filters of the R-Tile candidate generation (section
 * 4.2, step 1, and the supplementary algorithm), read for gfx950 --
 *   C1 compute alignment: whole 32x32 MFMA blocks per wavefront and per
 *      staged tile, whole 16-deep chunks over the head dim, 2-8 wavefronts;
 *   C2 memory alignment and capacity: the workgroups a CU holds fit its
 *      160 KB of LDS; staged rows whole 16-byte loads and staged tiles whole
 *      1 KB wavefront loads spread evenly over the wavefronts; the per-lane
 *      registers fit a wavefront's share of the register file;
 *   C3 shape: padding the sequence to whole workgroup row blocks and whole
 *      staged tiles adds at most 10%; if no tile qualifies, the C1/C2
 *      survivors of least padded volume.
 * Writes up to `cap` ids in increasing order and the count (which may exceed
 * cap).  bf16 descriptors only (FBL_ERR_DTYPE otherwise: fp32 storage has
 * one configuration per pass).  Host only.
 */
fbl_status fbl_attn_candidates(uint32_t pass, const fbl_layout* lq, const fbl_layout* lk, int32_t* tiles,
                               int32_t cap, int32_t* count);

/*
 * The R-Tile choice of section 4.2 for one shape, the per-shape lookup the
 * paper's runtime makes (section 5.5): the ids FBL_ATTN_TILE_AUTO resolves to
 * for (lq, lk, mask kind): tiles[0]
 * forward, tiles[1] kv pass, tiles[2] dQ pass -- the measured choice of
 * fbl_attn_tune for this shape when the process holds one, else the first
 * candidate in a preference order measured on MI355X.  Host only.
 */
fbl_status fbl_attn_auto_tiles(const fbl_layout* lq, const fbl_layout* lk, uint32_t mask_kind, int32_t* tiles);

/*
 * fbl_attn_fwd and fbl_attn_bwd_phases with explicit R-Tile shapes (section
 * 4.2; fbl_attn_bwd is
 * fbl_attn_bwd_tiled(FBL_BWD_ALL, ..., FBL_ATTN_TILE_AUTO, FBL_ATTN_TILE_AUTO,
 * stream)): `tile`, `kv_tile`, `dq_tile` are ids of the right pass that pass
 * C1 and C2 at this head dim
 * (FBL_ERR_ARG for an id of another pass or out of range, FBL_ERR_UNSUPPORTED
 * for one the filters exclude at this head dim), or FBL_ATTN_TILE_AUTO.  Any
 * legal tile runs any shape (C3 only ranks them); every tile gives results
 * within the same tolerance, and one tile is bitwise repeatable.  fp32
 * storage takes FBL_ATTN_TILE_AUTO only.  dq_tile applies when the dQ pass
 * reads stored dS (the workspace holds it).  Otherwise as fbl_attn_fwd /
 * fbl_attn_bwd.
 */
fbl_status fbl_attn_fwd_tiled(const fbl_layout* lq, const void* q, const fbl_layout* lk, const void* k,
                              const fbl_layout* lv, const void* v, const fbl_layout* lo, void* o, float* lse,
                              float scale, fbl_mask mask, int32_t tile, void* stream);
fbl_status fbl_attn_bwd_tiled(uint32_t phases, const fbl_layout* lq, const void* q, const fbl_layout* lk,
                              const void* k, const fbl_layout* lv, const void* v, const fbl_layout* lo, const void* o,
                              const fbl_layout* ldo, const void* dO, const float* lse, float scale, fbl_mask mask,
                              const fbl_layout* ldq, void* dq, const fbl_layout* ldk, void* dk, const fbl_layout* ldv,
                              void* dv, void* ws, size_t ws_bytes, int32_t kv_tile, int32_t dq_tile, void* stream);

/*
 * Measured tile selection for one attention shape (section 4.2's unified
 * selection, per pass; the per-shape table is the analogue of the paper's
 * lookup table for dynamic shapes).  Runs the forward, then the backward, on
 * the caller's buffers (the arguments of fbl_attn_fwd and fbl_attn_bwd
 * together); times every candidate of each pass (fbl_attn_candidates) once
 * untimed and `reps` (1..1000) times with HIP events on `stream` -- the kv
 * pass with the backward's statistics phase done once before, the dQ pass
 * (only when the workspace holds stored dS) on the dS the kv pass left --
 * and keeps, per pass, the id maximising
 *   FBL_TUNE_TIME              1 / average time, or
 *   FBL_TUNE_GFLOPS_X_MEMEFF   GFLOP/s x MemEfficiency (section 4.2): the
 *                              pass's minimal bytes over the bytes its tile
 *                              schedule stages (the forward re-reads a
 *                              query block's K/V rows once per block of
 *                              `rows` queries, the dQ pass its K rows).
 * The choices go to a per-process table keyed by pass, dtype, extents, heads,
 * head dim and mask kind, which FBL_ATTN_TILE_AUTO consults (thread-safe;
 * fbl_attn_tuned_tile reads it, -1 if absent; fbl_attn_tune_reset clears
 * it).  ms (optional, fbl_attn_tile_count() floats): each timed id's average
 * milliseconds, -1 for the others; best (optional, 3 int32): the chosen
 * forward, kv and dQ ids (-1 for dQ when it was not tuned).  Blocks until the
 * timed launches finish; on return o, lse, dq, dk, dv hold the results of
 * the chosen tiles.  bf16 only (FBL_ERR_DTYPE); FBL_ERR_ARG for an unknown
 * objective or reps out of range; otherwise the statuses of fbl_attn_fwd and
 * fbl_attn_bwd.
 */
fbl_status fbl_attn_tune(const fbl_layout* lq, const void* q, const fbl_layout* lk, const void* k,
                         const fbl_layout* lv, const void* v, const fbl_layout* lo, void* o, float* lse,
                         const fbl_layout* ldo, const void* dO, float scale, fbl_mask mask, const fbl_layout* ldq,
                         void* dq, const fbl_layout* ldk, void* dk, const fbl_layout* ldv, void* dv, void* ws,
                         size_t ws_bytes, uint32_t objective, int32_t reps, float* ms, int32_t* best, void* stream);
int32_t fbl_attn_tuned_tile(uint32_t pass, const fbl_layout* lq, const fbl_layout* lk, uint32_t mask_kind);
void fbl_attn_tune_reset(void);

/*
 * fbl_attn_bwd for callers that cannot allocate device memory -- code under
 * HIP graph capture, serving loops and harnesses that forbid hipMalloc.  The
 * arguments are fbl_attn_bwd's without the workspace: the backward's scratch
 * is one library-owned device array of FBL_NOALLOC_SCRATCH_BYTES per GPU,
 * held from the library's first use on that GPU until the process ends, and
 * used as the workspace of fbl_attn_bwd would be (so the stored-dS path and
 * the split key/value pass run exactly when their parts fit in it; results
 * equal fbl_attn_bwd's with a workspace of that size, bit for bit).  The
 * call allocates and frees nothing.  Returns FBL_ERR_WORKSPACE when even
 * fbl_attn_bwd_workspace_min exceeds the array (more than
 * FBL_NOALLOC_SCRATCH_BYTES / 8 query rows, B*Hq*S_q, about 8 million), and
 * fbl_attn_bwd's statuses otherwise.  All calls on one GPU share the array:
 * calls that can run at the same time on one GPU (on streams with no order
 * between them) race; calls on one stream, or ordered by events, do not.
 */
#define FBL_NOALLOC_SCRATCH_BYTES (64u << 20)
fbl_status fbl_attn_bwd_noalloc(const fbl_layout* lq, const void* q, const fbl_layout* lk, const void* k,
                                const fbl_layout* lv, const void* v, const fbl_layout* lo, const void* o,
                                const fbl_layout* ldo, const void* dO, const float* lse, float scale, fbl_mask mask,
                                const fbl_layout* ldq, void* dq, const fbl_layout* ldk, void* dk,
                                const fbl_layout* ldv, void* dv, void* stream);

/*
 * Projection matrix products of the linear layers around attention, on the
 * same token-major activations (bf16 operands and result, fp32 accumulation).
 * Section 4.1 classes matrix products as forward-tensor-dependent: the
 * gradients read the stored X, W and dY along other axes than the forward
 * (section 4.2).  No operand is transposed in memory; each product reads the
 * stored tiles row-wise or transposed as its contraction requires.
 *   FBL_PROJ_FWD         c = Y  [M, N] = X [M, K] . W [K, N]     a = X,  b = W
 *   FBL_PROJ_BWD_DATA    c = dX [M, K] = dY [M, N] . W^T         a = dY, b = W
 *   FBL_PROJ_BWD_WEIGHT  c = dW [K, N] = X^T . dY [M, N]         a = X,  b = dY
 * All matrices are row-major with leading dimensions (elements between rows)
 * lda, ldb, ldc, each at least its row width, so column views of wider
 * buffers (e.g. a packed QKV projection output) are accepted without copies.
 *   tile     the workgroup tile configuration: FBL_GEMM_TILE_AUTO, or an
 *            id in [0, fbl_gemm_tile_count()) (see fbl_gemm_tile_info;
 *            ids 0-3 have the names below, rows x cols of the op's output).
 *            AUTO takes the tile fbl_proj_tune measured best for this
 *            (op, M, K, N) in this process, else the first candidate (see
 *            fbl_proj_candidates) that gives at least 256 workgroups in a
 *            preference order set by the number of 128 x 128 output tiles
 *            (>= 1024: 4-wavefront tiles with small LDS; >= 256: the
 *            8-wavefront 128 x 128 tile; fewer: 64 x 64 tiles whose
 *            wavefronts split the contraction).
 * Supported: any number of output rows, output columns a multiple of 4 and
 * a contraction length a multiple of 8 (else FBL_ERR_UNSUPPORTED) -- so
 * ragged token counts and LoRA ranks (8, 16, ...) as the narrow side or the
 * contraction.  Any tile runs any shape: partial tiles are masked, and the
 * contraction positions of a partial last step are zeroed before use.
 * Checks: non-NULL pointers, positive
 * extents, leading dimensions >= widths, 16-byte aligned pointers and rows,
 * each operand's span below 2 GiB, c not overlapping a or b.  The caller owns
 * all memory; enqueued on `stream`; c is fully overwritten.
 */
#define FBL_PROJ_FWD 0u
#define FBL_PROJ_BWD_DATA 1u
#define FBL_PROJ_BWD_WEIGHT 2u
#define FBL_GEMM_TILE_AUTO (-1)
#define FBL_GEMM_TILE_128x128 0
#define FBL_GEMM_TILE_128x64 1
#define FBL_GEMM_TILE_64x128 2
#define FBL_GEMM_TILE_64x64 3
fbl_status fbl_proj(uint32_t op, int64_t M, int64_t K, int64_t N, const void* a, int64_t lda, const void* b,
                    int64_t ldb, void* c, int64_t ldc, int32_t tile, void* stream);

/*
 * fbl_proj (the projection products of section 2.2's LoRA example) for either
 * storage type: dtype FBL_BF16 is fbl_proj exactly;
 * FBL_F32 runs the same three products on fp32 operands and result (fp32
 * MFMAs, fp32 accumulation) with one tile shape -- tile must be
 * FBL_GEMM_TILE_AUTO (else FBL_ERR_ARG) -- any extents and leading
 * dimensions, and 4-byte (natural) alignment; the other checks are
 * fbl_proj's.  FBL_ERR_DTYPE for another dtype.
 */
fbl_status fbl_proj_dt(uint32_t op, int32_t dtype, int64_t M, int64_t K, int64_t N, const void* a, int64_t lda,
                       const void* b, int64_t ldb, void* c, int64_t ldc, int32_t tile, void* stream);

/*
 * Tile configurations of the projection products (their R-Tile shapes,
 * section 4.2).  fbl_gemm_tile_count gives
 * the number of ids; fbl_gemm_tile_info writes 8 values for one id:
 *   info[0..1]  bm, bn   output tile rows x cols of one workgroup
 *   info[2]     bk       contraction elements staged per step
 *   info[3]     stages   LDS stages (stages - 1 steps in flight)
 *   info[4..6]  wm, wn, wk  wavefront grid: wm x wn wavefront tiles, each
 *               computed by wk wavefronts that split every step's contraction
 *   info[7]     LDS bytes of one workgroup
 * FBL_ERR_NULL / FBL_ERR_ARG for a NULL info or an id out of range.
 */
int32_t fbl_gemm_tile_count(void);
fbl_status fbl_gemm_tile_info(int32_t tile, int32_t* info);

/*
 * Candidate tiles of one product shape: the three progressive filters of the
 * R-Tile shape candidate generation (section 4.2, step 1, and the
 * supplementary algorithm), read for gfx950 --
 *   C1 compute alignment: wavefront tiles of whole 32x32 MFMA blocks, whole
 *      16-deep MFMA chunks per wavefront and step;
 *   C2 memory alignment: the workgroup's LDS fits the 160 KB of a CU and
 *      every staged row is a whole number of 128-byte cache lines or spans
 *      the operand's whole (narrower) stored row;
 *   C3 shape: padding the output rows, the output columns and the
 *      contraction to whole tiles adds at most 10% to each; if no tile
 *      qualifies, the C1/C2 survivors of least padded volume.
 * Writes up to `cap` ids in increasing order to `tiles` and the number of
 * candidates to *count (which may exceed cap).  Host only, no GPU work.
 */
fbl_status fbl_proj_candidates(uint32_t op, int64_t M, int64_t K, int64_t N, int32_t* tiles, int32_t cap,
                               int32_t* count);

/*
 * Measured tile selection for one product: every candidate of
 * fbl_proj_candidates runs once untimed and `reps` (1..1000) times timed with
 * HIP events on `stream`, on the caller's operands.  The choice maximises
 *   FBL_TUNE_TIME              1 / average time, or
 *   FBL_TUNE_GFLOPS_X_MEMEFF   GFLOP/s x MemEfficiency (section 4.2, the
 *                              unified R-Tile objective, per product): minimal
 *                              bytes (each operand and the result once) over
 *                              the bytes the tile schedule stages (each row
 *                              block of A once per output column block, each
 *                              column block of B once per output row block,
 *                              plus the result).
 * The choice is kept in a per-process table keyed by (op, M, K, N) that
 * FBL_GEMM_TILE_AUTO consults (thread-safe; fbl_proj_tune_reset clears it,
 * fbl_proj_tuned_tile reads it, -1 if absent).  ms (optional,
 * fbl_gemm_tile_count() floats) receives each id's average milliseconds, -1
 * for ids that are not candidates; *best (optional) the chosen id.  Blocks
 * until the timed launches finish.  On return c holds the product computed
 * with the chosen tile.  Same checks as fbl_proj; FBL_ERR_ARG for an unknown
 * objective or reps out of range, FBL_ERR_UNSUPPORTED with no candidate.
 */
#define FBL_TUNE_TIME 0u
#define FBL_TUNE_GFLOPS_X_MEMEFF 1u
fbl_status fbl_proj_tune(uint32_t op, int64_t M, int64_t K, int64_t N, const void* a, int64_t lda, const void* b,
                         int64_t ldb, void* c, int64_t ldc, uint32_t objective, int32_t reps, float* ms,
                         int32_t* best, void* stream);
int32_t fbl_proj_tuned_tile(uint32_t op, int64_t M, int64_t K, int64_t N);
void fbl_proj_tune_reset(void);

/*
 * The tile id FBL_GEMM_TILE_AUTO resolves to (section 4.2's selection) for a
 * bf16 product (op, M, K,
 * N): the tuned choice when the table holds one, else the untuned preference
 * among the candidates -- by the number of 128 x 128 output tiles and the
 * contraction length, measured on MI355X.  The untuned choice depends on the
 * shape only (not on leading dimensions or pointers).  Pure host function.
 * FBL_ERR_NULL, FBL_ERR_ARG (unknown op) or FBL_ERR_SHAPE on bad arguments.
 */
fbl_status fbl_proj_auto_tile(uint32_t op, int64_t M, int64_t K, int64_t N, int32_t* tile);

/* Static, human-readable name of a status code. */
const char* fbl_status_str(fbl_status s);

#ifdef __cplusplus
}
#endif

#endif /* FBL_H */
