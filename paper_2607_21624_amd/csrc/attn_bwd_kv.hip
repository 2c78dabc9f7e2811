// attn_bwd_kv.hip -- key/value-major backward pass for bf16 storage, gfx950.
//
// Computes dV = P^T dO and dK = scale dS^T Q (section 4.1, the reductions
// over queries: the M direction of section 4.2) for one workgroup of 128
// keys of one (batch, kv head), over the query blocks of every query head of
// the GQA group.  Each wavefront keeps its 32 K and V rows as MFMA operands
// and its dK^T, dV^T accumulators in registers for the whole pass.
//
// Per query block i the wavefront runs four products and an elementwise step:
//   S_i  = Q_i K_w^T,  dP_i = dO_i V_w^T        (row reads of the Q/dO tiles)
//   P_i  = exp2(S_i scale log2e - LSE_i log2e), dS_i = P_i (dP_i - D_i)
//   dV^T += dO_i^T P_i,  dK^T += Q_i^T dS_i      (transposed reads)
// At D = 128 there is one wavefront per SIMD (the accumulators take half the
// register file; at D = 64 two workgroups share a CU) and little else hides
// latency: every instruction the wavefront issues besides the products costs
// time, so the loop is software-pipelined by hand:
//   phase X(i): S/dP products of block i+1  |  elementwise step of block i
//   barrier; DMA of block i+3
//   phase Y(i): dV/dK products of block i   |  LDS reads of block i's
//               transposed operands and block i+2's row operands
// (with one wavefront per SIMD, only the first kRowLead of block i+2's row
// operands in phase Y(i) and the rest during phase X(i+1), which frees the
// registers for the S/dP accumulators of two blocks: see mma_vgpr)
// Operands are read a few product slots ahead of their use (kLead).  Four
// LDS buffers: while blocks i..i+2 are resident, block i+3 streams in by DMA
// (global -> LDS, no registers) a full iteration before it is first read.  The
// loop is unrolled over the four buffers so that every LDS address is a
// per-lane base plus an immediate.
//
// With DS set the pass also stores dS (bf16, the values its dK product
// consumes) block by block into the workspace, for the dQ pass to contract
// with K instead of recomputing S and dP.  A 32-query x 32-key block is 2 KB
// (blocks of one query head key-block major: block (qb32, kb32) at
// (kb32*nq32 + qb32)*1024, so one wavefront's stores stream through
// consecutive blocks) in the accumulator order the fragments already have:
// element
// cc*512 + lane*8 + e holds dS[query acc_row(8cc + e, lane / 32)][key lane % 32],
// so each store is one coalesced 1 KB row of the wavefront.  Entries of keys
// at or past kv_end are stored unmasked (the dQ pass masks them); blocks
// wholly above the causal diagonal, or whose keys all lie past kv_end, are not
// stored (the dQ pass never reads them).
#include <type_traits>

#include "attn_tiles.hpp"
#include "cdna4.hpp"
#include "kernels.hpp"
#include "stage.hpp"
#include "tokmap.hpp"

namespace fbl {

namespace {

// S/dP product in the vector-register form, starting the sum from zero when
// `first`.  Built-in MFMAs of a kernel that also needs accumulation registers
// all take the accumulator form, whose results the elementwise step would have
// to copy out (32 instructions per block); these are written out instead.
// The destination is early-clobber so that it never shares registers with A or
// B.  The compiler sees an opaque instruction: the wait states the hardware
// needs around it (operands written by a vector instruction at least 2
// instructions before; results read at least a product phase later) are
// checked on the generated code by tests/test_isa_hazards.py.
FBL_DEV void mma_vgpr(f32x16& acc, const Frag<bf16>& a, const Frag<bf16>& b, bool first) {
    if (first)
        asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(acc) : "v"(a.v), "v"(b.v));
    else
        asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(acc) : "v"(a.v), "v"(b.v));
}

// The LDS DMA of one kv block -- NPQ loads of 1 KB from each of the Q and dO
// tiles and one 256-byte load of the statistics row -- in one statement, so
// one set of wait states covers every scalar operand (a load issued on its
// own needs them each time: the compiler may reload a spilled scalar operand
// with a vector instruction just before it).  The LDS address of load i is
// lq + i * kq (Q), lq + TB + i * kq (dO) and lst (statistics).
template <int NPQ>
FBL_DEV void kv_block_dma(Rsrc rq, Rsrc ro, Rsrc rst, uint32_t sq, uint32_t so, uint32_t sst, uint32_t lq, uint32_t lo,
                          uint32_t lst, uint32_t kq, const uint32_t* vq, const uint32_t* vo, uint32_t vst) {
    static_assert(NPQ == 1 || NPQ == 2, "one or two loads per tile");
    if constexpr (NPQ == 2) {
        asm volatile(
            "s_nop 4\n\t"
            "s_mov_b32 m0, %5\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %10, %13 offen lds\n\t"
            "s_mov_b32 m0, %6\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %10, %13 offen lds\n\t"
            "s_mov_b32 m0, %7\n\ts_nop 0\n\tbuffer_load_dwordx4 %2, %11, %14 offen lds\n\t"
            "s_mov_b32 m0, %8\n\ts_nop 0\n\tbuffer_load_dwordx4 %3, %11, %14 offen lds\n\t"
            "s_mov_b32 m0, %9\n\ts_nop 0\n\tbuffer_load_dword %4, %12, %15 offen lds"
            :
            : "v"(vq[0]), "v"(vq[1]), "v"(vo[0]), "v"(vo[1]), "v"(vst), "s"(lq), "s"(lq + kq), "s"(lo), "s"(lo + kq),
              "s"(lst), "s"(rq), "s"(ro), "s"(rst), "s"(sq), "s"(so), "s"(sst)
            : "memory", "m0");
    } else {
        asm volatile(
            "s_nop 4\n\t"
            "s_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %6, %9 offen lds\n\t"
            "s_mov_b32 m0, %4\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %7, %10 offen lds\n\t"
            "s_mov_b32 m0, %5\n\ts_nop 0\n\tbuffer_load_dword %2, %8, %11 offen lds"
            :
            : "v"(vq[0]), "v"(vo[0]), "v"(vst), "s"(lq), "s"(lo), "s"(lst), "s"(rq), "s"(ro), "s"(rst), "s"(sq),
              "s"(so), "s"(sst)
            : "memory", "m0");
    }
}

constexpr int kLead = 4;              // product slots between an operand read and its use

// BQ_ queries per block (the staged Q/dO tile rows of the tile table), NW_
// wavefronts of 32 keys per workgroup.  At D = 64 with 32-query blocks the
// wavefront's state fits 256 registers, so two wavefronts share a SIMD.
// OCC workgroups per CU; WPS wavefronts per SIMD.
template <int D, int BQ_, int NW_>
struct KvPipe {
    static constexpr int BQ = BQ_;
    static constexpr int NW = NW_;
    static constexpr int WPS = (D == 64 && BQ == 32) ? 2 : 1;
    static constexpr int OCC = WPS * 4 / NW;
    static constexpr int NQT = BQ / 32;
    static constexpr int TB = BQ * D * 2;  // bytes of one bf16 Q or dO tile
    static constexpr int NBUF = 4;
    static constexpr int BUFB = 2 * TB;            // buffer: Q tile, dO tile
    // per buffer, the block's LSE*log2e and D rows (64 floats each: one dword
    // per lane of a 64-lane DMA; the first BQ are used)
    static constexpr int OFF_ST = NBUF * BUFB;
    static constexpr int STB = 512;
    static constexpr int SPARE = OFF_ST + NBUF * STB;  // sink of the statistics loads of waves 2, 3
    static constexpr int BYTES = SPARE + 256;
    static_assert(BUFB % 256 == 0, "tiles start on a 256-byte (all-bank) boundary");
    static_assert((NBUF - 1) * BUFB + TB + 2 * 16 * D + (NQT - 1) * 32 * D * 2 < 65536,
                  "buffer offsets fit the 16-bit LDS immediate");
    static_assert(BYTES <= 160 * 1024, "LDS of one workgroup");
};

template <int D, int BQ_, int NW_, bool DS>
__global__ __launch_bounds__(64 * NW_, (KvPipe<D, BQ_, NW_>::WPS)) void attn_bwd_kv_bf16(BwdArgs a) {
    using P = KvPipe<D, BQ_, NW_>;
    constexpr int kPWaves = NW_;
    constexpr int kPKeys = 32 * kPWaves;  // keys per workgroup
    constexpr int NC = D / 16;
    constexpr int ND = D / 32;
    constexpr int BQ = P::BQ;
    constexpr int NQT = P::NQT;
    constexpr int TB = P::TB;
    constexpr int BUFB = P::BUFB;
    extern __shared__ __attribute__((aligned(1024))) unsigned char kvp_smem[];
    const uint32_t lds = lds_addr(kvp_smem);

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = lane >> 5;
    const int c32 = lane & 31;
    const int S = a.S, Skv = a.Skv;  // query tokens, key tokens
    const int nkb = (Skv + kPKeys - 1) / kPKeys;
    int rank, bh;  // causal: key block 0 meets the most queries; start it first
    if (!rank_major_item(blockIdx.x, nkb * a.kv_split, a.Hkv * a.B, rank, bh)) return;
    const int kblk = rank / a.kv_split, split = rank % a.kv_split;
    const int hk = bh % a.Hkv;
    const int b = bh / a.Hkv;
    const int G_ = a.Hq / a.Hkv;
    int kv_end = Skv;
    if (a.mask.kv_len) kv_end = min(max(a.mask.kv_len[b], 0), Skv);
    const int k0 = kblk * kPKeys;
    const int kw0 = k0 + wave * 32;  // first key of this wave
    const int key = kw0 + c32;       // this lane's key (column of S)

    // K and V rows of this wave's keys as B operands: lane <-> key, in-lane d = 16c + 8g + e
    Frag<bf16> kf[NC], vf[NC];
    {
        const bf16* kp = static_cast<const bf16*>(a.k) + a.mk.head_base(b, hk) + (int64_t)key * a.mk.ss + 8 * g;
        const bf16* vp = static_cast<const bf16*>(a.v) + a.mv.head_base(b, hk) + (int64_t)key * a.mv.ss + 8 * g;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            kf[c].v = bf16x8{};
            vf[c].v = bf16x8{};
            if (key < Skv) {
                kf[c].v = __builtin_bit_cast(bf16x8, load16(kp + 16 * c));
                vf[c].v = __builtin_bit_cast(bf16x8, load16(vp + 16 * c));
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
    // this workgroup's share of the key block's iterations (G_ heads x
    // per_head query blocks, head-major): [it_lo, it_hi) of split `split`
    const int n_all = (k0 < kv_end) ? G_ * per_head : 0;
    const int it_lo = (int)((int64_t)n_all * split / a.kv_split);
    const int n_iter = (int)((int64_t)n_all * (split + 1) / a.kv_split) - it_lo;
    const int h_lo = n_iter > 0 ? it_lo / per_head : 0;  // query head (within the group) of the first
    const int j_lo = n_iter > 0 ? it_lo % per_head : 0;  // and its block index within that head
    // Blocks of each head whose scores need the causal mask: those holding a
    // query before one of the workgroup's keys.  Keys at or past kv_end need no
    // mask: a key's P and dS only reach that key's own dK and dV rows, which are
    // stored as zeros.
    const int n_mask = a.mask.causal ? min(per_head, (k0 + kPKeys - 2) / BQ - qb_start + 1) : 0;

    // dS blocks of this wave's 32 keys (DS only): block (qb32, kb32) of query
    // head h starts at element ((b*Hq + h)*nk32 + kb32)*nq32*1024 + qb32*1024;
    // one buffer resource per query head, the block offset in the scalar
    // offset of the stores, which are non-temporal (read once, by the dQ
    // pass; they should not displace the Q/dO tiles other workgroups reuse).
    const int kb32 = kw0 / 32;
    const bool ds_live = DS && kw0 < kv_end;  // keys past kv_end: never read
    const uint32_t ds_head_elems = (uint32_t)a.nq32 * (uint32_t)a.nk32 * 1024u;
    const bf16* ds_head =
        DS ? static_cast<const bf16*>(a.ds) + ((int64_t)b * a.Hq + hk * G_ + h_lo) * ds_head_elems : nullptr;
    __amdgpu_buffer_rsrc_t ds_rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(ds_head), 0,
                                                                     (int)(ds_head_elems * 2u), 0x00020000);

    // ---- DMA of the Q, dO tiles and the row statistics of one block
    const uint32_t qbytes = (uint32_t)(a.mq.ss * 2), obytes = (uint32_t)(a.mdo.ss * 2);
    const uint32_t qspan = (uint32_t)((int64_t)(S - 1) * a.mq.ss * 2 + D * 2);
    const uint32_t ospan = (uint32_t)((int64_t)(S - 1) * a.mdo.ss * 2 + D * 2);
    DmaPlan<bf16, D, BQ, kPWaves> pq, po;
    pq.init(qbytes, wave, lane);
    po.init(obytes, wave, lane);
    const bf16* q_head = static_cast<const bf16*>(a.q) + a.mq.head_base(b, hk * G_ + h_lo);
    const bf16* o_head = static_cast<const bf16*>(a.dout) + a.mdo.head_base(b, hk * G_ + h_lo);
    // wave 0 loads the LSE*log2e row, wave 1 the D row, waves 2 and 3 nothing
    // (no records) into a spare slot
    const float* st_head = a.stats + (2 * ((int64_t)b * a.Hq + hk * G_ + h_lo) + (wave & 1)) * S;
    const uint32_t st_bytes = wave < 2 ? (uint32_t)S * 4u : 0u;
    const uint32_t st_lds0 = wave < 2 ? lds + P::OFF_ST + wave * 256 : lds + P::SPARE;
    const uint32_t st_step = wave < 2 ? P::STB : 0;
    Rsrc rq = make_rsrc(q_head, qspan), ro = make_rsrc(o_head, ospan), rst = make_rsrc(st_head, st_bytes);
    uint32_t dma_q0 = (uint32_t)((qb_start + j_lo) * BQ);  // first query of the next block to stage
    int dma_j = j_lo;                                      // its index within its head
    // A block is staged in NPART loads per wave (Q tile, dO tile, statistics
    // row).
    constexpr int NPQ = DmaPlan<bf16, D, BQ, kPWaves>::PER_WAVE;
    static_assert(DmaPlan<bf16, D, BQ, kPWaves>::INSTS % kPWaves == 0, "whole loads per wave");
    constexpr int NPART = 2 * NPQ + 1;
    auto issue_part = [&](auto buf_c, int part) {
        constexpr int BB = decltype(buf_c)::value;
        if (part < NPQ)
            dma16(rq, lds + BB * BUFB + (part * kPWaves + wave) * 1024, pq.voff[part], dma_q0 * qbytes);
        else if (part < 2 * NPQ)
            dma16(ro, lds + BB * BUFB + TB + ((part - NPQ) * kPWaves + wave) * 1024, po.voff[part - NPQ],
                  dma_q0 * obytes);
        else
            dma4(rst, st_lds0 + BB * st_step, (uint32_t)lane * 4u, dma_q0 * 4u);
    };
    auto advance_dma = [&]() {
        dma_q0 += BQ;
        if (++dma_j == per_head) {  // next query head of the group
            dma_j = 0;
            dma_q0 = (uint32_t)(qb_start * BQ);
            q_head += a.mq.sh;
            o_head += a.mdo.sh;
            st_head += 2 * S;
            rq = make_rsrc(q_head, qspan);
            ro = make_rsrc(o_head, ospan);
            rst = make_rsrc(st_head, st_bytes);
        }
    };
    auto issue_all = [&](auto buf_c) {
        constexpr int BB = decltype(buf_c)::value;
        if constexpr (NPQ <= 2) {
            const uint32_t lq = lds + BB * BUFB + wave * 1024;
            kv_block_dma<NPQ>(rq, ro, rst, dma_q0 * qbytes, dma_q0 * obytes, dma_q0 * 4u, lq, lq + TB,
                              st_lds0 + BB * st_step, kPWaves * 1024, pq.voff, po.voff, (uint32_t)lane * 4u);
        } else {
#pragma unroll
            for (int part = 0; part < NPART; ++part) issue_part(buf_c, part);
        }
    };
    auto issue = [&](auto buf_c) {
        issue_all(buf_c);
        advance_dma();
    };
    // (measured: spreading the loads over the products of phase Y, or moving
    // the accumulator reads there, is slower -- with one wavefront per SIMD
    // every non-product instruction costs issue time wherever it sits)

    // ---- per-lane LDS addresses of buffer 0; buffers are reached by immediates
    LaneOffsets<D> lo;
    lo.init(lds, lane);
    const uint32_t st_a = lds + P::OFF_ST + 16u * g;  // LSE of queries 4g.. (D at +256)

    // S/dP products of a block: product k is S (k even) or dP (k odd) of query
    // tile qt = k / (2 NC) over d-chunk c = (k / 2) % NC; its A operand is one
    // row fragment of the Q or dO tile.
    constexpr int NSDP = 2 * NQT * NC;
    // With one wavefront per SIMD (D = 128 with 32-query blocks, D = 64 with
    // 64-query blocks) the S and dP products run in the vector-register form
    // (mma_vgpr) into two accumulator sets, one per block parity, which the
    // elementwise step reads in place; the registers that takes come from
    // reading only a block's first kRowLead row operands in phase Y and the rest
    // during the previous phase X, kRowLead product slots ahead of their use.
    constexpr bool kVgprSdp = (D == 128 && NQT == 1) || (D == 64 && NQT == 2);
    constexpr int kRowLead = kVgprSdp ? (D == 128 ? 12 : 4) : NSDP;  // row operands of a block read in phase Y
    Frag<bf16> fa[NSDP];
    auto read_row = [&](auto buf_c, int k) {
        constexpr int BB = decltype(buf_c)::value;
        const int qt = k / (2 * NC), c = (k / 2) % NC;
        fa[k].v = lds_b128(lo.row[c], BB * BUFB + (k % 2 ? TB : 0) + qt * 32 * D * 2);
    };
    // S and dP accumulators of the block whose products are in flight: lane <->
    // key, in-lane query 32qt + acc_row.  With one set, at the start of each
    // phase X their values move to vector registers (the elementwise step reads
    // them there) and the accumulators start the next block; with two, block
    // it uses set it % 2.
    constexpr int NSET = kVgprSdp ? 2 : 1;
    f32x16 s_acc[NSET][NQT], dp_acc[NSET][NQT];  // [block parity when kVgprSdp]
    auto sdp_one = [&](auto set_c, int k) {
        constexpr int PS = decltype(set_c)::value;
        const int qt = k / (2 * NC), c = (k / 2) % NC;
        if constexpr (kVgprSdp) {
            if (k % 2 == 0) mma_vgpr(s_acc[PS][qt], fa[k], kf[c], c == 0);
            else mma_vgpr(dp_acc[PS][qt], fa[k], vf[c], c == 0);
        } else if (k % 2 == 0) {
            if (c == 0) s_acc[PS][qt] = f32x16{};
            mma(s_acc[PS][qt], fa[k], kf[c]);
        } else {
            if (c == 0) dp_acc[PS][qt] = f32x16{};
            mma(dp_acc[PS][qt], fa[k], vf[c]);
        }
    };
    // dV/dK products of a block: product m is dV^T += dO^T P (m even) or
    // dK^T += Q^T dS (m odd) for d-tile t = (m / 2) % ND over the 16 queries of
    // chunk cc = (m / (2 ND)) % 2 of query tile qt = m / (4 ND); its A operand is
    // two transposed reads.
    constexpr int NCM = NQT * 2 * ND * 2;
    static_assert(NCM == NSDP, "one row read per dV/dK product slot");
    bf16x4 trv[2 * NCM];
    auto read_tr = [&](auto buf_c, int m) {
        constexpr int BB = decltype(buf_c)::value;
        const int qt = m / (4 * ND), cc = (m / (2 * ND)) % 2, t = (m / 2) % ND;
        const uint32_t off = BB * BUFB + (qt * 32 + 16 * cc) * D * 2 + (m % 2 ? 0 : TB);
        trv[2 * m] = lds_tr(lo.tr[t][0], off);
        trv[2 * m + 1] = lds_tr(lo.tr[t][1], off);
    };
    // row statistics (LSE*log2e, D) of a block: per lane, its 16 query rows per tile
    constexpr int NST = 2 * NQT * 4;
    f32x4 st[NST];  // index (qt * 4 + rr) * 2 + {0: LSE, 1: D}
    auto read_st = [&](auto buf_c, int i) {
        constexpr int BB = decltype(buf_c)::value;
        const int qt = i / 8, rr = (i / 2) % 4;
        st[i] = *(const FBL_LDS f32x4*)(uintptr_t)(st_a + BB * P::STB + (i % 2) * 256 + (qt * 32 + 8 * rr) * 4);
    };

    // Elementwise work of phase X spread over its product slots: slot k takes
    // elements [el0(k), el0(k+1)); the first two slots take none (the
    // statistics reads are landing).
    constexpr int NEL = 16 * NQT;
    auto el0 = [](int k) { return k < 2 ? 0 : (k - 2) * NEL / (NSDP - 2); };

    // One iteration on block `it`, held in buffer B; j is its index within its
    // head's blocks.
    auto step = [&](auto buf_c, int it, int j) {
        constexpr int B = decltype(buf_c)::value;
        using B2 = std::integral_constant<int, (B + 2) % 4>;
        using B3 = std::integral_constant<int, (B + 3) % 4>;
        using B1 = std::integral_constant<int, (B + 1) % 4>;
        constexpr int PC = kVgprSdp ? B % 2 : 0;  // accumulator set of block it
        using PN = std::integral_constant<int, kVgprSdp ? 1 - PC : 0>;  // ... and of block it+1
        // ---------------- phase X
        __builtin_amdgcn_sched_barrier(0);
        float sv[NEL], dpv[NEL];  // S and dP of block it, out of the accumulators
#pragma unroll
        for (int e = 0; e < NEL; ++e) {
            sv[e] = s_acc[PC][e / 16][e % 16];
            dpv[e] = dp_acc[PC][e / 16][e % 16];
            if constexpr (!kVgprSdp) asm volatile("" : "+v"(sv[e]), "+v"(dpv[e]));
        }
        // row statistics of block it (the first element needs them two slots later)
#pragma unroll
        for (int i = 0; i < NST; ++i) read_st(buf_c, i);
        float pv[NEL], dsv[NEL];
        Frag<bf16> pb[NQT][2], dsb[NQT][2];
#pragma unroll
        for (int k = 0; k < NSDP; ++k) {
            // product k of block it+1 (stale operands past the last block: unused)
            sdp_one(PN{}, k);
            // row operands of block it+1 not read in phase Y, kRowLead slots ahead of their product
            if (k + kRowLead < NSDP) read_row(B1{}, k + kRowLead);
            // the first transposed operands of phase Y
            if (k >= NSDP - kLead) read_tr(buf_c, k - (NSDP - kLead));
#pragma unroll
            for (int e = el0(k); e < el0(k + 1); ++e) {
                const int qt = e / 16, r = e % 16, i = (qt * 4 + r / 4) * 2;
                float p = fast_exp2(__builtin_fmaf(sv[e], a.scale_log2, -st[i][r % 4]));
                float ds = p * (dpv[e] - st[i + 1][r % 4]);
                // pin: keeps this element's arithmetic in its slot (pure
                // arithmetic is otherwise free to drift towards its uses)
                asm volatile("" : "+v"(p), "+v"(ds));
                pv[e] = p;
                dsv[e] = ds;
                if (e % 8 == 7) {
                    pack_frag(pb[qt][r / 8], pv + e - 7);
                    pack_frag(dsb[qt][r / 8], dsv + e - 7);
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        // causal mask on the diagonal blocks, applied to the packed P and dS:
        // query row acc_row(r, 0) + 4g of tile qt (first query q0 + 32 qt) is
        // kept iff it does not precede the lane's key.  Bitwise, so that a
        // masked element's value (which may be inf) does not matter.
        if (j < n_mask) {
            const int q0 = (qb_start + j) * BQ;
#pragma unroll
            for (int qt = 0; qt < NQT; ++qt) {
                const int thr = key - 4 * g - (q0 + 32 * qt);  // keep iff acc_row(r, 0) >= thr
#pragma unroll
                for (int cc = 0; cc < 2; ++cc) {
                    uint32_t w[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int r = 8 * cc + 2 * u;
                        w[u] = (acc_row(r, 0) >= thr ? 0x0000ffffu : 0u) | (acc_row(r + 1, 0) >= thr ? 0xffff0000u : 0u);
                    }
                    using u32x4 = uint32_t __attribute__((ext_vector_type(4)));
                    const u32x4 wm = u32x4{w[0], w[1], w[2], w[3]};
                    pb[qt][cc].v = __builtin_bit_cast(bf16x8, __builtin_bit_cast(u32x4, pb[qt][cc].v) & wm);
                    dsb[qt][cc].v = __builtin_bit_cast(bf16x8, __builtin_bit_cast(u32x4, dsb[qt][cc].v) & wm);
                }
            }
        }
        // ---------------- block it+2 landed in every wave; block it-1's buffer is free
        wait_vmcnt<0>();
        __syncthreads();
        const bool stage = it + 3 < n_iter;  // block it+3 exists
        if (stage) issue_all(B3{});
        // dS of block it to the workspace; the stores retire during phase Y
        // and X(it+1), before the next vmcnt wait
        if constexpr (DS) {
            if (ds_live) {
#pragma unroll
                for (int qt = 0; qt < NQT; ++qt) {
                    const int qb32 = (qb_start + j) * NQT + qt;
                    if (qb32 < a.nq32 && (!a.mask.causal || qb32 >= kb32)) {
                        const int soff = (kb32 * a.nq32 + qb32) * 2048;
#pragma unroll
                        for (int cc = 0; cc < 2; ++cc) {
                            using i32x4 = int __attribute__((ext_vector_type(4)));
                            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, dsb[qt][cc].v), ds_rs,
                                                                   lane * 16 + cc * 1024, soff, 2 /* nt */);
                        }
                    }
                }
            }
        }
        __builtin_amdgcn_sched_barrier(0);
        // ---------------- phase Y
#pragma unroll
        for (int m = 0; m < NCM; ++m) {
            Frag<bf16> f;
            f.v = bf16x8{trv[2 * m][0], trv[2 * m][1], trv[2 * m][2], trv[2 * m][3],
                         trv[2 * m + 1][0], trv[2 * m + 1][1], trv[2 * m + 1][2], trv[2 * m + 1][3]};
            const int qt = m / (4 * ND), cc = (m / (2 * ND)) % 2, t = (m / 2) % ND;
            if (m % 2 == 0) mma(dv[t], f, pb[qt][cc]);
            else mma(dk[t], f, dsb[qt][cc]);
            if (m + kLead < NCM) read_tr(buf_c, m + kLead);
            // the first kRowLead row operands of block it+2, for phase X(it+1) (stale past the last block: unused)
            if (m >= NCM - kRowLead) read_row(B2{}, m - (NCM - kRowLead));
            // DMA of block it+3 into the buffer of block it-1
            __builtin_amdgcn_sched_barrier(0);
        }
        if (stage) advance_dma();
    };

    using C0 = std::integral_constant<int, 0>;
    using C1 = std::integral_constant<int, 1>;
    using C2 = std::integral_constant<int, 2>;
    using C3 = std::integral_constant<int, 3>;
    if (n_iter > 0) {
        issue(C0{});
        if (n_iter > 1) issue(C1{});
        if (n_iter > 2) issue(C2{});
        wait_vmcnt<0>();
        __syncthreads();
#pragma unroll
        for (int k = 0; k < NSDP; ++k) read_row(C0{}, k);
#pragma unroll
        for (int k = 0; k < NSDP; ++k) sdp_one(std::integral_constant<int, 0>{}, k);
#pragma unroll
        for (int k = 0; k < kRowLead; ++k) read_row(C1{}, k);  // stale when there is no block 1
    }
    // Blocks in order, four per trip (one per LDS buffer).
    int j = j_lo;  // index of block `it` within its head's blocks
    auto next_j = [&]() {
        if (++j == per_head) {
            j = 0;
            if constexpr (DS) {  // the next query head's dS blocks
                ds_head += ds_head_elems;
                ds_rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(ds_head), 0, (int)(ds_head_elems * 2u),
                                                          0x00020000);
            }
        }
    };
    for (int it = 0; it < n_iter; it += 4) {
        step(C0{}, it, j);
        next_j();
        if (it + 1 < n_iter) {
            step(C1{}, it + 1, j);
            next_j();
        }
        if (it + 2 < n_iter) {
            step(C2{}, it + 2, j);
            next_j();
        }
        if (it + 3 < n_iter) {
            step(C3{}, it + 3, j);
            next_j();
        }
    }

    // dK (times scale) and dV rows of this wave's keys: lane <-> key, 4
    // consecutive d per store.  Keys at or past kv_end take no part: their
    // accumulators hold unmasked (possibly non-finite) sums and are replaced
    // by zeros.
    if (key < Skv && a.kv_split > 1) {
        // fp32 partial sums of this split (zeros past kv_end)
        const bool live = key < kv_end;
        const int64_t plane = (int64_t)a.B * Skv * a.Hkv * D;
        float* pk = a.dkv_part + (int64_t)split * plane + (((int64_t)b * Skv + key) * a.Hkv + hk) * D;
        float* pv = pk + (int64_t)a.kv_split * plane;
#pragma unroll
        for (int t = 0; t < ND; ++t) {
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
                const int dcol = 32 * t + 8 * rr + 4 * g;
                float k4[4], v4[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    k4[e] = live ? dk[t][4 * rr + e] * a.scale : 0.f;
                    v4[e] = live ? dv[t][4 * rr + e] : 0.f;
                }
                store4(pk + dcol, k4[0], k4[1], k4[2], k4[3]);
                store4(pv + dcol, v4[0], v4[1], v4[2], v4[3]);
            }
        }
    } else if (key < Skv) {
        const bool live = key < kv_end;
        bf16* dkrow = static_cast<bf16*>(a.dk) + a.mdk.head_base(b, hk) + (int64_t)key * a.mdk.ss;
        bf16* dvrow = static_cast<bf16*>(a.dv) + a.mdv.head_base(b, hk) + (int64_t)key * a.mdv.ss;
#pragma unroll
        for (int t = 0; t < ND; ++t) {
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
                const int dcol = 32 * t + 8 * rr + 4 * g;
                float k4[4], v4[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    k4[e] = live ? dk[t][4 * rr + e] * a.scale : 0.f;
                    v4[e] = live ? dv[t][4 * rr + e] : 0.f;
                }
                store4(dkrow + dcol, k4[0], k4[1], k4[2], k4[3]);
                store4(dvrow + dcol, v4[0], v4[1], v4[2], v4[3]);
            }
        }
    }
}


// dK and dV of a split key/value pass: the kv_split partial sums of each
// element added in split order (deterministic), rounded once to bf16.  One
// thread per 4 consecutive d of one (b, key, kv head) row; dK rows first.
template <int D>
__global__ __launch_bounds__(256) void attn_bwd_kv_reduce(BwdArgs a) {
    constexpr int C4 = D / 4;
    const int64_t rows = (int64_t)a.B * a.Skv * a.Hkv;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= 2 * rows * C4) return;
    const bool is_v = i >= rows * C4;
    const int64_t r = is_v ? i - rows * C4 : i;
    const int c4 = (int)(r % C4);
    const int64_t row = r / C4;  // (b * Skv + key) * Hkv + hk
    const int hk = (int)(row % a.Hkv);
    const int key = (int)((row / a.Hkv) % a.Skv);
    const int b = (int)(row / ((int64_t)a.Hkv * a.Skv));
    const int64_t plane = rows * D;
    const float* src = a.dkv_part + (is_v ? (int64_t)a.kv_split * plane : 0) + row * D + 4 * c4;
    f32x4 acc = *reinterpret_cast<const f32x4*>(src);
    for (int s = 1; s < a.kv_split; ++s) acc += *reinterpret_cast<const f32x4*>(src + s * plane);
    const TokMap& m = is_v ? a.mdv : a.mdk;
    bf16* dst = static_cast<bf16*>(is_v ? a.dv : a.dk) + m.head_base(b, hk) + (int64_t)key * m.ss + 4 * c4;
    store4(dst, acc[0], acc[1], acc[2], acc[3]);
}

template <int D, int BQ, int NW, bool DS>
hipError_t launch_kv(const BwdArgs& a, hipStream_t stream) {
    using P = KvPipe<D, BQ, NW>;
    const hipError_t once = ensure_dynamic_lds<&attn_bwd_kv_bf16<D, BQ, NW, DS>>(P::BYTES);
    if (once != hipSuccess) return once;
    constexpr int lds = P::BYTES;
    const int nkb = (a.Skv + 32 * NW - 1) / (32 * NW);
    hipLaunchKernelGGL((attn_bwd_kv_bf16<D, BQ, NW, DS>), dim3(rank_major_grid(nkb * a.kv_split, a.Hkv * a.B)),
                       dim3(64 * NW), lds, stream, a);
    if (a.kv_split > 1) {
        const int64_t n = 2 * (int64_t)a.B * a.Skv * a.Hkv * (D / 4);
        hipLaunchKernelGGL((attn_bwd_kv_reduce<D>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace

// One tile of the table: its query block (the staged Q/dO rows); the split
// is the launch's a.kv_split.
template <int D, int TILE>
hipError_t launch_kv_tile(const BwdArgs& a, hipStream_t stream) {
    constexpr AttnTile t = kAttnTiles[TILE];
    static_assert(t.pass == kAttnKv && t.per_wave == 32 && t.bufs == 4, "a kv-pass tile");
    if constexpr (!attn_c1(t, D) || !attn_c2(t, D)) {
        return hipErrorInvalidValue;  // not built at this head dim (the filters exclude it)
    } else {
        using P = KvPipe<D, t.cols, t.waves>;
        static_assert(P::BYTES == attn_lds_bytes(t, D) && P::OCC == attn_occ(t, D),
                      "the kernel's LDS layout and occupancy are the tile table's");
        return a.ds ? launch_kv<D, t.cols, t.waves, true>(a, stream) : launch_kv<D, t.cols, t.waves, false>(a, stream);
    }
}

template <int D>
hipError_t launch_attn_bwd_kv_bf16(const BwdArgs& a, int tile, hipStream_t stream) {
    switch (tile) {
        case 5: return launch_kv_tile<D, 5>(a, stream);
        case 6: return launch_kv_tile<D, 6>(a, stream);
        case 10: return launch_kv_tile<D, 10>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

template hipError_t launch_attn_bwd_kv_bf16<32>(const BwdArgs&, int, hipStream_t);
template hipError_t launch_attn_bwd_kv_bf16<64>(const BwdArgs&, int, hipStream_t);
template hipError_t launch_attn_bwd_kv_bf16<128>(const BwdArgs&, int, hipStream_t);

}  // namespace fbl
