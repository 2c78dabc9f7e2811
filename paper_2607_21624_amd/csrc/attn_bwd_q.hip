// attn_bwd_q.hip -- query-major backward pass (dQ) for bf16 storage, gfx950.
//
// dQ = scale dS K (section 4.1; the reduction over keys, the N direction of
// section 4.2) for one workgroup of 128 queries of one (batch, query head);
// each wavefront owns 32 queries and keeps their Q and dO rows (as MFMA
// operands), their LSE and D and its dQ^T accumulator in registers, and walks
// the key blocks, recomputing S and dP (the key/value-major pass cannot sum
// over keys without atomics):
//   S^T_i = K_i Q^T,  dP^T_i = V_i dO^T          (row reads of the K/V tiles)
//   dS^T = P^T (dP^T - D),  P^T = exp2(S^T scale log2e - LSE log2e)
//   dQ^T += K_i^T dS^T                          (transposed reads of K)
// Scheduled like the key/value-major pass (one wavefront per SIMD, the loop
// pipelined by hand):
//   phase X(i): S/dP products of block i+1  |  elementwise step of block i
//   barrier; DMA of block i+3
//   phase Y(i): dQ products of block i      |  LDS reads of block i's
//               transposed operands and block i+2's row operands
// with four LDS buffers reached by immediate offsets (loop unrolled over
// them) and operands read a few product slots ahead of their use.
#include <type_traits>

#include "cdna4.hpp"
#include "kernels.hpp"
#include "stage.hpp"
#include "tokmap.hpp"

namespace fbl {

namespace {

constexpr int kQWaves = 4;
constexpr int kQRows = 32 * kQWaves;  // queries per workgroup
constexpr int kQLead = 4;             // product slots between an operand read and its use

template <int D>
struct QPipe {
    static constexpr int BK = D == 128 ? 32 : 64;  // keys per block
    static constexpr int NKT = BK / 32;
    static constexpr int TB = BK * D * 2;  // bytes of one bf16 K or V tile
    static constexpr int NBUF = 4;
    static constexpr int BUFB = 2 * TB;  // buffer: K tile, V tile
    static constexpr int BYTES = NBUF * BUFB;
    static_assert(BUFB % 256 == 0, "tiles start on a 256-byte (all-bank) boundary");
    static_assert((NBUF - 1) * BUFB + TB + (BK - 16) * D * 2 < 65536, "buffer offsets fit the 16-bit LDS immediate");
};

template <int D>
__global__ __launch_bounds__(256, 1) void attn_bwd_q_bf16(BwdArgs a) {
    using P = QPipe<D>;
    constexpr int NC = D / 16;
    constexpr int ND = D / 32;
    constexpr int BK = P::BK;
    constexpr int NKT = P::NKT;
    constexpr int TB = P::TB;
    constexpr int BUFB = P::BUFB;
    constexpr int NB = P::NBUF;
    extern __shared__ __attribute__((aligned(1024))) unsigned char qp_smem[];
    const uint32_t lds = lds_addr(qp_smem);

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = lane >> 5;
    const int c32 = lane & 31;
    const int S = a.S;
    const int nqb = (S + kQRows - 1) / kQRows;
    int rank, bh;
    if (!rank_major_item(blockIdx.x, nqb, a.Hq * a.B, rank, bh)) return;
    const int h = bh % a.Hq;
    const int b = bh / a.Hq;
    // causal: the last query blocks see the most keys; start them first
    const int qb = a.mask.causal ? (nqb - 1 - rank) : rank;
    const int hk = h / (a.Hq / a.Hkv);
    const int Skv = a.Skv;  // key tokens
    int kv_end = Skv;
    if (a.mask.kv_len) kv_end = min(max(a.mask.kv_len[b], 0), Skv);
    const int q0 = qb * kQRows;
    const int qi = q0 + wave * 32 + c32;  // this lane's query (column of S^T)
    int k_hi = kv_end;
    if (a.mask.causal) k_hi = min(k_hi, q0 + kQRows);
    const int n_iter = (k_hi + BK - 1) / BK;
    // blocks every query of the workgroup sees whole: inside kv_end and (causal)
    // at or below the workgroup's first query
    const int n_full = min(n_iter, min(kv_end, a.mask.causal ? q0 + 1 : Skv) / BK);

    // Q^T and dO^T rows of this wave's queries as B operands: lane <-> query,
    // in-lane d = 16c + 8g + e
    Frag<bf16> qf[NC], of[NC];
    {
        const bf16* qrow = static_cast<const bf16*>(a.q) + a.mq.head_base(b, h) + (int64_t)qi * a.mq.ss + 8 * g;
        const bf16* orow = static_cast<const bf16*>(a.dout) + a.mdo.head_base(b, h) + (int64_t)qi * a.mdo.ss + 8 * g;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            qf[c].v = bf16x8{};
            of[c].v = bf16x8{};
            if (qi < S) {
                qf[c].v = __builtin_bit_cast(bf16x8, load16(qrow + 16 * c));
                of[c].v = __builtin_bit_cast(bf16x8, load16(orow + 16 * c));
            }
        }
    }
    float lse2 = INFINITY, drow = 0.f;  // this lane's query row statistics
    if (qi < S) {
        const int64_t bh = (int64_t)b * a.Hq + h;
        lse2 = a.stats[2 * bh * S + qi];
        drow = a.stats[(2 * bh + 1) * S + qi];
    }
    // dQ^T: accumulator rows = d (32t + acc_row), columns = queries (lane)
    f32x16 dq[ND];
#pragma unroll
    for (int t = 0; t < ND; ++t) dq[t] = f32x16{};

    // ---- DMA of the K and V tiles of one block
    const uint32_t kbytes = (uint32_t)(a.mk.ss * 2), vbytes = (uint32_t)(a.mv.ss * 2);
    const Rsrc rk = make_rsrc(static_cast<const bf16*>(a.k) + a.mk.head_base(b, hk),
                              (uint32_t)((int64_t)(Skv - 1) * a.mk.ss * 2 + D * 2));
    const Rsrc rv = make_rsrc(static_cast<const bf16*>(a.v) + a.mv.head_base(b, hk),
                              (uint32_t)((int64_t)(Skv - 1) * a.mv.ss * 2 + D * 2));
    DmaPlan<bf16, D, BK, kQWaves> pk, pv;
    pk.init(kbytes, wave, lane);
    pv.init(vbytes, wave, lane);
    auto issue = [&](auto buf_c, int blk) __attribute__((always_inline)) {
        constexpr int BB = decltype(buf_c)::value;
        const uint32_t k0 = (uint32_t)(blk * BK);
        pk.issue(lds + BB * BUFB, rk, k0 * kbytes, wave);
        pv.issue(lds + BB * BUFB + TB, rv, k0 * vbytes, wave);
    };

    // ---- per-lane LDS addresses of buffer 0; buffers are reached by immediates
    LaneOffsets<D> lo;
    lo.init(lds, lane);

    // S/dP products of a block: product k is S^T (k even) or dP^T (k odd) of key
    // half kt = k / (2 NC) over d-chunk c = (k / 2) % NC; its A operand is one row
    // fragment of the K or V tile.
    constexpr int NSDP = 2 * NKT * NC;
    Frag<bf16> fa[NSDP];
    auto read_row = [&](auto buf_c, int k) __attribute__((always_inline)) {
        constexpr int BB = decltype(buf_c)::value;
        const int kt = k / (2 * NC), c = (k / 2) % NC;
        fa[k].v = lds_b128(lo.row[c], BB * BUFB + (k % 2 ? TB : 0) + kt * 32 * D * 2);
    };
    f32x16 s_acc[NKT], dp_acc[NKT];  // S^T and dP^T of the block in flight: lane <-> query
    auto sdp_one = [&](int k) __attribute__((always_inline)) {
        const int kt = k / (2 * NC), c = (k / 2) % NC;
        if (k % 2 == 0) {
            if (c == 0) s_acc[kt] = f32x16{};
            mma(s_acc[kt], fa[k], qf[c]);
        } else {
            if (c == 0) dp_acc[kt] = f32x16{};
            mma(dp_acc[kt], fa[k], of[c]);
        }
    };
    // dQ products of a block: product m accumulates d-block t = m % ND over the
    // 16 keys of chunk cc = (m / ND) % 2 of half kt = m / (2 ND); its A operand is
    // two transposed reads of the K tile.
    constexpr int NDQ = NKT * 2 * ND;
    bf16x4 trv[2 * NDQ];
    auto read_tr = [&](auto buf_c, int m) __attribute__((always_inline)) {
        constexpr int BB = decltype(buf_c)::value;
        const int t = m % ND, cc = (m / ND) % 2, kt = m / (2 * ND);
        const uint32_t off = BB * BUFB + (kt * 32 + 16 * cc) * D * 2;
        trv[2 * m] = lds_tr(lo.tr[t][0], off);
        trv[2 * m + 1] = lds_tr(lo.tr[t][1], off);
    };

    // Elementwise work of phase X spread over its product slots: slot k takes
    // elements [el0(k), el0(k+1)).
    constexpr int NEL = 16 * NKT;
    auto el0 = [](int k) { return k * NEL / NSDP; };
    // Row reads of phase Y spread over its dQ products: slot m takes [rr0(m), rr0(m+1)).
    auto rr0 = [](int m) { return m * NSDP / NDQ; };

    // One iteration on block `it`, held in buffer B.
    auto step = [&](auto buf_c, int it) __attribute__((always_inline)) {
        constexpr int B = decltype(buf_c)::value;
        using B2 = std::integral_constant<int, (B + 2) % NB>;
        using B3 = std::integral_constant<int, (B + 3) % NB>;
        // ---------------- phase X
        __builtin_amdgcn_sched_barrier(0);
        float sv[NEL], dpv[NEL];  // S^T and dP^T of block it, out of the accumulators
#pragma unroll
        for (int e = 0; e < NEL; ++e) {
            sv[e] = s_acc[e / 16][e % 16];
            dpv[e] = dp_acc[e / 16][e % 16];
            asm volatile("" : "+v"(sv[e]), "+v"(dpv[e]));
        }
        float dsv[NEL];
        Frag<bf16> dsb[NKT][2];
#pragma unroll
        for (int k = 0; k < NSDP; ++k) {
            // product k of block it+1 (stale operands past the last block: unused)
            sdp_one(k);
            // the first transposed operands of phase Y
            if (k >= NSDP - kQLead && k - (NSDP - kQLead) < NDQ) read_tr(buf_c, k - (NSDP - kQLead));
#pragma unroll
            for (int e = el0(k); e < el0(k + 1); ++e) {
                const float p = fast_exp2(__builtin_fmaf(sv[e], a.scale_log2, -lse2));
                float ds = p * (dpv[e] - drow);
                // pin: keeps this element's arithmetic in its slot (pure
                // arithmetic is otherwise free to drift towards its uses)
                asm volatile("" : "+v"(ds));
                dsv[e] = ds;
                if (e % 8 == 7) pack_frag(dsb[e / 16][(e % 16) / 8], dsv + e - 7);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        // masked blocks: dS^T of key kk = k0 + 32kt + acc_row(r, g) is kept iff
        // kk < kv_end and (causal) kk <= the lane's query.  Bitwise, so that a
        // masked element's value (which may be inf or nan) does not matter.
        if (it >= n_full) {
            const int k0 = it * BK;
            const int lim = min(kv_end - 1, a.mask.causal ? qi : kv_end - 1);  // keep iff kk <= lim
#pragma unroll
            for (int kt = 0; kt < NKT; ++kt) {
                const int thr = lim - k0 - 32 * kt - 4 * g;  // keep iff acc_row(r, 0) <= thr
#pragma unroll
                for (int cc = 0; cc < 2; ++cc) {
                    uint32_t w[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int r = 8 * cc + 2 * u;
                        w[u] = (acc_row(r, 0) <= thr ? 0x0000ffffu : 0u) | (acc_row(r + 1, 0) <= thr ? 0xffff0000u : 0u);
                    }
                    using u32x4 = uint32_t __attribute__((ext_vector_type(4)));
                    const u32x4 wm = u32x4{w[0], w[1], w[2], w[3]};
                    dsb[kt][cc].v = __builtin_bit_cast(bf16x8, __builtin_bit_cast(u32x4, dsb[kt][cc].v) & wm);
                }
            }
        }
        // ---------------- block it+2 landed in every wave; block it-1's buffer is free
        wait_vmcnt<0>();
        __syncthreads();
        if (it + 3 < n_iter) issue(B3{}, it + 3);
        __builtin_amdgcn_sched_barrier(0);
        // ---------------- phase Y
#pragma unroll
        for (int m = 0; m < NDQ; ++m) {
            Frag<bf16> f;
            f.v = bf16x8{trv[2 * m][0], trv[2 * m][1], trv[2 * m][2], trv[2 * m][3],
                         trv[2 * m + 1][0], trv[2 * m + 1][1], trv[2 * m + 1][2], trv[2 * m + 1][3]};
            const int t = m % ND, cc = (m / ND) % 2, kt = m / (2 * ND);
            mma(dq[t], f, dsb[kt][cc]);
            if (m + kQLead < NDQ) read_tr(buf_c, m + kQLead);
            // row operands of block it+2, for phase X(it+1) (stale past the last block: unused)
#pragma unroll
            for (int k = rr0(m); k < rr0(m + 1); ++k) read_row(B2{}, k);
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    using C0 = std::integral_constant<int, 0>;
    using C1 = std::integral_constant<int, 1>;
    using C2 = std::integral_constant<int, 2>;
    using C3 = std::integral_constant<int, 3>;
    if (n_iter > 0) {
        issue(C0{}, 0);
        if (n_iter > 1) issue(C1{}, 1);
        if (n_iter > 2) issue(C2{}, 2);
        wait_vmcnt<0>();
        __syncthreads();
#pragma unroll
        for (int k = 0; k < NSDP; ++k) read_row(C0{}, k);
#pragma unroll
        for (int k = 0; k < NSDP; ++k) sdp_one(k);
#pragma unroll
        for (int k = 0; k < NSDP; ++k) read_row(C1{}, k);  // stale when there is no block 1
    }
    // Blocks in order, four per trip (one per LDS buffer).
    for (int it = 0; it < n_iter; it += 4) {
        step(C0{}, it);
        if (it + 1 < n_iter) step(C1{}, it + 1);
        if (it + 2 < n_iter) step(C2{}, it + 2);
        if (it + 3 < n_iter) step(C3{}, it + 3);
    }

    if (qi < S) {
        bf16* dqrow = static_cast<bf16*>(a.dq) + a.mdq.head_base(b, h) + (int64_t)qi * a.mdq.ss;
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

template __global__ void attn_bwd_q_bf16<32>(BwdArgs);
template __global__ void attn_bwd_q_bf16<64>(BwdArgs);
template __global__ void attn_bwd_q_bf16<128>(BwdArgs);

}  // namespace

template <int D>
hipError_t launch_attn_bwd_q_bf16(const BwdArgs& a, hipStream_t stream) {
    const hipError_t once = ensure_dynamic_lds<&attn_bwd_q_bf16<D>>(QPipe<D>::BYTES);
    if (once != hipSuccess) return once;
    constexpr int lds = QPipe<D>::BYTES;
    hipLaunchKernelGGL((attn_bwd_q_bf16<D>), dim3(rank_major_grid((a.S + kQRows - 1) / kQRows, a.Hq * a.B)), dim3(256),
                       lds, stream, a);
    return hipGetLastError();
}

template hipError_t launch_attn_bwd_q_bf16<32>(const BwdArgs&, hipStream_t);
template hipError_t launch_attn_bwd_q_bf16<64>(const BwdArgs&, hipStream_t);
template hipError_t launch_attn_bwd_q_bf16<128>(const BwdArgs&, hipStream_t);

}  // namespace fbl
