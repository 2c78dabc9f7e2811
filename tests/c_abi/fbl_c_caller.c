/*
 * A caller of the C ABI written in plain C11, with no PyTorch: the boundary
 * is usable from any language that can call C.
 *
 *   fbl_c_caller host
 *       host-only entry points: descriptors and their index map (against the
 *       token-major closed form), packed-QKV descriptors, status strings,
 *       workspace sizes, the tile table and the projection candidates.
 *   fbl_c_caller attn IN OUT
 *       attention forward and backward on the GPU through fbl_attn_fwd /
 *       fbl_attn_bwd, device memory from hipMalloc, the null stream.  IN holds
 *       int32 B, S, Hq, Hkv, D, causal, then float32 scale, then the bf16 bit
 *       patterns of q, k, v, dO ([B, S, H*D] token-major each).  OUT receives
 *       the bf16 bit patterns of o, dq, dk, dv and the float32 lse, in that
 *       order.
 *   fbl_c_caller proj IN OUT
 *       the three projection products through fbl_proj (automatic tile),
 *       row-major operands with no padding.  IN holds int32 M, K, N, then the
 *       bf16 bit patterns of X [M, K], W [K, N], dY [M, N]; OUT receives those
 *       of Y = X W [M, N], dX = dY W^T [M, K] and dW = X^T dY [K, N].
 * Exit status 0 on success; a message on stderr otherwise.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "fbl.h"

static int failures = 0;

#define CHECK(cond)                                                                 \
    do {                                                                            \
        if (!(cond)) {                                                              \
            fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
            ++failures;                                                             \
        }                                                                           \
    } while (0)

static int host_checks(void) {
    fbl_layout l;
    /* token-major defaults and the index map */
    CHECK(fbl_layout_desc(&l, FBL_BF16, 2, 5, 3, 64, 0, 0, 0) == FBL_OK);
    CHECK(l.ss == 3 * 64 && l.sh == 64 && l.sd == 1 && l.sb == 5 * 3 * 64 && l.tile_d == 64);
    for (int64_t b = 0; b < 2; ++b)
        for (int64_t h = 0; h < 3; ++h)
            for (int64_t s = 0; s < 5; ++s)
                for (int64_t i = 0; i < 64; i += 7)
                    CHECK(fbl_layout_offset(&l, b, h, s, i) == ((b * 5 + s) * 3 + h) * 64 + i);
    CHECK(fbl_layout_offset(&l, 2, 0, 0, 0) == -1);
    CHECK(fbl_layout_offset(NULL, 0, 0, 0, 0) == -1);
    /* a row stride wider than H*D (a view into a packed projection output) */
    CHECK(fbl_layout_desc(&l, FBL_F32, 1, 4, 2, 32, 320, 0, 0) == FBL_OK);
    CHECK(fbl_layout_offset(&l, 0, 1, 3, 5) == 3 * 320 + 32 + 5);
    /* rejections leave the descriptor zeroed */
    CHECK(fbl_layout_desc(&l, FBL_BF16, 0, 5, 3, 64, 0, 0, 0) == FBL_ERR_SHAPE && l.D == 0);
    CHECK(fbl_layout_desc(&l, FBL_BF16, 1, 5, 3, 64, 100, 0, 0) == FBL_ERR_LAYOUT);
    CHECK(fbl_layout_desc(&l, 7, 1, 5, 3, 64, 0, 0, 0) == FBL_ERR_DTYPE);
    CHECK(fbl_layout_desc(NULL, FBL_BF16, 1, 5, 3, 64, 0, 0, 0) == FBL_ERR_NULL);
    /* packed QKV: Q, K, V share the packed row stride, K and V start after Q */
    fbl_layout lq, lk, lv;
    int64_t ko = 0, vo = 0;
    CHECK(fbl_layout_packed_qkv(&lq, &lk, &lv, &ko, &vo, FBL_BF16, 2, 7, 8, 2, 128, 0, 0) == FBL_OK);
    CHECK(lq.ss == 12 * 128 && lk.ss == lq.ss && lv.ss == lq.ss && lk.H == 2 && ko == 8 * 128 && vo == 10 * 128);
    CHECK(fbl_layout_offset(&lk, 1, 1, 6, 3) + ko == (1 * 7 + 6) * 12 * 128 + 8 * 128 + 128 + 3);
    /* status strings */
    CHECK(strstr(fbl_status_str(FBL_ERR_UNSUPPORTED), "UNSUPPORTED") != NULL);
    CHECK(fbl_status_str(FBL_OK) != NULL);
    /* backward workspace: [B, Hq, 2, S] fp32 statistics (256-byte rounded) plus, for bf16,
       B*Hq*ceil(S/32)^2 blocks of 2 KB */
    size_t ws = 0, ws_min = 0;
    CHECK(fbl_layout_desc(&lq, FBL_BF16, 2, 100, 6, 64, 0, 0, 0) == FBL_OK);
    CHECK(fbl_layout_desc(&lk, FBL_BF16, 2, 100, 3, 64, 0, 0, 0) == FBL_OK);
    CHECK(fbl_attn_bwd_workspace(&lq, &lk, &ws) == FBL_OK);
    CHECK(fbl_attn_bwd_workspace_min(&lq, &lk, &ws_min) == FBL_OK);
    const size_t stats = (2 * 6 * 100 * 2 * 4 + 255) / 256 * 256;
    CHECK(ws_min == stats && ws == stats + (size_t)2 * 6 * 4 * 4 * 2048);
    /* tile table and candidates */
    const int32_t nt = fbl_gemm_tile_count();
    CHECK(nt > 0);
    int32_t info[8];
    CHECK(fbl_gemm_tile_info(0, info) == FBL_OK && info[0] == 128 && info[1] == 128);
    CHECK(fbl_gemm_tile_info(nt, info) == FBL_ERR_ARG);
    int32_t ids[64], n = 0;
    CHECK(fbl_proj_candidates(FBL_PROJ_FWD, 512, 2048, 8192, ids, 64, &n) == FBL_OK && n > 0 && n <= nt);
    if (failures) return 1;
    printf("host checks passed (%d tiles, %d forward candidates at 512 x 2048 x 8192)\n", nt, n);
    return 0;
}

static int read_all(FILE* f, void* p, size_t n) { return fread(p, 1, n, f) == n; }

#define HIP(call)                                                                       \
    do {                                                                                \
        hipError_t e_ = (call);                                                         \
        if (e_ != hipSuccess) {                                                         \
            fprintf(stderr, "%s:%d: %s: %s\n", __FILE__, __LINE__, #call, hipGetErrorString(e_)); \
            return 1;                                                                   \
        }                                                                               \
    } while (0)
#define FBL(call)                                                                       \
    do {                                                                                \
        fbl_status s_ = (call);                                                         \
        if (s_ != FBL_OK) {                                                             \
            fprintf(stderr, "%s:%d: %s: %s\n", __FILE__, __LINE__, #call, fbl_status_str(s_)); \
            return 1;                                                                   \
        }                                                                               \
    } while (0)

static int attn_run(const char* in_path, const char* out_path) {
    FILE* f = fopen(in_path, "rb");
    if (!f) { fprintf(stderr, "cannot open %s\n", in_path); return 1; }
    int32_t hdr[6];
    float scale;
    if (!read_all(f, hdr, sizeof hdr) || !read_all(f, &scale, sizeof scale)) { fclose(f); return 1; }
    const int64_t B = hdr[0], S = hdr[1], Hq = hdr[2], Hkv = hdr[3], D = hdr[4];
    const int causal = hdr[5];
    if (B <= 0 || S <= 0 || Hq <= 0 || Hkv <= 0 || D <= 0 || B * S * Hq * D > ((int64_t)1 << 28)) {
        fclose(f);
        fprintf(stderr, "bad header\n");
        return 1;
    }
    const size_t nq = (size_t)(B * S * Hq * D), nk = (size_t)(B * S * Hkv * D);
    uint16_t* hq = malloc(2 * nq);
    uint16_t* hk = malloc(2 * nk);
    uint16_t* hv = malloc(2 * nk);
    uint16_t* hdo = malloc(2 * nq);
    float* hlse = malloc(4 * (size_t)(B * Hq * S));
    if (!hq || !hk || !hv || !hdo || !hlse) { fclose(f); return 1; }
    const int ok = read_all(f, hq, 2 * nq) && read_all(f, hk, 2 * nk) && read_all(f, hv, 2 * nk) &&
                   read_all(f, hdo, 2 * nq);
    fclose(f);
    if (!ok) { fprintf(stderr, "short input\n"); return 1; }

    fbl_layout lq, lk;
    FBL(fbl_layout_desc(&lq, FBL_BF16, B, S, Hq, D, 0, 0, 0));
    FBL(fbl_layout_desc(&lk, FBL_BF16, B, S, Hkv, D, 0, 0, 0));
    void *q, *k, *v, *o, *dO, *dq, *dk, *dv, *ws;
    float* lse;
    size_t ws_bytes = 0;
    FBL(fbl_attn_bwd_workspace(&lq, &lk, &ws_bytes));
    HIP(hipMalloc(&q, 2 * nq));
    HIP(hipMalloc(&k, 2 * nk));
    HIP(hipMalloc(&v, 2 * nk));
    HIP(hipMalloc(&o, 2 * nq));
    HIP(hipMalloc(&dO, 2 * nq));
    HIP(hipMalloc(&dq, 2 * nq));
    HIP(hipMalloc(&dk, 2 * nk));
    HIP(hipMalloc(&dv, 2 * nk));
    HIP(hipMalloc((void**)&lse, 4 * (size_t)(B * Hq * S)));
    HIP(hipMalloc(&ws, ws_bytes));
    HIP(hipMemcpy(q, hq, 2 * nq, hipMemcpyHostToDevice));
    HIP(hipMemcpy(k, hk, 2 * nk, hipMemcpyHostToDevice));
    HIP(hipMemcpy(v, hv, 2 * nk, hipMemcpyHostToDevice));
    HIP(hipMemcpy(dO, hdo, 2 * nq, hipMemcpyHostToDevice));

    fbl_mask mask;
    memset(&mask, 0, sizeof mask);
    mask.kind = causal ? FBL_MASK_CAUSAL : 0u;
    FBL(fbl_attn_fwd(&lq, q, &lk, k, &lk, v, &lq, o, lse, scale, mask, NULL));
    FBL(fbl_attn_bwd(&lq, q, &lk, k, &lk, v, &lq, o, &lq, dO, lse, scale, mask, &lq, dq, &lk, dk, &lk, dv, ws,
                     ws_bytes, NULL));
    HIP(hipDeviceSynchronize());

    FILE* g = fopen(out_path, "wb");
    if (!g) { fprintf(stderr, "cannot open %s\n", out_path); return 1; }
    const void* outs[4] = {o, dq, dk, dv};
    const size_t sizes[4] = {2 * nq, 2 * nq, 2 * nk, 2 * nk};
    for (int i = 0; i < 4; ++i) {
        void* h = malloc(sizes[i]);
        if (!h) { fclose(g); return 1; }
        HIP(hipMemcpy(h, outs[i], sizes[i], hipMemcpyDeviceToHost));
        fwrite(h, 1, sizes[i], g);
        free(h);
    }
    HIP(hipMemcpy(hlse, lse, 4 * (size_t)(B * Hq * S), hipMemcpyDeviceToHost));
    fwrite(hlse, 4, (size_t)(B * Hq * S), g);
    fclose(g);
    void* bufs[10] = {q, k, v, o, dO, dq, dk, dv, lse, ws};
    for (int i = 0; i < 10; ++i) HIP(hipFree(bufs[i]));
    free(hq); free(hk); free(hv); free(hdo); free(hlse);
    printf("attention forward and backward done (B=%d S=%d Hq=%d Hkv=%d D=%d causal=%d)\n", (int)B, (int)S,
           (int)Hq, (int)Hkv, (int)D, causal);
    return 0;
}

static int proj_run(const char* in_path, const char* out_path) {
    FILE* f = fopen(in_path, "rb");
    if (!f) { fprintf(stderr, "cannot open %s\n", in_path); return 1; }
    int32_t hdr[3];
    if (!read_all(f, hdr, sizeof hdr)) { fclose(f); return 1; }
    const int64_t M = hdr[0], K = hdr[1], N = hdr[2];
    if (M <= 0 || K <= 0 || N <= 0 || M * K > ((int64_t)1 << 26) || K * N > ((int64_t)1 << 26) ||
        M * N > ((int64_t)1 << 26)) {
        fclose(f);
        fprintf(stderr, "bad header\n");
        return 1;
    }
    const size_t nx = (size_t)(M * K), nw = (size_t)(K * N), ny = (size_t)(M * N);
    uint16_t* hx = malloc(2 * nx);
    uint16_t* hw = malloc(2 * nw);
    uint16_t* hdy = malloc(2 * ny);
    if (!hx || !hw || !hdy) { fclose(f); return 1; }
    const int ok = read_all(f, hx, 2 * nx) && read_all(f, hw, 2 * nw) && read_all(f, hdy, 2 * ny);
    fclose(f);
    if (!ok) { fprintf(stderr, "short input\n"); return 1; }
    void *x, *w, *dy, *y, *dx, *dw;
    HIP(hipMalloc(&x, 2 * nx));
    HIP(hipMalloc(&w, 2 * nw));
    HIP(hipMalloc(&dy, 2 * ny));
    HIP(hipMalloc(&y, 2 * ny));
    HIP(hipMalloc(&dx, 2 * nx));
    HIP(hipMalloc(&dw, 2 * nw));
    HIP(hipMemcpy(x, hx, 2 * nx, hipMemcpyHostToDevice));
    HIP(hipMemcpy(w, hw, 2 * nw, hipMemcpyHostToDevice));
    HIP(hipMemcpy(dy, hdy, 2 * ny, hipMemcpyHostToDevice));
    /* leading dimensions: the stored row lengths */
    FBL(fbl_proj(FBL_PROJ_FWD, M, K, N, x, K, w, N, y, N, FBL_GEMM_TILE_AUTO, NULL));
    FBL(fbl_proj(FBL_PROJ_BWD_DATA, M, K, N, dy, N, w, N, dx, K, FBL_GEMM_TILE_AUTO, NULL));
    FBL(fbl_proj(FBL_PROJ_BWD_WEIGHT, M, K, N, x, K, dy, N, dw, N, FBL_GEMM_TILE_AUTO, NULL));
    HIP(hipDeviceSynchronize());
    FILE* g = fopen(out_path, "wb");
    if (!g) { fprintf(stderr, "cannot open %s\n", out_path); return 1; }
    const void* outs[3] = {y, dx, dw};
    const size_t sizes[3] = {2 * ny, 2 * nx, 2 * nw};
    for (int i = 0; i < 3; ++i) {
        void* h = malloc(sizes[i]);
        if (!h) { fclose(g); return 1; }
        HIP(hipMemcpy(h, outs[i], sizes[i], hipMemcpyDeviceToHost));
        fwrite(h, 1, sizes[i], g);
        free(h);
    }
    fclose(g);
    void* bufs[6] = {x, w, dy, y, dx, dw};
    for (int i = 0; i < 6; ++i) HIP(hipFree(bufs[i]));
    free(hx); free(hw); free(hdy);
    printf("projection products done (M=%d K=%d N=%d)\n", (int)M, (int)K, (int)N);
    return 0;
}

int main(int argc, char** argv) {
    if (argc == 2 && strcmp(argv[1], "host") == 0) return host_checks();
    if (argc == 4 && strcmp(argv[1], "attn") == 0) return attn_run(argv[2], argv[3]);
    if (argc == 4 && strcmp(argv[1], "proj") == 0) return proj_run(argv[2], argv[3]);
    fprintf(stderr, "usage: %s host | attn IN OUT | proj IN OUT\n", argv[0]);
    return 2;
}
