"""GPU parity of the projection products (fbl_proj, through the C ABI) against
the fp64 oracle: Y = X W, dX = dY W^T, dW = X^T dY on bf16 token-major
operands, every tile configuration, strided (column-view) operands and outputs, and the
paper-scale shape on sampled output rows.

Tolerance: max|gpu - ref| / max|ref| <= 2e-2 (bf16 storage, fp32 accumulation).
"""
import numpy as np
import pytest

import oracle
import synth
from parity_util import note, rel_err, to_dev, to_np

pytestmark = pytest.mark.gpu
TOL = 2e-2


def _lib():
    import paper_2607_21624_amd as fbl
    return fbl


def _inputs(M, K, N, seed):
    rng = np.random.default_rng(seed)
    return (synth.round_to_bf16(rng.standard_normal((M, K))), synth.round_to_bf16(rng.standard_normal((K, N))),
            synth.round_to_bf16(rng.standard_normal((M, N))))


# M, K, N: multiples of the tiles; ragged (no extent a multiple of 32: every tile masks rows and columns and
# the last step holds a half chunk); LoRA ranks 16 and 8 as the narrow output or the contraction
SHAPES = [(64, 64, 64), (128, 192, 64), (192, 256, 128), (256, 128, 320), (256, 256, 256), (512, 128, 384),
          (104, 72, 40), (200, 136, 264), (512, 2048, 16), (512, 16, 2048), (256, 8, 512), (256, 512, 8)]


NTILES = 21  # fbl_gemm_tile_count(); tests/test_boundary.py pins it


@pytest.mark.parametrize("tile", ["auto"] + list(range(NTILES)))
@pytest.mark.parametrize("M,K,N", SHAPES)
def test_proj_products_match_oracle(M, K, N, tile):
    """Every tile configuration (output tile, staged depth, wavefront grid and
    contraction split) on every product and shape, whether or not the tile
    divides the extents (partial tiles are masked)."""
    import torch
    fbl = _lib()
    x, w, dy = _inputs(M, K, N, M + 3 * K + 7 * N)
    X, W, dY = to_dev(x, "bf16"), to_dev(w, "bf16"), to_dev(dy, "bf16")
    note(f"proj M={M} K={K} N={N} tile={tile}")
    cases = [(fbl.FBL_PROJ_FWD, X, W, oracle.proj_fwd(x, w)),
             (fbl.FBL_PROJ_BWD_DATA, dY, W, oracle.proj_bwd_data(dy, w)),
             (fbl.FBL_PROJ_BWD_WEIGHT, X, dY, oracle.proj_bwd_weight(x, dy))]
    t = fbl.FBL_GEMM_TILE_AUTO if tile == "auto" else tile
    for op, a, b, ref in cases:
        # the output, poisoned, also checks that nothing is written past its extent
        out = torch.full((ref.shape[0] + 8, ref.shape[1] + 8), float("nan"), dtype=torch.bfloat16, device="cuda")
        got = fbl.proj(op, a, b, out=out[:ref.shape[0], :ref.shape[1]], tile=t)
        torch.cuda.synchronize()
        rest = torch.cat([out[ref.shape[0]:].flatten(), out[:ref.shape[0], ref.shape[1]:].flatten()])
        assert torch.isnan(rest.float()).all(), f"op {op} tile {tile}: wrote outside the output"
        torch.cuda.synchronize()
        assert got.shape == ref.shape
        e = rel_err(to_np(got), ref)
        assert e <= TOL, f"op {op} tile {tile}: rel err {e}"


def test_proj_strided_operands_and_packed_output():
    """X and dY as column views of wider buffers; the Q, K, V projections
    written straight into the column blocks of one packed QKV buffer."""
    import torch
    fbl = _lib()
    M, K, Hq, Hkv, d = 128, 256, 4, 2, 64
    rng = np.random.default_rng(17)
    xw = synth.round_to_bf16(rng.standard_normal((M, K + 64)))   # X = first K columns
    wq, wk, wv = (synth.round_to_bf16(rng.standard_normal((K, h * d))) for h in (Hq, Hkv, Hkv))
    Xw = to_dev(xw, "bf16")
    X = Xw[:, :K]
    qkv = torch.zeros((M, (Hq + 2 * Hkv) * d), dtype=torch.bfloat16, device="cuda")
    cols = [(0, Hq * d, wq), (Hq * d, (Hq + Hkv) * d, wk), ((Hq + Hkv) * d, (Hq + 2 * Hkv) * d, wv)]
    note("proj packed QKV output")
    for c0, c1, wmat in cols:
        fbl.proj(fbl.FBL_PROJ_FWD, X, to_dev(wmat, "bf16"), out=qkv[:, c0:c1])
    torch.cuda.synchronize()
    got = to_np(qkv)
    for c0, c1, wmat in cols:
        assert rel_err(got[:, c0:c1], oracle.proj_fwd(xw[:, :K], wmat)) <= TOL
    # weight gradient from a strided dY view (the Q block of a packed gradient)
    dqkv = synth.round_to_bf16(rng.standard_normal((M, (Hq + 2 * Hkv) * d)))
    dW = fbl.proj(fbl.FBL_PROJ_BWD_WEIGHT, X, to_dev(dqkv, "bf16")[:, :Hq * d])
    torch.cuda.synchronize()
    assert rel_err(to_np(dW), oracle.proj_bwd_weight(xw[:, :K], dqkv[:, :Hq * d])) <= TOL


def test_proj_paper_shape_sampled_rows():
    """M=512 tokens, K=2048, N=8192: full launches, the oracle checks 64 rows
    of each output (rows are independent, so a subset is exactly the oracle's
    answer for those rows)."""
    import torch
    fbl = _lib()
    M, K, N = 512, 2048, 8192
    x, w, dy = _inputs(M, K, N, 2024)
    X, W, dY = to_dev(x, "bf16"), to_dev(w, "bf16"), to_dev(dy, "bf16")
    note("proj paper shape 512 x 2048 x 8192")
    rows = np.arange(0, 512, 8)
    y = fbl.proj(fbl.FBL_PROJ_FWD, X, W)
    dx = fbl.proj(fbl.FBL_PROJ_BWD_DATA, dY, W)
    dw = fbl.proj(fbl.FBL_PROJ_BWD_WEIGHT, X, dY)
    torch.cuda.synchronize()
    assert rel_err(to_np(y[rows]), oracle.proj_fwd(x[rows], w)) <= TOL
    assert rel_err(to_np(dx[rows]), oracle.proj_bwd_data(dy[rows], w)) <= TOL
    krows = np.arange(0, K, 32)
    assert rel_err(to_np(dw[krows]), oracle.proj_bwd_weight(x[:, krows], dy)) <= TOL


@pytest.mark.parametrize("objective", [0, 1])
def test_proj_tune_picks_a_measured_candidate(objective):
    """fbl_proj_tune times exactly the candidate tiles, picks the one its
    objective ranks first (recomputed here from the returned times and the
    staged-bytes model), leaves the product in `out`, and FBL_GEMM_TILE_AUTO
    then runs the chosen tile (bit-identical output to the explicit id)."""
    import torch
    fbl = _lib()
    M, K, N = 256, 256, 512
    x, w, dy = _inputs(M, K, N, 99 + objective)
    X, W, dY = to_dev(x, "bf16"), to_dev(w, "bf16"), to_dev(dy, "bf16")
    tiles = fbl.gemm_tiles()
    fbl.proj_tune_reset()
    for op, a, b, ref, (rows, cols, kc) in [
            (fbl.FBL_PROJ_FWD, X, W, oracle.proj_fwd(x, w), (M, N, K)),
            (fbl.FBL_PROJ_BWD_DATA, dY, W, oracle.proj_bwd_data(dy, w), (M, K, N)),
            (fbl.FBL_PROJ_BWD_WEIGHT, X, dY, oracle.proj_bwd_weight(x, dy), (K, N, M))]:
        note(f"proj_tune op={op} objective={objective}")
        out = torch.empty(ref.shape, dtype=torch.bfloat16, device="cuda")
        assert fbl.proj_tuned_tile(op, M, K, N) == -1
        best, ms = fbl.proj_tune(op, a, b, out, objective=objective, reps=3)
        torch.cuda.synchronize()
        assert sorted(ms) == fbl.proj_candidates(op, M, K, N)
        assert all(v > 0 for v in ms.values())
        flops = 2.0 * rows * cols * kc
        min_bytes = 2.0 * (rows * kc + kc * cols + rows * cols)

        def score(t):
            if objective == 0:
                return 1.0 / ms[t]
            g = tiles[t]
            staged = 2.0 * (rows * kc * (cols // g["bn"]) + kc * cols * (rows // g["bm"]) + rows * cols)
            return flops / (ms[t] * 1e-3) * (min_bytes / staged)
        assert best == max(sorted(ms), key=score)
        assert fbl.proj_tuned_tile(op, M, K, N) == best
        assert rel_err(to_np(out), ref) <= TOL
        auto = fbl.proj(op, a, b)
        explicit = fbl.proj(op, a, b, tile=best)
        torch.cuda.synchronize()
        assert torch.equal(auto, explicit)
    fbl.proj_tune_reset()
    assert fbl.proj_tuned_tile(fbl.FBL_PROJ_FWD, M, K, N) == -1


@pytest.mark.parametrize("r", [8, 16, 64])
def test_lora_chain(r):
    """A LoRA adapter on a frozen projection (section 2.2's example): H = X A,
    Y = X W + H B, and the backward dB = H^T dY, dH = dY B^T, dA = X^T dH,
    dX = dY W^T + dH A^T -- eight products at rank r on token-major operands,
    against the fp64 oracle's chain (the GPU rounds H and dH to bf16 between
    products)."""
    import torch
    fbl = _lib()
    M, K, N = 512, 1024, 1536
    rng = np.random.default_rng(300 + r)
    bf = lambda *s: synth.round_to_bf16(rng.standard_normal(s))
    x, w, a_, b_, dy = bf(M, K), bf(K, N), bf(K, r), bf(r, N), bf(M, N)
    X, W, A, B, dY = (to_dev(t, "bf16") for t in (x, w, a_, b_, dy))
    note(f"lora chain r={r}")
    H = fbl.proj(fbl.FBL_PROJ_FWD, X, A)
    Y = fbl.proj(fbl.FBL_PROJ_FWD, X, W).float() + fbl.proj(fbl.FBL_PROJ_FWD, H, B).float()
    dB = fbl.proj(fbl.FBL_PROJ_BWD_WEIGHT, H, dY)
    dH = fbl.proj(fbl.FBL_PROJ_BWD_DATA, dY, B)
    dA = fbl.proj(fbl.FBL_PROJ_BWD_WEIGHT, X, dH)
    dX = fbl.proj(fbl.FBL_PROJ_BWD_DATA, dY, W).float() + fbl.proj(fbl.FBL_PROJ_BWD_DATA, dH, A).float()
    torch.cuda.synchronize()
    h = oracle.proj_fwd(x, a_)
    dh = oracle.proj_bwd_data(dy, b_)
    refs = {"H": (H, h), "Y": (Y, oracle.proj_fwd(x, w) + oracle.proj_fwd(h, b_)),
            "dB": (dB, oracle.proj_bwd_weight(h, dy)), "dH": (dH, dh),
            "dA": (dA, oracle.proj_bwd_weight(x, dh)),
            "dX": (dX, oracle.proj_bwd_data(dy, w) + oracle.proj_bwd_data(dh, a_))}
    for name, (got, ref) in refs.items():
        assert got.shape == ref.shape, name
        assert rel_err(to_np(got), ref) <= TOL, name


# the smallest extents each product accepts: output rows any, output columns a multiple of 4,
# contraction a multiple of 8
TINY = [(op, M, K, N) for op, (M, K, N) in
        [(0, (1, 8, 4)), (0, (5, 24, 12)), (1, (1, 4, 8)), (1, (7, 12, 40)), (2, (8, 1, 4)), (2, (16, 9, 20))]]


@pytest.mark.parametrize("tile", ["auto"] + list(range(NTILES)))
@pytest.mark.parametrize("op,M,K,N", TINY)
def test_proj_tiny_extents(op, M, K, N, tile):
    """One token, a handful of columns, a contraction of 8: every tile masks
    almost all of its rows and columns and zeroes most of its only step."""
    import torch
    fbl = _lib()
    rng = np.random.default_rng(M * 7 + K * 3 + N + op)
    bf = lambda *s: synth.round_to_bf16(rng.standard_normal(s))
    if op == 0:
        a, b = bf(M, K), bf(K, N)
        ref = oracle.proj_fwd(a, b)
    elif op == 1:
        a, b = bf(M, N), bf(K, N)
        ref = oracle.proj_bwd_data(a, b)
    else:
        a, b = bf(M, K), bf(M, N)
        ref = oracle.proj_bwd_weight(a, b)
    note(f"proj tiny op={op} M={M} K={K} N={N} tile={tile}")
    pad8 = lambda n: (n + 7) // 8 * 8   # rows must start on 16-byte boundaries: views of padded buffers

    def view_of(x):
        buf = torch.zeros((x.shape[0], pad8(x.shape[1])), dtype=torch.bfloat16, device="cuda")
        buf[:, :x.shape[1]] = to_dev(x, "bf16")
        return buf[:, :x.shape[1]]
    out = torch.full((ref.shape[0] + 8, pad8(ref.shape[1]) + 8), float("nan"), dtype=torch.bfloat16, device="cuda")
    view = out[:ref.shape[0], :ref.shape[1]]
    t = fbl.FBL_GEMM_TILE_AUTO if tile == "auto" else tile
    fbl.proj(op, view_of(a), view_of(b), out=view, tile=t)
    torch.cuda.synchronize()
    rest = torch.cat([out[ref.shape[0]:].flatten(), out[:ref.shape[0], ref.shape[1]:].flatten()])
    assert torch.isnan(rest.float()).all(), "wrote outside the output"
    assert rel_err(to_np(view), ref) <= TOL


@pytest.mark.parametrize("M,K,N", [(64, 64, 64), (100, 37, 53), (1, 3, 5), (257, 130, 66), (512, 1024, 384)])
def test_proj_fp32_matches_oracle(M, K, N):
    """fp32 storage (fbl_proj_dt): any extents, odd widths, every product, to
    1e-4 of max|ref|; outputs written into NaN-poisoned wider buffers."""
    import torch
    fbl = _lib()
    rng = np.random.default_rng(M + 5 * K + 11 * N)
    x, w, dy = rng.standard_normal((M, K)), rng.standard_normal((K, N)), rng.standard_normal((M, N))
    X, W, dY = (torch.tensor(t, dtype=torch.float32, device="cuda") for t in (x, w, dy))
    note(f"proj fp32 M={M} K={K} N={N}")
    for op, a, b, ref in ((fbl.FBL_PROJ_FWD, X, W, oracle.proj_fwd(x, w)),
                          (fbl.FBL_PROJ_BWD_DATA, dY, W, oracle.proj_bwd_data(dy, w)),
                          (fbl.FBL_PROJ_BWD_WEIGHT, X, dY, oracle.proj_bwd_weight(x, dy))):
        out = torch.full((ref.shape[0] + 3, ref.shape[1] + 5), float("nan"), dtype=torch.float32, device="cuda")
        view = out[:ref.shape[0], :ref.shape[1]]
        fbl.proj(op, a, b, out=view)
        torch.cuda.synchronize()
        rest = torch.cat([out[ref.shape[0]:].flatten(), out[:ref.shape[0], ref.shape[1]:].flatten()])
        assert torch.isnan(rest).all(), f"op {op}: wrote outside the output"
        assert rel_err(to_np(view), ref) <= 1e-4, f"op {op}"


@pytest.mark.parametrize("op,M,K,N", [(0, 512, 2048, 8192), (1, 512, 4096, 12288), (2, 512, 1024, 4096),
                                      (0, 1024, 512, 4096), (1, 300, 1000, 2048)])
def test_auto_tile_query_matches_dispatch(op, M, K, N):
    """The id fbl_proj_auto_tile reports is the tile FBL_GEMM_TILE_AUTO runs:
    the two products are equal bit for bit (each tile's summation order is
    its own)."""
    import torch
    fbl = _lib()
    fbl.proj_tune_reset()
    g = torch.Generator(device="cpu").manual_seed(M + K + N + op)
    rows_a, cols_a = {0: (M, K), 1: (M, N), 2: (M, K)}[op]
    rows_b, cols_b = {0: (K, N), 1: (K, N), 2: (M, N)}[op]
    a = torch.randn(rows_a, cols_a, generator=g).to(device="cuda", dtype=torch.bfloat16)
    b = torch.randn(rows_b, cols_b, generator=g).to(device="cuda", dtype=torch.bfloat16)
    t = fbl.proj_auto_tile(op, M, K, N)
    note(f"auto tile query op={op} M={M} K={K} N={N} -> t{t}")
    assert t in fbl.proj_candidates(op, M, K, N)
    auto = fbl.proj(op, a, b)
    named = fbl.proj(op, a, b, tile=t)
    torch.cuda.synchronize()
    assert torch.equal(auto, named)
