"""The C ABI boundary on the CPU: the library loads, exports what include/fbl.h
declares, and rejects every invalid call before any launch.

No test here ever passes validation with made-up pointers: each call carries
exactly one defect, so nothing reaches a GPU launch.
"""
import ctypes
import os
import re

import pytest

import paper_2607_21624_amd as fbl
from paper_2607_21624_amd import fbl as F

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fbl.h")

FAKE = 1 << 20          # 16-byte aligned made-up device addresses (never dereferenced)
BF16, F32 = fbl.FBL_BF16, fbl.FBL_F32


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fbl_[a-z_]+)\s*\(", text)))


def test_header_symbols_exported():
    names = header_functions()
    assert set(names) == set(fbl.EXPORTED)
    lib = ctypes.CDLL(fbl.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    for s in range(10):
        assert fbl.status_str(s).startswith("FBL_")
    assert "UNKNOWN" in fbl.status_str(99)


# ------------------------------------------------------------- descriptors
def test_layout_desc_defaults_and_tile():
    l = fbl.fbl_layout_desc(BF16, 4, 1024, 16, 64)
    assert (l.sd, l.sh, l.ss, l.sb) == (1, 64, 1024, 1024 * 1024)
    assert l.tile_d == 64 and l.reserved0 == 0 and l.reserved1 == 0


@pytest.mark.parametrize("args,status", [
    ((7, 1, 4, 2, 64), F.FBL_ERR_DTYPE),
    ((BF16, 0, 4, 2, 64), F.FBL_ERR_SHAPE),
    ((BF16, 1, 0, 2, 64), F.FBL_ERR_SHAPE),
    ((BF16, 1, 4, 0, 64), F.FBL_ERR_SHAPE),
    ((BF16, 1, 4, 2, -64), F.FBL_ERR_SHAPE),
])
def test_layout_desc_rejects(args, status):
    st, l = fbl.fbl_layout_desc_status(*args)
    assert st == status
    assert l.B == 0 and l.D == 0  # left zeroed


def test_layout_desc_row_stride_checks():
    # rows overlapping the previous row's heads
    st, _ = fbl.fbl_layout_desc_status(BF16, 2, 8, 4, 64, row_stride=4 * 64 - 8)
    assert st == F.FBL_ERR_LAYOUT
    # batches overlapping
    st, _ = fbl.fbl_layout_desc_status(BF16, 2, 8, 4, 64, row_stride=256, batch_stride=256 * 7)
    assert st == F.FBL_ERR_LAYOUT
    # 16-byte alignment of rows: 4*64 + 4 bf16 elements = 520 bytes
    st, _ = fbl.fbl_layout_desc_status(BF16, 2, 8, 4, 64, row_stride=260)
    assert st == F.FBL_ERR_ALIGN
    # a packed QKV row (12 query heads + 2*4 kv heads) is a legal view
    st, l = fbl.fbl_layout_desc_status(BF16, 2, 8, 4, 64, row_stride=(12 + 8) * 64)
    assert st == F.FBL_OK and l.ss == 20 * 64


def test_paper_tile_boundary_examples():
    import json
    cases = json.load(open(os.path.join(ROOT, "tests", "golden", "layout_cases.json")))["head_split_examples"]
    for c in cases:
        st, _ = fbl.fbl_layout_desc_status(BF16, 1, 16, c["heads"], c["head_dim"], tile_d=c["tile_d"])
        assert (st == F.FBL_OK) == c["legal"], c["cite"]
        assert c["heads"] * c["head_dim"] == c["hidden"]


def test_layout_offset_matches_oracle_bit_exact():
    import numpy as np
    import oracle
    for (B, S, H, D) in [(1, 64, 2, 32), (8, 128, 12, 64), (2, 37, 3, 128)]:
        l = fbl.fbl_layout_desc(BF16, B, S, H, D)
        want = oracle.token_major_offsets(B, S, H, D)
        got = np.empty_like(want)
        for b in range(B):
            for h in range(H):
                for s in range(S):
                    base = fbl.fbl_layout_offset(l, b, h, s, 0)
                    got[b, h, s, :] = base + np.arange(D)
                    assert fbl.fbl_layout_offset(l, b, h, s, D - 1) == base + D - 1
        assert np.array_equal(got, want)


def test_layout_offset_strided_view_matches_oracle():
    import numpy as np
    import oracle
    B, S, H, D, row = 2, 9, 4, 32, 10 * 32
    l = fbl.fbl_layout_desc(F32, B, S, H, D, row_stride=row)
    want = oracle.head_split_offsets(B, S, H, D, row_stride=row, batch_stride=S * row)
    got = np.array([[[[fbl.fbl_layout_offset(l, b, h, s, i) for i in range(D)] for s in range(S)]
                     for h in range(H)] for b in range(B)])
    assert np.array_equal(got, want)


def test_layout_offset_out_of_range():
    l = fbl.fbl_layout_desc(BF16, 2, 4, 3, 32)
    assert fbl.fbl_layout_offset(l, 2, 0, 0, 0) == -1
    assert fbl.fbl_layout_offset(l, 0, 3, 0, 0) == -1
    assert fbl.fbl_layout_offset(l, 0, 0, 4, 0) == -1
    assert fbl.fbl_layout_offset(l, 0, 0, 0, 32) == -1
    assert fbl.fbl_layout_offset(l, -1, 0, 0, 0) == -1
    assert F.LIB.fbl_layout_offset(None, 0, 0, 0, 0) == -1


# ------------------------------------------------------------ attention calls
def _fwd_setup(dtype=BF16, B=2, S=16, Hq=4, Hkv=2, D=64):
    lq = fbl.fbl_layout_desc(dtype, B, S, Hq, D)
    lk = fbl.fbl_layout_desc(dtype, B, S, Hkv, D)
    lv = fbl.fbl_layout_desc(dtype, B, S, Hkv, D)
    lo = fbl.fbl_layout_desc(dtype, B, S, Hq, D)
    es = 2 if dtype == BF16 else 4
    nq = B * S * Hq * D * es
    nk = B * S * Hkv * D * es
    ptr = {"q": FAKE, "k": FAKE + nq + 4096, "v": FAKE + nq + nk + 8192, "o": FAKE + nq + 2 * nk + 12288}
    ptr["lse"] = ptr["o"] + nq + 4096
    return lq, lk, lv, lo, ptr


def _fwd(lq, lk, lv, lo, p, scale=0.125, kind=0, kv_len=None):
    return fbl.fbl_attn_fwd_raw(lq, p["q"], lk, p["k"], lv, p["v"], lo, p["o"], p["lse"], scale,
                                F.Mask(kind, 0, kv_len), stream=0)


def _copy(l, **kw):
    n = F.Layout()
    ctypes.memmove(ctypes.byref(n), ctypes.byref(l), ctypes.sizeof(l))
    for k, v in kw.items():
        setattr(n, k, v)
    return n


def test_fwd_rejections():
    lq, lk, lv, lo, p = _fwd_setup()
    E = F
    assert _fwd(None, lk, lv, lo, p) == E.FBL_ERR_NULL
    assert _fwd(lq, lk, lv, lo, dict(p, q=None)) == E.FBL_ERR_NULL
    assert _fwd(lq, lk, lv, lo, dict(p, lse=None)) == E.FBL_ERR_NULL
    assert _fwd(lq, lk, _copy(lv, dtype=F32), lo, p) == E.FBL_ERR_DTYPE
    assert _fwd(lq, lk, lv, _copy(lo, dtype=F32), p) == E.FBL_ERR_DTYPE
    assert _fwd(lq, _copy(lk, S=8, sb=8 * 128), lv, lo, p) == E.FBL_ERR_SHAPE
    assert _fwd(lq, _copy(lk, H=3, ss=3 * 64, sb=16 * 192), _copy(lv, H=3, ss=3 * 64, sb=16 * 192), lo, p) \
        == E.FBL_ERR_SHAPE  # Hq % Hkv != 0
    assert _fwd(lq, lk, lv, _copy(lo, H=2, ss=128, sb=16 * 128), p) == E.FBL_ERR_SHAPE
    # unsupported head dim (legal layout, no kernel)
    lq2, lk2, lv2, lo2, p2 = _fwd_setup(D=48)
    assert _fwd(lq2, lk2, lv2, lo2, p2) == E.FBL_ERR_UNSUPPORTED
    # intra-tile continuity and tile boundary
    assert _fwd(_copy(lq, sd=2), lk, lv, lo, p) == E.FBL_ERR_LAYOUT
    assert _fwd(_copy(lq, tile_d=48), lk, lv, lo, p) == E.FBL_ERR_LAYOUT
    # alignment
    assert _fwd(lq, lk, lv, lo, dict(p, k=p["k"] + 2)) == E.FBL_ERR_ALIGN
    # mask
    assert _fwd(lq, lk, lv, lo, p, kind=F.FBL_MASK_KEY_PADDING, kv_len=None) == E.FBL_ERR_NULL
    assert _fwd(lq, lk, lv, lo, p, kind=8) == E.FBL_ERR_ARG
    # scale
    assert _fwd(lq, lk, lv, lo, p, scale=float("nan")) == E.FBL_ERR_ARG
    assert _fwd(lq, lk, lv, lo, p, scale=float("inf")) == E.FBL_ERR_ARG
    # cross-attention (S_kv != S_q) takes no causal mask
    lk8, lv8 = _copy(lk, S=8, sb=8 * 128), _copy(lv, S=8, sb=8 * 128)
    assert _fwd(lq, lk8, lv8, lo, p, kind=F.FBL_MASK_CAUSAL) == E.FBL_ERR_UNSUPPORTED
    assert _fwd(lq, lk8, lv8, lo, p, kind=F.FBL_MASK_CAUSAL | F.FBL_MASK_KEY_PADDING, kv_len=64) \
        == E.FBL_ERR_UNSUPPORTED
    # output aliasing an input
    assert _fwd(lq, lk, lv, lo, dict(p, o=p["q"])) == E.FBL_ERR_ARG
    assert _fwd(lq, lk, lv, lo, dict(p, lse=p["v"] + 64)) == E.FBL_ERR_ARG


def _bwd_setup(D=64, dtype=BF16):
    lq, lk, lv, lo, p = _fwd_setup(dtype=dtype, D=D)
    B, S, Hq, Hkv = 2, 16, 4, 2
    es = 2 if dtype == BF16 else 4
    nq = B * S * Hq * D * es
    nk = B * S * Hkv * D * es
    base = p["lse"] + 4096 * 4
    p.update({"do": base, "dq": base + nq + 4096, "dk": base + 2 * nq + 8192, "dv": base + 2 * nq + nk + 12288})
    p["ws"] = p["dv"] + nk + 4096
    p["ws"] = (p["ws"] + 255) // 256 * 256
    ws_bytes = fbl.fbl_attn_bwd_workspace(lq, lk)
    return lq, lk, lv, lo, p, ws_bytes


def _bwd(lq, lk, lv, lo, p, ws_bytes, ldo=None, ldq=None, ldk=None, ldv=None, kind=0, kv_len=None, scale=0.1):
    ldo = ldo or lo
    ldq = ldq or lq
    ldk = ldk or lk
    ldv = ldv or lv
    return fbl.fbl_attn_bwd_raw(lq, p["q"], lk, p["k"], lv, p["v"], lo, p["o"], ldo, p["do"], p["lse"], scale,
                                F.Mask(kind, 0, kv_len), ldq, p["dq"], ldk, p["dk"], ldv, p["dv"], p["ws"],
                                ws_bytes, stream=0)


def test_row_offset_limit():
    """Every attention tensor's rows are addressed with 32-bit offsets from
    its (batch, head) base, tiles reaching 128 rows past the last token:
    (S + 128) * ss * element size must stay within 2^31 bytes, for inputs and
    outputs alike (each layout carries its own row stride)."""
    E = F
    S = 16
    big = 1 << 23    # (16 + 128) * 2^23 * 2 bytes > 2^31, yet the 16 rows span only 0.25 GB
    lq, lk, lv, lo, p = _fwd_setup(S=S)
    wide = lambda l: _copy(l, ss=big, sb=S * big)
    for role in ("q", "k", "v", "o"):
        ls = {"q": lq, "k": lk, "v": lv, "o": lo}
        ls[role] = wide(ls[role])
        assert _fwd(ls["q"], ls["k"], ls["v"], ls["o"], p) == E.FBL_ERR_UNSUPPORTED, role
    lq, lk, lv, lo, p, ws = _bwd_setup()
    for kw in ({"ldo": wide(lo)}, {"ldq": wide(lq)}, {"ldk": wide(lk)}, {"ldv": wide(lv)}):
        assert _bwd(lq, lk, lv, lo, p, ws, **kw) == E.FBL_ERR_UNSUPPORTED, kw
    assert _bwd(lq, lk, lv, wide(lo), p, ws, ldo=lo) == E.FBL_ERR_UNSUPPORTED


def kv_split(B, Sq, Skv, Hq, Hkv, D):
    """The key/value pass split rule under a causal mask, restated: items are
    key blocks of 128 per (batch, kv head); split 2 (then 4) while there are
    fewer than 512 items and the first key block keeps 16 iterations (of 32
    queries, 64 at D = 32) per share."""
    items = -(-Skv // 128) * Hkv * B
    iters = Hq // Hkv * -(-Sq // (64 if D == 32 else 32))
    split = 1
    while split < 4 and items * split < 512 and iters >= 16 * split:
        split *= 2
    return split


def test_bwd_workspace_size():
    """Minimum: the row statistics, [B, Hq, 2, S] fp32 rounded up to 256 bytes.
    Full (bf16): plus B*Hq*ceil(S/32)^2 dS blocks of 2 KB, plus, when the
    key/value pass is split, the fp32 partial dK and dV [2][split][B, S, Hkv, D];
    fp32: statistics only."""
    for dt, with_ds in ((BF16, True), (F32, False)):
        for S in (16, 100, 1024):
            lq = fbl.fbl_layout_desc(dt, 2, S, 6, 64)
            lk = fbl.fbl_layout_desc(dt, 2, S, 3, 64)
            stats = (2 * 6 * S * 2 * 4 + 255) // 256 * 256
            assert fbl.fbl_attn_bwd_workspace_min(lq, lk) == stats
            nb = (S + 31) // 32
            split = kv_split(2, S, S, 6, 3, 64)
            part = 2 * split * 2 * S * 3 * 64 * 4 if split > 1 else 0
            assert fbl.fbl_attn_bwd_workspace(lq, lk) == stats + ((2 * 6 * nb * nb * 2048 + part) if with_ds else 0)
    assert kv_split(2, 1024, 1024, 6, 3, 64) == 4 and kv_split(2, 100, 100, 6, 3, 64) == 1
    # the Llama-3.2-1B-like GQA shape: 256 items, split in two; the Llama-7B-like shape: 1024 items, no split
    assert kv_split(2, 2048, 2048, 32, 8, 64) == 2 and kv_split(1, 4096, 4096, 32, 32, 128) == 1
    for (B, S, Hq, Hkv, D) in ((2, 2048, 32, 8, 64), (1, 4096, 32, 32, 128), (4, 1024, 16, 16, 64)):
        lq, lk = fbl.fbl_layout_desc(BF16, B, S, Hq, D), fbl.fbl_layout_desc(BF16, B, S, Hkv, D)
        nb = (S + 31) // 32
        rest = fbl.fbl_attn_bwd_workspace(lq, lk) - fbl.fbl_attn_bwd_workspace_min(lq, lk) - B * Hq * nb * nb * 2048
        split = kv_split(B, S, S, Hq, Hkv, D)
        assert rest == (2 * split * B * S * Hkv * D * 4 if split > 1 else 0), (B, S, Hq, Hkv, D)
    # cross-attention: statistics per query row, dS blocks ceil(S_q/32) x ceil(S_kv/32)
    lq = fbl.fbl_layout_desc(BF16, 2, 100, 6, 64)
    lk = fbl.fbl_layout_desc(BF16, 2, 70, 3, 64)
    stats = (2 * 6 * 100 * 2 * 4 + 255) // 256 * 256
    assert fbl.fbl_attn_bwd_workspace_min(lq, lk) == stats
    assert fbl.fbl_attn_bwd_workspace(lq, lk) == stats + 2 * 6 * 4 * 3 * 2048
    # one head's dS blocks would reach 2 GiB: no stored-dS part
    lq = fbl.fbl_layout_desc(BF16, 1, 32768, 1, 64)
    assert fbl.fbl_attn_bwd_workspace(lq, lq) == fbl.fbl_attn_bwd_workspace_min(lq, lq)


def test_bwd_rejections():
    lq, lk, lv, lo, p, ws = _bwd_setup()
    E = F
    assert _bwd(lq, lk, lv, lo, dict(p, do=None), ws) == E.FBL_ERR_NULL
    assert _bwd(lq, lk, lv, lo, dict(p, dk=None), ws) == E.FBL_ERR_NULL
    assert _bwd(lq, lk, lv, lo, dict(p, ws=None), ws) == E.FBL_ERR_WORKSPACE
    ws_min = fbl.fbl_attn_bwd_workspace_min(lq, lk)
    assert _bwd(lq, lk, lv, lo, p, ws_min - 256) == E.FBL_ERR_WORKSPACE
    assert _bwd(lq, lk, lv, lo, dict(p, ws=p["ws"] + 16), ws) == E.FBL_ERR_ALIGN
    assert _bwd(lq, lk, lv, lo, p, ws, ldq=_copy(lq, dtype=F32)) == E.FBL_ERR_DTYPE
    assert _bwd(lq, lk, lv, lo, p, ws, ldk=_copy(lq)) == E.FBL_ERR_SHAPE
    assert _bwd(lq, lk, lv, lo, p, ws, ldv=_copy(lv, sd=3)) == E.FBL_ERR_LAYOUT
    assert _bwd(lq, lk, lv, lo, dict(p, dq=p["do"]), ws) == E.FBL_ERR_ARG      # output aliases input
    assert _bwd(lq, lk, lv, lo, dict(p, dv=p["dk"]), ws) == E.FBL_ERR_ARG      # outputs alias each other
    assert _bwd(lq, lk, lv, lo, dict(p, dq=p["ws"]), ws) == E.FBL_ERR_ARG      # output aliases workspace
    # the workspace overlapping an input or the saved LSE
    for name in ("q", "k", "v", "o", "do"):
        assert _bwd(lq, lk, lv, lo, dict(p, ws=(p[name] + 255) // 256 * 256), ws) == E.FBL_ERR_ARG, name
    assert _bwd(lq, lk, lv, lo, dict(p, ws=p["lse"] // 256 * 256), ws) == E.FBL_ERR_ARG
    assert _bwd(lq, lk, lv, lo, p, ws, kind=F.FBL_MASK_KEY_PADDING) == E.FBL_ERR_NULL
    assert _bwd(lq, lk, lv, lo, p, ws, scale=float("nan")) == E.FBL_ERR_ARG
    assert _bwd(lq, lk, lv, lo, dict(p, lse=p["lse"] + 4), ws) == E.FBL_ERR_ALIGN
    # phase masks: none, or a bit outside FBL_BWD_ALL
    for ph in (0, 8, F.FBL_BWD_ALL | 16):
        assert fbl.fbl_attn_bwd_raw(lq, p["q"], lk, p["k"], lv, p["v"], lo, p["o"], lo, p["do"], p["lse"], 0.1,
                                    F.Mask(0, 0, None), lq, p["dq"], lk, p["dk"], lv, p["dv"], p["ws"], ws,
                                    stream=0, phases=ph) == E.FBL_ERR_ARG, ph


def test_layout_map_device_rejects_null():
    l = fbl.fbl_layout_desc(BF16, 1, 4, 2, 32)
    assert F.LIB.fbl_layout_map_device(ctypes.byref(l), None, None) == F.FBL_ERR_NULL
    assert F.LIB.fbl_layout_map_device(None, FAKE, None) == F.FBL_ERR_NULL


def test_bwd_rejects_overlapping_packed_views():
    """Column views of one packed gradient buffer: interleaved but disjoint views
    are legal (exercised on the GPU); views sharing columns are rejected here."""
    lq, lk, lv, lo, p, ws = _bwd_setup()
    B, S, Hq, Hkv, D = 2, 16, 4, 2, 64
    row = (Hq + 2 * Hkv) * D
    ldq = fbl.fbl_layout_desc(BF16, B, S, Hq, D, row_stride=row)
    ldk = fbl.fbl_layout_desc(BF16, B, S, Hkv, D, row_stride=row)
    ldv = fbl.fbl_layout_desc(BF16, B, S, Hkv, D, row_stride=row)
    base = p["ws"] + ws + 4096 * 16
    # dk starts one head early: shares dq's last head columns
    bad = dict(p, dq=base, dk=base + (Hq - 1) * D * 2, dv=base + (Hq + Hkv) * D * 2)
    assert _bwd(lq, lk, lv, lo, bad, ws, ldq=ldq, ldk=ldk, ldv=ldv) == F.FBL_ERR_ARG
    # dv starts inside dk's columns
    bad = dict(p, dq=base, dk=base + Hq * D * 2, dv=base + (Hq + 1) * D * 2)
    assert _bwd(lq, lk, lv, lo, bad, ws, ldq=ldq, ldk=ldk, ldv=ldv) == F.FBL_ERR_ARG


@pytest.mark.parametrize("B,S,Hq,Hkv,D,bstride", [(2, 5, 4, 2, 64, 0), (3, 7, 6, 3, 32, 0), (2, 4, 8, 8, 128, 0),
                                                   (2, 6, 4, 1, 64, 6 * 6 * 64 + 128)])
def test_packed_qkv_descriptors_bit_exact(B, S, Hq, Hkv, D, bstride):
    """fbl_layout_packed_qkv + fbl_layout_offset against the oracle's split of
    a packed projection output (numpy slicing of flat indices)."""
    import numpy as np
    import oracle
    lq, lk, lv, ko, vo = fbl.fbl_layout_packed_qkv(BF16, B, S, Hq, Hkv, D, batch_stride=bstride)
    W = (Hq + 2 * Hkv) * D
    assert (lq.ss, lk.ss, lv.ss) == (W, W, W) and (ko, vo) == (Hq * D, (Hq + Hkv) * D)
    assert lq.sb == (bstride or S * W)
    want = oracle.packed_qkv_offsets(B, S, Hq, Hkv, D)
    if bstride:  # batches further apart than S rows: shift the oracle's batch index
        want = tuple(x - (np.arange(B)[:, None, None, None] * S * W) + np.arange(B)[:, None, None, None] * bstride
                     for x in want)
    for l, off, base in ((lq, want[0], 0), (lk, want[1], ko), (lv, want[2], vo)):
        got = np.zeros_like(off)
        for b, h, s, i in np.ndindex(*off.shape):
            got[b, h, s, i] = base + fbl.fbl_layout_offset(l, b, h, s, i)
        assert np.array_equal(got, off)


def test_packed_qkv_rejections():
    st = F.LIB.fbl_layout_packed_qkv(None, None, None, None, None, BF16, 1, 1, 1, 1, 64, 0, 0)
    assert st == F.FBL_ERR_NULL
    with pytest.raises(F.FblError) as e:
        fbl.fbl_layout_packed_qkv(BF16, 2, 4, 0, 1, 64)
    assert e.value.status == F.FBL_ERR_SHAPE
    with pytest.raises(F.FblError) as e:
        fbl.fbl_layout_packed_qkv(BF16, 2, 4, 4, 2, 64, tile_d=48)
    assert e.value.status == F.FBL_ERR_LAYOUT
    with pytest.raises(F.FblError) as e:
        fbl.fbl_layout_packed_qkv(BF16, 2, 4, 4, 2, 64, batch_stride=100)  # batches overlap
    assert e.value.status == F.FBL_ERR_LAYOUT


# ------------------------------------------------------ projection products
def test_proj_rejections():
    P = lambda op, M, K, N, a=FAKE, lda=None, b=FAKE + (1 << 24), ldb=None, c=FAKE + (1 << 26), ldc=None, tile=-1: \
        fbl.fbl_proj_raw(op, M, K, N, a, lda if lda is not None else 4096, b, ldb if ldb is not None else 4096, c,
                         ldc if ldc is not None else 4096, tile, stream=0)
    E = F
    assert P(3, 64, 64, 64) == E.FBL_ERR_ARG                       # unknown op
    assert P(E.FBL_PROJ_FWD, 64, 64, 64, a=None) == E.FBL_ERR_NULL
    assert P(E.FBL_PROJ_FWD, 0, 64, 64) == E.FBL_ERR_SHAPE
    assert P(E.FBL_PROJ_FWD, 64, 64, 64, lda=32) == E.FBL_ERR_LAYOUT  # lda < K
    assert P(E.FBL_PROJ_BWD_DATA, 64, 64, 128, lda=64) == E.FBL_ERR_LAYOUT  # dY rows hold N
    assert P(E.FBL_PROJ_FWD, 64, 64, 64, a=FAKE + 2) == E.FBL_ERR_ALIGN
    assert P(E.FBL_PROJ_FWD, 64, 64, 64, lda=4100) == E.FBL_ERR_ALIGN  # row not 16-byte aligned
    assert P(E.FBL_PROJ_FWD, 64, 60, 64) == E.FBL_ERR_UNSUPPORTED     # contraction not a multiple of 8
    assert P(E.FBL_PROJ_BWD_WEIGHT, 100, 64, 64) == E.FBL_ERR_UNSUPPORTED  # contraction M = 100
    assert P(E.FBL_PROJ_FWD, 64, 64, 66, ldc=4104) == E.FBL_ERR_UNSUPPORTED  # output columns not a multiple of 4
    assert P(E.FBL_PROJ_BWD_DATA, 64, 66, 64) == E.FBL_ERR_UNSUPPORTED  # dX columns K = 66
    assert P(E.FBL_PROJ_FWD, 64, 64, 64, tile=21) == E.FBL_ERR_ARG    # no such tile id
    assert P(E.FBL_PROJ_FWD, 64, 64, 64, tile=-2) == E.FBL_ERR_ARG
    assert P(E.FBL_PROJ_FWD, 64, 64, 64, c=FAKE + 64) == E.FBL_ERR_ARG  # output overlaps an input


def test_gemm_tile_table():
    """The tile table the GPU tests enumerate: 21 configurations, ids 0-3 the
    named output shapes, LDS within the 160 KB of a CU, and the contraction
    split and wavefront grid consistent with the output tile."""
    tiles = fbl.gemm_tiles()
    assert len(tiles) == 21 and fbl.LIB.fbl_gemm_tile_count() == 21
    named = {F.FBL_GEMM_TILE_128x128: (128, 128), F.FBL_GEMM_TILE_128x64: (128, 64),
             F.FBL_GEMM_TILE_64x128: (64, 128), F.FBL_GEMM_TILE_64x64: (64, 64)}
    for t, (bm, bn) in named.items():
        assert (tiles[t]["bm"], tiles[t]["bn"]) == (bm, bn)
    for t, g in tiles.items():
        assert g["wm"] * g["wn"] * g["wk"] in (4, 8)
        assert g["bm"] % (32 * g["wm"]) == 0 and g["bn"] % (32 * g["wn"]) == 0
        assert (g["bk"] // 16) % g["wk"] == 0
        stages = g["stages"] * (g["bm"] + g["bn"]) * g["bk"] * 2
        partial = (g["wk"] - 1) * g["bm"] * g["bn"] * 4
        assert g["lds_bytes"] == max(stages, partial) <= 160 * 1024
    info = (ctypes.c_int32 * 8)()
    assert fbl.LIB.fbl_gemm_tile_info(21, info) == F.FBL_ERR_ARG
    assert fbl.LIB.fbl_gemm_tile_info(0, None) == F.FBL_ERR_NULL


def test_proj_candidates_filters():
    """C2 keeps staged rows that are whole 128-byte lines (or span the whole
    stored row of a narrower operand); C3 keeps tiles that pad every extent by
    at most 10%, and falls back to the least padded volume.  At 512 x 2048 x
    8192: the forward (A row-read: bk elements per row; B row-read: bn) keeps
    bk >= 64 and bn >= 64; the data gradient (both operands staged with bk
    per row) keeps bk >= 64; the weight gradient (both transposed: bm, bn per
    row) keeps bm >= 64 and bn >= 64."""
    tiles = fbl.gemm_tiles()
    M, K, N = 512, 2048, 8192
    fwd = fbl.proj_candidates(F.FBL_PROJ_FWD, M, K, N)
    assert fwd == [t for t in sorted(tiles) if tiles[t]["bk"] >= 64 and tiles[t]["bn"] >= 64]
    assert fbl.proj_candidates(F.FBL_PROJ_BWD_DATA, M, K, N) == [t for t in sorted(tiles) if tiles[t]["bk"] >= 64]
    assert fbl.proj_candidates(F.FBL_PROJ_BWD_WEIGHT, M, K, N) == \
        [t for t in sorted(tiles) if tiles[t]["bm"] >= 64 and tiles[t]["bn"] >= 64]
    # 192 output rows: 128-row tiles pad by 33%
    assert all(tiles[t]["bm"] <= 64 for t in fbl.proj_candidates(F.FBL_PROJ_FWD, 192, 128, 256))
    # contraction 96: every depth pads by 33%; least padded volume among C1/C2 survivors (bk 64 or 128 with
    # 64 x 64 output; 32-deep steps fail C2 and 32-column tiles stage 64-byte rows of a 128-byte-wide B)
    assert fbl.proj_candidates(F.FBL_PROJ_FWD, 64, 96, 64) == [7, 9]
    # LoRA, rank 16: X A (2048 -> 16), H B (16 -> 2048) and the gradients
    assert fbl.proj_candidates(F.FBL_PROJ_FWD, 512, 2048, 16) == [13, 14, 16]      # narrow output columns
    assert fbl.proj_candidates(F.FBL_PROJ_FWD, 512, 16, 2048) == [0, 1, 2, 3, 17]  # contraction 16: 32-deep steps
    assert fbl.proj_candidates(F.FBL_PROJ_BWD_WEIGHT, 512, 16, 2048) == [15]        # dB: 16 output rows
    assert fbl.proj_candidates(F.FBL_PROJ_BWD_WEIGHT, 512, 2048, 16) == [13, 14]    # dA: 16 output columns
    n = ctypes.c_int32()
    assert fbl.LIB.fbl_proj_candidates(F.FBL_PROJ_FWD, M, K, N, None, 0, ctypes.byref(n)) == F.FBL_OK
    assert n.value == len(fwd)
    assert fbl.LIB.fbl_proj_candidates(3, M, K, N, None, 0, ctypes.byref(n)) == F.FBL_ERR_ARG
    assert fbl.LIB.fbl_proj_candidates(F.FBL_PROJ_FWD, 0, K, N, None, 0, ctypes.byref(n)) == F.FBL_ERR_SHAPE
    assert fbl.LIB.fbl_proj_candidates(F.FBL_PROJ_FWD, M, K, N, None, 4, ctypes.byref(n)) == F.FBL_ERR_NULL


def test_proj_auto_tile_measured_regimes():
    """FBL_GEMM_TILE_AUTO without a tuned entry follows the measured preference
    orders: 256 x 256 tiles from 1024 output tiles of 128 x 128 with a long
    contraction (8 wavefronts for row-read A, 4 for the weight gradient; 128 x
    128 with a short one), the
    8-wavefront 256 x 128 tile from 384, 64 x 128 from 256, the deep-contraction
    split tile below; the choice is always a candidate."""
    fbl.proj_tune_reset()
    A = fbl.proj_auto_tile
    FWD, BD, BW = F.FBL_PROJ_FWD, F.FBL_PROJ_BWD_DATA, F.FBL_PROJ_BWD_WEIGHT
    assert A(FWD, 4096, 4096, 12288) == 19 and A(BD, 4096, 4096, 12288) == 19
    assert A(BW, 4096, 4096, 12288) == 18 and A(BW, 2048, 4096, 4096) == 18
    assert A(BW, 512, 4096, 12288) == 0                      # 3072 output tiles, contraction 512
    assert A(FWD, 512, 4096, 12288) == 11 and A(FWD, 2048, 4096, 4096) == 11   # 384 and 512 output tiles
    assert A(BD, 2048, 4096, 4096) == 12 and A(BW, 4096, 2048, 4096) == 0     # 512 output tiles
    assert A(FWD, 512, 2048, 8192) == 6                      # 256 output tiles
    assert A(BD, 512, 4096, 12288) == 10                     # 128 output tiles, a grid of 256
    assert A(BD, 512, 2048, 8192) == 9                       # 64 output tiles: the 64 x 64 split tile fills the CUs
    for op, M, K, N in ((FWD, 512, 2048, 16), (BW, 512, 16, 2048), (FWD, 64, 96, 64), (BD, 192, 128, 256)):
        assert A(op, M, K, N) in fbl.proj_candidates(op, M, K, N)
    t = ctypes.c_int32()
    assert fbl.LIB.fbl_proj_auto_tile(FWD, 64, 64, 64, None) == F.FBL_ERR_NULL
    assert fbl.LIB.fbl_proj_auto_tile(3, 64, 64, 64, ctypes.byref(t)) == F.FBL_ERR_ARG
    assert fbl.LIB.fbl_proj_auto_tile(FWD, 0, 64, 64, ctypes.byref(t)) == F.FBL_ERR_SHAPE


def test_proj_tune_rejections():
    """Argument checks that return before any GPU work."""
    T = lambda op=0, obj=0, reps=5, a=FAKE: fbl.LIB.fbl_proj_tune(
        op, 64, 64, 64, ctypes.c_void_p(a) if a else None, 4096, ctypes.c_void_p(FAKE + (1 << 24)), 4096,
        ctypes.c_void_p(FAKE + (1 << 26)), 4096, obj, reps, None, None, None)
    assert T(op=3) == F.FBL_ERR_ARG
    assert T(a=0) == F.FBL_ERR_NULL
    assert T(obj=2) == F.FBL_ERR_ARG
    assert T(reps=0) == F.FBL_ERR_ARG
    assert T(reps=1001) == F.FBL_ERR_ARG
    assert fbl.proj_tuned_tile(F.FBL_PROJ_FWD, 64, 64, 64) == -1


def test_proj_dt_rejections():
    """fbl_proj_dt: the dtype, the single fp32 tile and fp32's natural alignment."""
    D = lambda op=0, dt=F.FBL_F32, a=FAKE, lda=4096, tile=-1, M=64, K=64, N=64: fbl.LIB.fbl_proj_dt(
        op, dt, M, K, N, ctypes.c_void_p(a), lda, ctypes.c_void_p(FAKE + (1 << 24)), 4096,
        ctypes.c_void_p(FAKE + (1 << 26)), 4096, tile, None)
    assert D(dt=7) == F.FBL_ERR_DTYPE
    assert D(tile=0) == F.FBL_ERR_ARG                  # fp32 has one tile shape
    assert D(a=FAKE + 2) == F.FBL_ERR_ALIGN            # fp32 needs 4-byte alignment
    assert D(lda=32) == F.FBL_ERR_LAYOUT
    assert D(op=3) == F.FBL_ERR_ARG
    assert D(M=0) == F.FBL_ERR_SHAPE
    # bf16 through fbl_proj_dt keeps fbl_proj's rules
    assert D(dt=F.FBL_BF16, K=60) == F.FBL_ERR_UNSUPPORTED
    assert D(dt=F.FBL_BF16, a=FAKE + 4) == F.FBL_ERR_ALIGN


# ---------------------------------------------- the Python binding's own checks
def test_binding_rejects_kv_len_and_host_tensors():
    """The binding hands raw pointers to the kernels, so it checks what the C
    ABI cannot see: kv_len is int32 with unit stride and at least B entries,
    and every tensor is on the GPU (a host pointer would be read on the
    device).  All of this raises before any library call."""
    import torch
    B, S, H, D = 2, 16, 2, 64
    q = torch.zeros(B, S, H * D, dtype=torch.bfloat16)
    for bad, status in ((torch.tensor([100, 37], dtype=torch.int64), F.FBL_ERR_DTYPE),
                        (torch.tensor([5], dtype=torch.int32), F.FBL_ERR_SHAPE),
                        (torch.tensor([[5, 6]], dtype=torch.int32), F.FBL_ERR_LAYOUT),
                        (torch.tensor([5, 0, 6, 0], dtype=torch.int32)[::2], F.FBL_ERR_LAYOUT),
                        ([5, 6], F.FBL_ERR_ARG)):
        with pytest.raises(F.FblError) as ei:
            F.attn_fwd(q, q, q, H, H, kv_len=bad)
        assert ei.value.status == status, bad
        with pytest.raises(F.FblError) as ei:
            F.attn_bwd(q, q, q, q, q, None, H, H, kv_len=bad)
        assert ei.value.status == status, bad
    # host tensors: q itself, or an int32 kv_len left on the host
    ok_len = torch.tensor([5, 6], dtype=torch.int32)
    for call in (lambda: F.attn_fwd(q, q, q, H, H),
                 lambda: F.attn_fwd(q, q, q, H, H, kv_len=ok_len),
                 lambda: F.attn_bwd(q, q, q, q, q, torch.zeros(B, H, S), H, H),
                 lambda: F.attn_fwd_packed(torch.zeros(B, S, 3 * H * D, dtype=torch.bfloat16), H, H),
                 lambda: F.proj(F.FBL_PROJ_FWD, torch.zeros(4, 8, dtype=torch.bfloat16),
                                torch.zeros(8, 4, dtype=torch.bfloat16))):
        with pytest.raises(F.FblError) as ei:
            call()
        assert ei.value.status == F.FBL_ERR_ARG


def test_binding_checks_lse_and_workspace():
    """The saved log-sum-exp and the workspace reach the kernels as raw spans:
    lse must be a contiguous float32 [B, Hq, S_q] tensor and the workspace
    contiguous, else the binding raises (the kernels would read or write past
    them)."""
    import torch
    B, Hq, S = 2, 4, 16
    F._check_lse(None, B, Hq, S, "t")
    F._check_lse(torch.zeros(B, Hq, S), B, Hq, S, "t")
    for bad, status in ((torch.zeros(B, Hq, S, dtype=torch.bfloat16), F.FBL_ERR_DTYPE),
                        (torch.zeros(B, Hq, S - 1), F.FBL_ERR_SHAPE),
                        (torch.zeros(B * Hq * S), F.FBL_ERR_SHAPE),
                        (torch.zeros(B, S, Hq).transpose(1, 2), F.FBL_ERR_LAYOUT),
                        ([0.0] * (B * Hq * S), F.FBL_ERR_ARG)):
        with pytest.raises(F.FblError) as ei:
            F._check_lse(bad, B, Hq, S, "t")
        assert ei.value.status == status
    F._check_workspace(torch.zeros(1024, dtype=torch.uint8), "t")
    with pytest.raises(F.FblError) as ei:
        F._check_workspace(torch.zeros(2048, dtype=torch.uint8)[::2], "t")
    assert ei.value.status == F.FBL_ERR_LAYOUT


def test_autograd_rejects_broadcast_gradient():
    """The autograd wrappers read the incoming gradient in place; a broadcast
    view (inner stride 0) is refused instead of silently copied."""
    import torch
    from paper_2607_21624_amd import autograd as ag
    g = torch.zeros(1, dtype=torch.bfloat16).expand(2, 4, 64)
    with pytest.raises(F.FblError) as ei:
        ag._unit(g, "attention")
    assert ei.value.status == F.FBL_ERR_LAYOUT
    t = torch.zeros(2, 4, 64, dtype=torch.bfloat16)
    assert ag._unit(t, "attention") is t
    assert ag._unit(t[:, :, :32], "attention").data_ptr() == t.data_ptr()  # strided rows pass as views


def test_noalloc_rejects_too_many_rows():
    """fbl_attn_bwd_noalloc with more query rows than its scratch holds
    statistics for: FBL_ERR_WORKSPACE, before any HIP call."""
    macro = re.search(r"#define FBL_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", open(HEADER).read())
    assert int(macro.group(1)) << int(macro.group(2)) == fbl.NOALLOC_SCRATCH_BYTES
    rows = fbl.NOALLOC_SCRATCH_BYTES // 8 + 256
    lq = fbl.fbl_layout_desc(fbl.FBL_BF16, 1, rows // 64, 64, 64)
    lk = fbl.fbl_layout_desc(fbl.FBL_BF16, 1, rows // 64, 64, 64)
    assert fbl.fbl_attn_bwd_workspace_min(lq, lk) > fbl.NOALLOC_SCRATCH_BYTES
    st = F.fbl_attn_bwd_noalloc_raw(lq, FAKE, lk, FAKE, lk, FAKE, lq, FAKE, lq, FAKE, FAKE, 0.1, F.Mask(0, 0, None),
                                    lq, FAKE, lk, FAKE, lk, FAKE, stream=0)
    assert st == F.FBL_ERR_WORKSPACE


# ------------------------------------------------------ attention tile table
def _attn_c123(t, D, Sq, Skv):
    """The three candidate filters restated from their definitions: C1 whole
    32x32 MFMA blocks per wavefront and staged tile, 16-deep chunks over d,
    2-8 wavefronts; C2 LDS per CU, whole 1 KB loads spread evenly, registers
    within a wavefront's share of the file; C3 padding at most 10%."""
    c1 = t["per_wave"] % 32 == 0 and t["cols"] % 32 == 0 and D % 16 == 0 and 2 <= t["waves"] <= 8
    pad = lambda n, m: -(-n // m) * m
    rows_seq, cols_seq = (Skv, Sq) if t["pass"] == F.FBL_ATTN_BWD_KV else (Sq, Skv)
    c3 = 10 * (pad(rows_seq, t["rows"]) - rows_seq) <= rows_seq and 10 * (pad(cols_seq, t["cols"]) - cols_seq) <= cols_seq
    return c1 and t["legal"] == 1, c3, pad(rows_seq, t["rows"]) * pad(cols_seq, t["cols"])


@pytest.mark.parametrize("D", [32, 64, 128])
def test_attn_tile_table_and_filters(D):
    tiles = fbl.attn_tiles(D)
    assert len(tiles) == F.LIB.fbl_attn_tile_count()
    for t, i in tiles.items():
        assert i["rows"] == i["per_wave"] * i["waves"] and i["lds_bytes"] * i["occupancy"] <= 160 * 1024, (t, i)
    # every pass has a runnable tile at every head dim
    for p in (F.FBL_ATTN_FWD, F.FBL_ATTN_BWD_KV, F.FBL_ATTN_BWD_DQ):
        assert any(i["pass"] == p and i["legal"] for i in tiles.values())
    # kv tiles staging 64-query blocks do not fit the registers at d = 128; 32-query
    # blocks at d = 32 (2 KB) are half a 1 KB load per wavefront of a 4-wavefront workgroup
    kv = {t: i for t, i in tiles.items() if i["pass"] == F.FBL_ATTN_BWD_KV}
    for t, i in kv.items():
        short = D == 32 and i["cols"] == 32 and i["waves"] == 4
        assert i["legal"] == (not (D == 128 and i["cols"] == 64) and not short), (D, t)
    for Sq, Skv in ((4096, 4096), (200, 200), (1024, 1024), (448, 300), (128, 128), (64, 64)):
        lq = fbl.fbl_layout_desc(BF16, 2, Sq, 4, D)
        lk = fbl.fbl_layout_desc(BF16, 2, Skv, 2, D)
        for p in (F.FBL_ATTN_FWD, F.FBL_ATTN_BWD_KV, F.FBL_ATTN_BWD_DQ):
            legal = {t: _attn_c123(i, D, Sq, Skv) for t, i in tiles.items() if i["pass"] == p}
            legal = {t: v for t, v in legal.items() if v[0]}
            want = sorted(t for t, v in legal.items() if v[1])
            if not want:  # C3 fallback: the least padded volume
                least = min(v[2] for v in legal.values())
                want = sorted(t for t, v in legal.items() if v[2] == least)
            assert fbl.attn_candidates(p, lq, lk) == want, (D, Sq, Skv, p)
        # the automatic choice (nothing tuned in this process) is a candidate of each pass
        auto = fbl.attn_auto_tiles(lq, lk, 1)
        for p, t in enumerate(auto):
            assert t in fbl.attn_candidates(p, lq, lk), (D, Sq, Skv, p, t)


def test_attn_tile_rejections():
    lq, lk, lv, lo, p = _fwd_setup(D=128)
    assert fbl.fbl_attn_fwd_raw(lq, p["q"], lk, p["k"], lv, p["v"], lo, p["o"], p["lse"], 0.1, F.Mask(0, 0, None),
                                stream=0, tile=5) == F.FBL_ERR_ARG  # a kv tile for the forward
    assert fbl.fbl_attn_fwd_raw(lq, p["q"], lk, p["k"], lv, p["v"], lo, p["o"], p["lse"], 0.1, F.Mask(0, 0, None),
                                stream=0, tile=99) == F.FBL_ERR_ARG
    lq, lk, lv, lo, p, ws = _bwd_setup(D=128)
    call = lambda kt, qt, phases=F.FBL_BWD_ALL, lq_=lq, lk_=lk, lv_=lv, lo_=lo: fbl.fbl_attn_bwd_raw(
        lq_, p["q"], lk_, p["k"], lv_, p["v"], lo_, p["o"], lo_, p["do"], p["lse"], 0.1, F.Mask(0, 0, None), lq_,
        p["dq"], lk_, p["dk"], lv_, p["dv"], p["ws"], ws, stream=0, phases=phases, kv_tile=kt, dq_tile=qt)
    assert call(6, -1) == F.FBL_ERR_UNSUPPORTED   # 64-query kv tiles exceed the registers at d = 128
    assert call(0, -1) == F.FBL_ERR_ARG           # a forward tile as the kv tile
    assert call(-1, 5) == F.FBL_ERR_ARG           # a kv tile as the dQ tile
    assert call(5, 7, phases=0) == F.FBL_ERR_ARG
    # fp32 storage: one configuration per pass, explicit ids refused
    lq, lk, lv, lo, p, ws = _bwd_setup(D=64, dtype=F32)
    assert call(5, -1, lq_=lq, lk_=lk, lv_=lv, lo_=lo) == F.FBL_ERR_ARG
    assert fbl.fbl_attn_fwd_raw(lq, p["q"], lk, p["k"], lv, p["v"], lo, p["o"], p["lse"], 0.1, F.Mask(0, 0, None),
                                stream=0, tile=0) == F.FBL_ERR_ARG
    info = (ctypes.c_int32 * 8)()
    assert F.LIB.fbl_attn_tile_info(0, 48, info) == F.FBL_ERR_UNSUPPORTED
    assert F.LIB.fbl_attn_tile_info(-1, 64, info) == F.FBL_ERR_ARG
    assert F.LIB.fbl_attn_tile_info(0, 64, None) == F.FBL_ERR_NULL
    with pytest.raises(F.FblError):
        fbl.attn_candidates(F.FBL_ATTN_FWD, fbl.fbl_layout_desc(F32, 1, 64, 2, 64), fbl.fbl_layout_desc(F32, 1, 64, 2, 64))


def test_bwd_launch_counts():
    """fbl_attn_bwd_launches: the one-launch backward up to 128 keys with
    automatic tiles (fp32 only at d <= 64), three launches otherwise, four
    where the key/value pass is split (its partial sums reduced by a fourth),
    one per phase bit when the phases are called one by one."""
    ALL, KV = F.FBL_BWD_ALL, F.FBL_BWD_KV

    def count(dt, B, Sq, Skv, Hq, Hkv, D, mask, ws="full", **kw):
        lq = fbl.fbl_layout_desc(dt, B, Sq, Hq, D)
        lk = fbl.fbl_layout_desc(dt, B, Skv, Hkv, D)
        n = {"full": fbl.fbl_attn_bwd_workspace, "min": fbl.fbl_attn_bwd_workspace_min}[ws](lq, lk)
        return fbl.attn_bwd_launches(lq, lk, mask, n, **kw)

    assert count(BF16, 8, 128, 128, 12, 12, 64, 2) == 1             # BERT-base-like, key padding
    assert count(BF16, 8, 128, 128, 12, 12, 64, 2, kv_tile=5) == 3  # a named tile: three launches
    assert count(BF16, 8, 128, 128, 12, 12, 64, 2, phases=KV) == 1
    assert count(BF16, 2, 300, 128, 4, 4, 128, 0) == 1              # cross attention, 128 keys
    assert count(BF16, 2, 129, 129, 4, 4, 64, 1) == 3               # one key too many
    # 128 keys but two (batch, head) pairs of 128 query blocks: the split three-launch path
    assert count(BF16, 1, 8192, 128, 2, 2, 64, 0) == 4
    assert count(BF16, 128, 8192, 128, 2, 1, 64, 0) == 1            # 128 pairs: one launch
    assert count(BF16, 1, 4096, 128, 2, 2, 64, 0) == 1              # 64 query blocks: one launch
    assert count(F32, 1, 64, 64, 2, 2, 32, 0) == 1
    assert count(F32, 1, 64, 64, 2, 2, 128, 0) == 3                 # fp32 at d = 128 does not fuse
    assert count(BF16, 1, 4096, 4096, 32, 32, 128, 1) == 3          # Llama-7B-like causal
    assert count(BF16, 2, 2048, 2048, 32, 8, 64, 1) == 4            # Llama-3.2-1B-like GQA: split kv pass
    assert count(BF16, 2, 2048, 2048, 32, 8, 64, 1, ws="min") == 3  # no dS store, no split
    assert count(BF16, 2, 2048, 2048, 32, 8, 64, 1, phases=KV) == 2
    lq = fbl.fbl_layout_desc(F32, 1, 64, 2, 32)
    n = ctypes.c_int32()
    assert F.LIB.fbl_attn_bwd_launches(0, ctypes.byref(lq), ctypes.byref(lq), 0, 1 << 20, -1, -1,
                                       ctypes.byref(n)) == F.FBL_ERR_ARG
    assert F.LIB.fbl_attn_bwd_launches(ALL, ctypes.byref(lq), ctypes.byref(lq), 0, 1 << 20, 5, -1,
                                       ctypes.byref(n)) == F.FBL_ERR_ARG    # fp32: automatic tiles only
    assert F.LIB.fbl_attn_bwd_launches(ALL, ctypes.byref(lq), ctypes.byref(lq), 0, 1 << 20, -1, -1,
                                       None) == F.FBL_ERR_NULL
    l48 = fbl.fbl_layout_desc(BF16, 1, 64, 2, 48)
    assert F.LIB.fbl_attn_bwd_launches(ALL, ctypes.byref(l48), ctypes.byref(l48), 0, 1 << 20, -1, -1,
                                       ctypes.byref(n)) == F.FBL_ERR_UNSUPPORTED
