"""Pins of the oracle's logical -> physical index map (CPU)."""
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "layout_cases.json")


def _closed_form(B, S, H, d, b, h, s, i):
    # token-major: rows of H*d elements, batches of S rows
    return ((b * S + s) * H + h) * d + i


def test_paper_bert_example_closed_form():
    """hidden 768 = 12 heads x 64 (the paper's tile-boundary example), B=2, S=5."""
    B, S, H, d = 2, 5, 12, 64
    off = oracle.token_major_offsets(B, S, H, d)
    b, h, s, i = np.meshgrid(np.arange(B), np.arange(H), np.arange(S), np.arange(d), indexing="ij")
    assert np.array_equal(off, _closed_form(B, S, H, d, b, h, s, i))


@pytest.mark.parametrize("B,S,H,d", [(1, 1, 1, 1), (3, 7, 5, 3), (2, 13, 4, 32)])
def test_offsets_enumerated(B, S, H, d):
    off = oracle.token_major_offsets(B, S, H, d)
    # walk memory in order and check each element lands where its logical index says
    flat = 0
    for b in range(B):
        for s in range(S):
            for h in range(H):
                for i in range(d):
                    assert off[b, h, s, i] == flat
                    flat += 1


def test_strided_view_inside_packed_projection():
    """K as a view inside a packed [B, S, (Hq + 2 Hkv) d] projection output."""
    B, S, Hq, Hkv, d = 2, 6, 4, 2, 8
    row = (Hq + 2 * Hkv) * d
    packed = np.arange(B * S * row).reshape(B, S, row)
    k_view = packed[:, :, Hq * d:(Hq + Hkv) * d]
    off = oracle.head_split_offsets(B, S, Hkv, d, row_stride=row, batch_stride=S * row)
    want = k_view.reshape(B, S, Hkv, d).transpose(0, 2, 1, 3) - Hq * d
    assert np.array_equal(off, want)


def test_strength_reduction_identity_from_paper():
    cases = json.load(open(GOLDEN))["strength_reduction"]
    for c in cases:
        i = np.arange(0, 4 * c["Ca"] * c["Cb"] + 17, dtype=np.int64)
        assert c["Ca"] % c["Cb"] == 0
        assert np.array_equal((i % c["Ca"]) % c["Cb"], i % c["Cb"])


@pytest.mark.parametrize("B,S,Hq,Hkv,d", [(1, 1, 1, 1, 1), (2, 5, 4, 2, 8), (3, 7, 6, 3, 4), (2, 4, 12, 12, 64)])
def test_packed_qkv_offsets_closed_form(B, S, Hq, Hkv, d):
    """Packed [B, S, (Hq + 2 Hkv) d] rows: Q heads, then K heads, then V heads."""
    W = Hq + 2 * Hkv
    q, k, v = oracle.packed_qkv_offsets(B, S, Hq, Hkv, d)
    for off, H, first in ((q, Hq, 0), (k, Hkv, Hq), (v, Hkv, Hq + Hkv)):
        assert off.shape == (B, H, S, d)
        b, h, s, i = np.meshgrid(np.arange(B), np.arange(H), np.arange(S), np.arange(d), indexing="ij")
        assert np.array_equal(off, ((b * S + s) * W + first + h) * d + i)
    # together they cover every element of the packed tensor exactly once
    allo = np.concatenate([x.ravel() for x in (q, k, v)])
    assert np.array_equal(np.sort(allo), np.arange(B * S * W * d))
