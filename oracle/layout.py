"""Logical-to-physical index map of token-major tensors (oracle side).

The paper (section 4.3.1, Tile Propagation, with the multi-head attention
example) describes a projection output of logical shape (B, S, D) that is
reshaped to (B, S, H, HD) and then transposed to (B, H, S, HD) before the
attention matrix products.  The tile-based index transformation (section
4.3.2, the composed map f3 o f2 o f1) replaces the copies with one coordinate
map.  Here that map is produced by carrying out the chain on an array of flat
indices with numpy's own reshape and transpose, so the result is, by
construction, "where logical element (b, h, s, i) lives in memory".

Pins: tests/test_layout_oracle.py checks it against the closed affine form for the
paper's hidden=768 / 12 heads x 64 example and against explicit per-element
enumeration on ragged shapes.
"""
import numpy as np


def token_major_offsets(B: int, S: int, H: int, d: int) -> np.ndarray:
    """Offsets of a contiguous token-major [B, S, H*d] tensor, indexed [b, h, s, i].

    Chain: flat (B, S, H*d) --reshape--> (B, S, H, d) --transpose(0,2,1,3)-->
    (B, H, S, d).  Returns an int64 array of shape (B, H, S, d).
    """
    flat = np.arange(B * S * H * d, dtype=np.int64)
    return flat.reshape(B, S, H * d).reshape(B, S, H, d).transpose(0, 2, 1, 3)


def head_split_offsets(B: int, S: int, H: int, d: int, row_stride: int, batch_stride: int) -> np.ndarray:
    """Offsets when token rows are ``row_stride`` elements apart and batches
    ``batch_stride`` apart (e.g. one tensor viewed inside a wider packed
    projection output).  Built by the same reshape/transpose chain applied to a
    strided index grid.  Returns int64 (B, H, S, d).
    """
    b = np.arange(B, dtype=np.int64)[:, None, None] * batch_stride
    s = np.arange(S, dtype=np.int64)[None, :, None] * row_stride
    c = np.arange(H * d, dtype=np.int64)[None, None, :]
    grid = b + s + c                       # logical (B, S, H*d) -> physical offset
    return grid.reshape(B, S, H, d).transpose(0, 2, 1, 3)


def packed_qkv_offsets(B: int, S: int, Hq: int, Hkv: int, d: int):
    """Offsets of Q, K and V inside one packed projection output
    [B, S, (Hq + 2 Hkv) d] whose rows hold Hq query heads, then Hkv key heads,
    then Hkv value heads.  Built by splitting an array of flat indices of the
    packed tensor with numpy slicing, then the reshape/transpose chain.
    Returns three int64 arrays shaped (B, H, S, d)."""
    H = Hq + 2 * Hkv
    flat = np.arange(B * S * H * d, dtype=np.int64).reshape(B, S, H, d)
    q = flat[:, :, :Hq]
    k = flat[:, :, Hq:Hq + Hkv]
    v = flat[:, :, Hq + Hkv:]
    return tuple(x.transpose(0, 2, 1, 3) for x in (q, k, v))
