"""Attention forward and backward in float64 numpy (oracle; test infrastructure only).

What is computed (the plain definition; the paper's method reaches the same
result, only without layout copies):

* The paper's attention module (section 2.2, the LoRA fine-tuning example)
  forms P = softmax(Q K^T) and multiplies by V.  The softmax scale is an
  explicit argument (1/sqrt(d) in every workload here).
* Heads come from the token-major projection output by the reshape/transpose
  chain of section 4.3.1; query head h reads key/value head floor(h / G) with
  G = Hq / Hkv (grouped-query attention, whose K/V expansion the same
  section mentions), i.e. repeat-interleave semantics.
* The backward pass is the chain rule applied to these definitions.  The paper
  states the matrix-product gradients (section 4.1, FTD-D; section 4.2: the
  forward reduces along K, the gradients along M or N) and classes softmax as
  forward-tensor-dependent with consistent access (section 4.1, FTD-C).  With
  L = sum(O * dO):
      dP = dO V^T,  D_i = sum_k dO_ik O_ik,  dS = P * (dP - D),
      dQ = scale dS K,  dK = scale dS^T Q,  dV = P^T dO,
  with dK and dV summed over the G query heads that share a key/value head.

Readings where the paper is silent (each listed with its reason in the design
notes of the repository):
* mask: key j is allowed for query i iff (not causal or j <= i) and
  (no key padding or j < kv_len[b]); a disallowed score is -inf (hard mask).
  Padded query rows are computed like any other row.
* a row with no allowed key has O = 0, LSE = -inf and no gradient.
* LSE is the natural-log log-sum-exp of the scaled, masked scores, [B, Hq, S_q].
* Cross-attention: queries (S_q tokens) and keys/values (S_k tokens) may
  differ in length (encoder-decoder attention, the layout-incompatible
  attention variant the paper lists among its workloads); the causal rule
  j <= i is then aligned at the first token of both.

Everything runs one (batch, head) at a time with full S_q x S_k matrices.
Inputs are upcast exactly to float64.

Pins (tests/test_oracle.py): scalar brute force (oracle/brute.py), float64
torch scaled_dot_product_attention with autograd, central finite differences of
sum(O * dO), closed forms (single key; Q = 0), shift/permutation invariances,
dV = P^T dO with P from brute force, D computed two ways, column-sum
invariants of dK and dV, and GQA equal to MHA on repeat-interleaved K/V.
"""
from __future__ import annotations

from typing import Optional

import numpy as np


def split_heads(x: np.ndarray, H: int) -> np.ndarray:
    """Token-major (B, S, H*d) -> logical (B, H, S, d) view, float64."""
    B, S, HD = x.shape
    d = HD // H
    return np.asarray(x, dtype=np.float64).reshape(B, S, H, d).transpose(0, 2, 1, 3)


def merge_heads(x: np.ndarray) -> np.ndarray:
    """Logical (B, H, S, d) -> token-major (B, S, H*d)."""
    B, H, S, d = x.shape
    return np.ascontiguousarray(x.transpose(0, 2, 1, 3)).reshape(B, S, H * d)


def kv_head_of(h: int, Hq: int, Hkv: int) -> int:
    """Key/value head read by query head h: contiguous groups of G = Hq/Hkv."""
    G = Hq // Hkv
    return h // G


def allowed_mask(S_q: int, S_k: int, causal: bool, kv_len_b: Optional[int]) -> np.ndarray:
    """Boolean (S_q, S_k): True where key j may be attended by query i."""
    i = np.arange(S_q)[:, None]
    j = np.arange(S_k)[None, :]
    m = np.ones((S_q, S_k), dtype=bool)
    if causal:
        m &= j <= i
    if kv_len_b is not None:
        m &= j < kv_len_b
    return m


def masked_scores(qh: np.ndarray, kh: np.ndarray, scale: float, allowed: np.ndarray) -> np.ndarray:
    """s_ij = scale * q_i . k_j where allowed, -inf elsewhere."""
    s = scale * (qh @ kh.T)
    return np.where(allowed, s, -np.inf)


def softmax_rows(s: np.ndarray):
    """Row softmax of masked scores.  Returns (P, LSE); empty rows give P=0, LSE=-inf."""
    m = s.max(axis=1, keepdims=True)
    empty = ~np.isfinite(m[:, 0])
    m_safe = np.where(np.isfinite(m), m, 0.0)
    e = np.exp(s - m_safe)              # exp(-inf) = 0 for masked entries
    l = e.sum(axis=1, keepdims=True)
    p = np.where(l > 0, e / np.where(l > 0, l, 1.0), 0.0)
    lse = np.where(empty, -np.inf, m_safe[:, 0] + np.log(np.where(l[:, 0] > 0, l[:, 0], 1.0)))
    return p, lse


def _mask_for(b: int, S_q: int, S_k: int, causal: bool, kv_len) -> np.ndarray:
    return allowed_mask(S_q, S_k, causal, None if kv_len is None else int(kv_len[b]))


def head_probs(q, k, Hq: int, Hkv: int, scale: float, causal: bool = False, kv_len=None):
    """Full probability tensor P, float64 (B, Hq, S_q, S_k).  For tests of small shapes."""
    Q = split_heads(q, Hq)
    K = split_heads(k, Hkv)
    B, _, S, _ = Q.shape
    Sk = K.shape[2]
    P = np.zeros((B, Hq, S, Sk))
    for b in range(B):
        allowed = _mask_for(b, S, Sk, causal, kv_len)
        for h in range(Hq):
            g = kv_head_of(h, Hq, Hkv)
            P[b, h], _ = softmax_rows(masked_scores(Q[b, h], K[b, g], scale, allowed))
    return P


def attn_fwd(q, k, v, Hq: int, Hkv: int, scale: float, causal: bool = False, kv_len=None):
    """Forward pass.

    q: (B, S_q, Hq*d), k, v: (B, S_k, Hkv*d) token-major (any float dtype; upcast).
    Returns (O (B, S_q, Hq*d) float64, LSE (B, Hq, S_q) float64).
    """
    Q = split_heads(q, Hq)
    K = split_heads(k, Hkv)
    V = split_heads(v, Hkv)
    B, _, S, d = Q.shape
    Sk = K.shape[2]
    O = np.zeros((B, Hq, S, d))
    LSE = np.zeros((B, Hq, S))
    for b in range(B):
        allowed = _mask_for(b, S, Sk, causal, kv_len)
        for h in range(Hq):
            g = kv_head_of(h, Hq, Hkv)
            p, lse = softmax_rows(masked_scores(Q[b, h], K[b, g], scale, allowed))
            O[b, h] = p @ V[b, g]
            LSE[b, h] = lse
    return merge_heads(O), LSE


def attn_bwd(q, k, v, do, Hq: int, Hkv: int, scale: float, causal: bool = False, kv_len=None):
    """Backward pass of L = sum(O * dO) with O = attn_fwd(q, k, v).

    P is recomputed from q and k (the oracle saves nothing between passes).
    Returns (dQ (B, S_q, Hq*d), dK (B, S_k, Hkv*d), dV (B, S_k, Hkv*d)), float64.
    """
    Q = split_heads(q, Hq)
    K = split_heads(k, Hkv)
    V = split_heads(v, Hkv)
    dO = split_heads(do, Hq)
    B, _, S, d = Q.shape
    Sk = K.shape[2]
    dQ = np.zeros((B, Hq, S, d))
    dK = np.zeros((B, Hkv, Sk, d))
    dV = np.zeros((B, Hkv, Sk, d))
    for b in range(B):
        allowed = _mask_for(b, S, Sk, causal, kv_len)
        for h in range(Hq):
            g = kv_head_of(h, Hq, Hkv)
            p, _ = softmax_rows(masked_scores(Q[b, h], K[b, g], scale, allowed))
            dq, dk, dv = head_bwd(p, Q[b, h], K[b, g], V[b, g], dO[b, h], scale)
            dQ[b, h] = dq
            dK[b, g] += dk
            dV[b, g] += dv
    return merge_heads(dQ), merge_heads(dK), merge_heads(dV)


def head_bwd(p, qh, kh, vh, doh, scale):
    """Gradients of one (batch, query head) given its probabilities p (S_q, S_k).

    Returns (dq, dk, dv), the latter two being this head's contribution to its
    key/value head.
    """
    o = p @ vh
    dp = doh @ vh.T
    D = np.sum(doh * o, axis=1)
    ds = p * (dp - D[:, None])
    return scale * (ds @ kh), scale * (ds.T @ qh), p.T @ doh


def bwd_row_dot(o, do, Hq: int) -> np.ndarray:
    """D[b, h, i] = sum_k dO[b, i, h, k] * O[b, i, h, k], float64 (B, Hq, S_q)."""
    return np.sum(split_heads(o, Hq) * split_heads(do, Hq), axis=3)
