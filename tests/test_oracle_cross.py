"""Pins of the fp64 oracle for cross-attention: queries and keys/values of
different lengths (S_q != S_k), as in encoder-decoder attention.

Same kinds of pins as tests/test_oracle.py -- scalar brute force, float64
torch scaled_dot_product_attention with autograd, central finite differences,
the single-key and zero-query closed forms, and the column-sum invariants --
at rectangular shapes, so that a place where the oracle still confuses the
query length with the key length fails.  All CPU.
"""
import itertools
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import brute


def _rand(rng, B, S, H, d):
    return rng.standard_normal((B, S, H * d))


def _rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


@pytest.mark.parametrize("Sq,Sk", [(3, 1), (3, 7), (7, 3), (5, 9)])
@pytest.mark.parametrize("causal,keypad", [(False, False), (False, True), (True, False)])
@pytest.mark.parametrize("Hq,Hkv", [(2, 2), (4, 2)])
def test_cross_matches_scalar_brute_force(Sq, Sk, causal, keypad, Hq, Hkv):
    rng = np.random.default_rng(100 * Sq + Sk + 7 * Hq)
    B, d = 2, 4
    q, do = _rand(rng, B, Sq, Hq, d), _rand(rng, B, Sq, Hq, d)
    k, v = _rand(rng, B, Sk, Hkv, d), _rand(rng, B, Sk, Hkv, d)
    kv_len = rng.integers(1, Sk + 1, size=B).astype(np.int32) if keypad else None
    scale = 1 / math.sqrt(d)
    O, LSE = oracle.attn_fwd(q, k, v, Hq, Hkv, scale, causal, kv_len)
    dQ, dK, dV = oracle.attn_bwd(q, k, v, do, Hq, Hkv, scale, causal, kv_len)
    assert O.shape == (B, Sq, Hq * d) and LSE.shape == (B, Hq, Sq)
    assert dQ.shape == (B, Sq, Hq * d) and dK.shape == (B, Sk, Hkv * d) and dV.shape == (B, Sk, Hkv * d)
    Ob, LSEb, _ = brute.fwd(q, k, v, B, Sq, Hq, Hkv, d, scale, causal, kv_len, S_k=Sk)
    dQb, dKb, dVb = brute.bwd(q, k, v, do, B, Sq, Hq, Hkv, d, scale, causal, kv_len, S_k=Sk)
    np.testing.assert_allclose(O, np.array(Ob), rtol=0, atol=1e-12)
    np.testing.assert_allclose(LSE, np.array(LSEb), rtol=0, atol=1e-12)
    np.testing.assert_allclose(dQ, np.array(dQb), rtol=0, atol=1e-12)
    np.testing.assert_allclose(dK, np.array(dKb), rtol=0, atol=1e-12)
    np.testing.assert_allclose(dV, np.array(dVb), rtol=0, atol=1e-12)


def _torch_cross(q, k, v, do, Hq, Hkv, scale, kv_len):
    B, Sq, _ = q.shape
    Sk = k.shape[1]
    d = q.shape[2] // Hq
    G = Hq // Hkv
    T = lambda x, S, H: torch.tensor(x, dtype=torch.float64).reshape(B, S, H, d).permute(0, 2, 1, 3).contiguous()
    tq, tk, tv, tdo = T(q, Sq, Hq), T(k, Sk, Hkv), T(v, Sk, Hkv), T(do, Sq, Hq)
    tq.requires_grad_(True); tk.requires_grad_(True); tv.requires_grad_(True)
    mask = torch.ones(B, 1, Sq, Sk, dtype=torch.bool)
    if kv_len is not None:
        for b in range(B):
            mask[b, :, :, int(kv_len[b]):] = False
    out = torch.nn.functional.scaled_dot_product_attention(tq, tk.repeat_interleave(G, dim=1),
                                                           tv.repeat_interleave(G, dim=1), attn_mask=mask,
                                                           scale=scale)
    out.backward(tdo)
    back = lambda x, S: x.detach().permute(0, 2, 1, 3).reshape(B, S, -1).numpy()
    return back(out, Sq), back(tq.grad, Sq), back(tk.grad, Sk), back(tv.grad, Sk)


@pytest.mark.parametrize("Sq,Sk", [(29, 41), (50, 13), (1, 17)])
@pytest.mark.parametrize("keypad", [False, True])
@pytest.mark.parametrize("Hq,Hkv,d", [(2, 2, 16), (4, 1, 8)])
def test_cross_matches_torch_sdpa_float64(Sq, Sk, keypad, Hq, Hkv, d):
    rng = np.random.default_rng(Sq * 3 + Sk + d)
    B = 3
    q, do = _rand(rng, B, Sq, Hq, d), _rand(rng, B, Sq, Hq, d)
    k, v = _rand(rng, B, Sk, Hkv, d), _rand(rng, B, Sk, Hkv, d)
    kv_len = rng.integers(1, Sk + 1, size=B).astype(np.int32) if keypad else None
    scale = 1 / math.sqrt(d)
    O, _ = oracle.attn_fwd(q, k, v, Hq, Hkv, scale, False, kv_len)
    dQ, dK, dV = oracle.attn_bwd(q, k, v, do, Hq, Hkv, scale, False, kv_len)
    tO, tdQ, tdK, tdV = _torch_cross(q, k, v, do, Hq, Hkv, scale, kv_len)
    for a, b in ((O, tO), (dQ, tdQ), (dK, tdK), (dV, tdV)):
        assert _rel(a, b) < 1e-12


@pytest.mark.parametrize("keypad", [False, True])
def test_cross_gradients_match_central_differences(keypad):
    rng = np.random.default_rng(31 + keypad)
    B, Sq, Sk, d, Hq, Hkv = 2, 3, 5, 3, 2, 1
    q, do = _rand(rng, B, Sq, Hq, d), _rand(rng, B, Sq, Hq, d)
    k, v = _rand(rng, B, Sk, Hkv, d), _rand(rng, B, Sk, Hkv, d)
    kv_len = np.array([4, 2], dtype=np.int32) if keypad else None
    scale = 0.7
    loss = lambda q_, k_, v_: float(np.sum(oracle.attn_fwd(q_, k_, v_, Hq, Hkv, scale, False, kv_len)[0] * do))
    grads = oracle.attn_bwd(q, k, v, do, Hq, Hkv, scale, False, kv_len)
    h = 1e-5
    for which, g in zip(range(3), grads):
        base = [q, k, v]
        fd = np.zeros_like(base[which])
        for idx in itertools.product(*(range(n) for n in base[which].shape)):
            plus = [x.copy() for x in base]
            minus = [x.copy() for x in base]
            plus[which][idx] += h
            minus[which][idx] -= h
            fd[idx] = (loss(*plus) - loss(*minus)) / (2 * h)
        np.testing.assert_allclose(g, fd, rtol=0, atol=1e-6)


def test_cross_single_key_closed_form():
    """S_k = 1: every query attends the one key, so O_i = v_0, LSE_i = s_i0,
    dQ = dK = 0 and dV_0 = sum over queries and the group's heads of dO."""
    rng = np.random.default_rng(41)
    B, Sq, Hq, Hkv, d = 2, 6, 4, 2, 8
    q, do = _rand(rng, B, Sq, Hq, d), _rand(rng, B, Sq, Hq, d)
    k, v = _rand(rng, B, 1, Hkv, d), _rand(rng, B, 1, Hkv, d)
    scale = 0.3
    O, LSE = oracle.attn_fwd(q, k, v, Hq, Hkv, scale)
    dQ, dK, dV = oracle.attn_bwd(q, k, v, do, Hq, Hkv, scale)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            g = h // G
            for i in range(Sq):
                np.testing.assert_allclose(O[b, i, h * d:(h + 1) * d], v[b, 0, g * d:(g + 1) * d], atol=1e-15)
                s = scale * np.dot(q[b, i, h * d:(h + 1) * d], k[b, 0, g * d:(g + 1) * d])
                assert abs(LSE[b, h, i] - s) < 1e-14
    assert np.max(np.abs(dQ)) < 1e-14 and np.max(np.abs(dK)) < 1e-14
    for g in range(Hkv):
        want = sum(do[:, :, h * d:(h + 1) * d].sum(axis=1) for h in range(g * G, (g + 1) * G))
        np.testing.assert_allclose(dV[:, 0, g * d:(g + 1) * d], want, atol=1e-13)


@pytest.mark.parametrize("keypad", [False, True])
def test_cross_zero_query_gives_uniform_average(keypad):
    rng = np.random.default_rng(43)
    B, Sq, Sk, H, d = 2, 5, 11, 2, 4
    q = np.zeros((B, Sq, H * d))
    k, v = _rand(rng, B, Sk, H, d), _rand(rng, B, Sk, H, d)
    kv_len = np.array([4, 11], dtype=np.int32) if keypad else None
    O, LSE = oracle.attn_fwd(q, k, v, H, H, 1.0, False, kv_len)
    for b in range(B):
        n = Sk if kv_len is None else int(kv_len[b])
        for h in range(H):
            want = v[b, :n, h * d:(h + 1) * d].mean(axis=0)
            for i in range(Sq):
                np.testing.assert_allclose(O[b, i, h * d:(h + 1) * d], want, atol=1e-14)
                assert abs(LSE[b, h, i] - math.log(n)) < 1e-14


def test_cross_gradient_column_sums():
    """sum_j dK_j = 0 (rows of dS sum to zero) and sum_j dV_j = sum_i dO_i,
    per (batch, kv head), over the query heads of the group."""
    rng = np.random.default_rng(47)
    B, Sq, Sk, Hq, Hkv, d = 2, 13, 21, 4, 2, 8
    q, do = _rand(rng, B, Sq, Hq, d), _rand(rng, B, Sq, Hq, d)
    k, v = _rand(rng, B, Sk, Hkv, d), _rand(rng, B, Sk, Hkv, d)
    dQ, dK, dV = oracle.attn_bwd(q, k, v, do, Hq, Hkv, 0.4)
    G = Hq // Hkv
    for g in range(Hkv):
        assert np.max(np.abs(dK[:, :, g * d:(g + 1) * d].sum(axis=1))) < 1e-12
        want = sum(do[:, :, h * d:(h + 1) * d].sum(axis=1) for h in range(g * G, (g + 1) * G))
        np.testing.assert_allclose(dV[:, :, g * d:(g + 1) * d].sum(axis=1), want, atol=1e-12)
