"""Pins of the fp64 attention oracle against things other than itself.

Each check ties the oracle to brute force, a library special case, calculus,
a closed form or an invariant, so that a dropped term, a wrong sign or index,
a transposed operand or a wrong head map fails at least one of them (the
mutation tests at the end plant such mistakes in the oracle and check that a
pin catches each one).  All CPU.
"""
import itertools
import math

import numpy as np
import pytest
import torch

import oracle
import oracle.attention as oatt
from oracle import brute

MASKS = [(False, False), (True, False), (False, True), (True, True)]


def _rand(rng, B, S, H, d):
    return rng.standard_normal((B, S, H * d))


def _lens(rng, B, S, keypad):
    if not keypad:
        return None
    return rng.integers(1, S + 1, size=B).astype(np.int32)


def _rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


# ---------------------------------------------------------------- brute force
@pytest.mark.parametrize("causal,keypad", MASKS)
@pytest.mark.parametrize("Hq,Hkv", [(2, 2), (4, 2), (3, 1)])
@pytest.mark.parametrize("S", [1, 5, 8])
def test_matches_scalar_brute_force(causal, keypad, Hq, Hkv, S):
    rng = np.random.default_rng(1000 + S * 7 + Hq)
    B, d = 2, 4
    q, k, v, do = (_rand(rng, B, S, H, d) for H in (Hq, Hkv, Hkv, Hq))
    kv_len = _lens(rng, B, S, keypad)
    scale = 1 / math.sqrt(d)
    O, LSE = oracle.attn_fwd(q, k, v, Hq, Hkv, scale, causal, kv_len)
    dQ, dK, dV = oracle.attn_bwd(q, k, v, do, Hq, Hkv, scale, causal, kv_len)
    Ob, LSEb, _ = brute.fwd(q, k, v, B, S, Hq, Hkv, d, scale, causal, kv_len)
    dQb, dKb, dVb = brute.bwd(q, k, v, do, B, S, Hq, Hkv, d, scale, causal, kv_len)
    np.testing.assert_allclose(O, np.array(Ob), rtol=0, atol=1e-12)
    np.testing.assert_allclose(LSE, np.array(LSEb), rtol=0, atol=1e-12)
    np.testing.assert_allclose(dQ, np.array(dQb), rtol=0, atol=1e-12)
    np.testing.assert_allclose(dK, np.array(dKb), rtol=0, atol=1e-12)
    np.testing.assert_allclose(dV, np.array(dVb), rtol=0, atol=1e-12)


# ------------------------------------------------------- softmax normalisation
@pytest.mark.parametrize("causal,keypad", MASKS)
def test_softmax_rows_sum_to_one(causal, keypad):
    rng = np.random.default_rng(7)
    B, S, H, d = 2, 33, 2, 8
    q, k = _rand(rng, B, S, H, d), _rand(rng, B, S, H, d)
    kv_len = _lens(rng, B, S, keypad)
    P = oracle.head_probs(q, k, H, H, 0.3, causal, kv_len)
    assert np.all(P >= 0)
    np.testing.assert_allclose(P.sum(axis=3), 1.0, rtol=0, atol=1e-12)
    # masked entries carry exactly zero probability
    for b in range(B):
        allowed = oatt.allowed_mask(S, S, causal, None if kv_len is None else int(kv_len[b]))
        assert np.all(P[b][:, ~allowed] == 0.0)


# --------------------------------------------- library special case (torch fp64)
def _torch_reference(q, k, v, do, Hq, Hkv, scale, causal, kv_len):
    B, S, _ = q.shape
    d = q.shape[2] // Hq
    G = Hq // Hkv
    T = lambda x, H: torch.tensor(x, dtype=torch.float64).reshape(B, S, H, d).permute(0, 2, 1, 3).contiguous()
    tq, tk, tv, tdo = T(q, Hq), T(k, Hkv), T(v, Hkv), T(do, Hq)
    tq.requires_grad_(True); tk.requires_grad_(True); tv.requires_grad_(True)
    mask = torch.ones(B, 1, S, S, dtype=torch.bool)
    if causal:
        mask &= torch.tril(torch.ones(S, S, dtype=torch.bool))
    if kv_len is not None:
        for b in range(B):
            mask[b, :, :, int(kv_len[b]):] = False
    kr = tk.repeat_interleave(G, dim=1)
    vr = tv.repeat_interleave(G, dim=1)
    out = torch.nn.functional.scaled_dot_product_attention(tq, kr, vr, attn_mask=mask, scale=scale)
    out.backward(tdo)
    back = lambda x: x.detach().permute(0, 2, 1, 3).reshape(B, S, -1).numpy()
    return back(out), back(tq.grad), back(tk.grad), back(tv.grad)


@pytest.mark.parametrize("causal,keypad", MASKS)
@pytest.mark.parametrize("Hq,Hkv,d", [(2, 2, 16), (4, 1, 8), (8, 2, 32)])
def test_matches_torch_sdpa_float64(causal, keypad, Hq, Hkv, d):
    rng = np.random.default_rng(11 + Hq + d)
    B, S = 3, 37
    q, k, v, do = (_rand(rng, B, S, H, d) for H in (Hq, Hkv, Hkv, Hq))
    kv_len = None
    if keypad:
        kv_len = rng.integers(1, S + 1, size=B).astype(np.int32)
    scale = 1 / math.sqrt(d)
    O, _ = oracle.attn_fwd(q, k, v, Hq, Hkv, scale, causal, kv_len)
    dQ, dK, dV = oracle.attn_bwd(q, k, v, do, Hq, Hkv, scale, causal, kv_len)
    tO, tdQ, tdK, tdV = _torch_reference(q, k, v, do, Hq, Hkv, scale, causal, kv_len)
    for a, b in ((O, tO), (dQ, tdQ), (dK, tdK), (dV, tdV)):
        assert _rel(a, b) < 1e-12


# --------------------------------------------------------- finite differences
def _loss(q, k, v, do, Hq, Hkv, scale, causal, kv_len):
    O, _ = oracle.attn_fwd(q, k, v, Hq, Hkv, scale, causal, kv_len)
    return float(np.sum(O * do))


@pytest.mark.parametrize("causal,keypad", MASKS)
@pytest.mark.parametrize("Hq,Hkv", [(2, 2), (2, 1)])
def test_gradients_match_central_differences(causal, keypad, Hq, Hkv):
    rng = np.random.default_rng(23 + 2 * causal + keypad)
    B, S, d = 2, 4, 3
    q, k, v, do = (_rand(rng, B, S, H, d) for H in (Hq, Hkv, Hkv, Hq))
    kv_len = np.array([3, 2], dtype=np.int32) if keypad else None
    scale = 0.7
    grads = oracle.attn_bwd(q, k, v, do, Hq, Hkv, scale, causal, kv_len)
    h = 1e-5
    for which, g in zip(range(3), grads):
        base = [q, k, v]
        fd = np.zeros_like(base[which])
        for idx in itertools.product(*(range(n) for n in base[which].shape)):
            plus = [x.copy() for x in base]
            minus = [x.copy() for x in base]
            plus[which][idx] += h
            minus[which][idx] -= h
            fd[idx] = (_loss(*plus, do, Hq, Hkv, scale, causal, kv_len)
                       - _loss(*minus, do, Hq, Hkv, scale, causal, kv_len)) / (2 * h)
        np.testing.assert_allclose(g, fd, rtol=0, atol=1e-6)


# ------------------------------------------------------------- closed forms
@pytest.mark.parametrize("Hq,Hkv", [(2, 2), (4, 2)])
def test_single_key_closed_form(Hq, Hkv):
    rng = np.random.default_rng(5)
    B, S, d = 3, 1, 8
    q, k, v, do = (_rand(rng, B, S, H, d) for H in (Hq, Hkv, Hkv, Hq))
    scale = 0.25
    O, LSE = oracle.attn_fwd(q, k, v, Hq, Hkv, scale)
    dQ, dK, dV = oracle.attn_bwd(q, k, v, do, Hq, Hkv, scale)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            g = h // G
            np.testing.assert_allclose(O[b, 0, h * d:(h + 1) * d], v[b, 0, g * d:(g + 1) * d], atol=1e-15)
            s00 = scale * np.dot(q[b, 0, h * d:(h + 1) * d], k[b, 0, g * d:(g + 1) * d])
            assert abs(LSE[b, h, 0] - s00) < 1e-14
    assert np.max(np.abs(dQ)) < 1e-14 and np.max(np.abs(dK)) < 1e-14
    # dV of a key/value head = sum of dO over the query heads in its group
    for g in range(Hkv):
        want = sum(do[:, :, h * d:(h + 1) * d] for h in range(g * G, (g + 1) * G))
        np.testing.assert_allclose(dV[:, :, g * d:(g + 1) * d], want, atol=1e-14)


@pytest.mark.parametrize("causal,keypad", MASKS)
def test_zero_query_gives_uniform_average(causal, keypad):
    rng = np.random.default_rng(9)
    B, S, H, d = 2, 9, 2, 4
    q = np.zeros((B, S, H * d))
    k, v = _rand(rng, B, S, H, d), _rand(rng, B, S, H, d)
    kv_len = np.array([4, 9], dtype=np.int32) if keypad else None
    O, LSE = oracle.attn_fwd(q, k, v, H, H, 1.0, causal, kv_len)
    for b in range(B):
        L = S if kv_len is None else int(kv_len[b])
        for i in range(S):
            n = min(i + 1, L) if causal else L
            for h in range(H):
                want = v[b, :n, h * d:(h + 1) * d].mean(axis=0)
                np.testing.assert_allclose(O[b, i, h * d:(h + 1) * d], want, atol=1e-14)
                assert abs(LSE[b, h, i] - math.log(n)) < 1e-14


def test_key_shift_invariance():
    rng = np.random.default_rng(13)
    B, S, H, d = 2, 11, 2, 6
    q, k, v, do = (_rand(rng, B, S, H, d) for _ in range(4))
    c = rng.standard_normal(d)
    k2 = k + np.tile(c, H)[None, None, :]
    for causal in (False, True):
        O1, L1 = oracle.attn_fwd(q, k, v, H, H, 0.5, causal)
        O2, L2 = oracle.attn_fwd(q, k2, v, H, H, 0.5, causal)
        np.testing.assert_allclose(O1, O2, atol=1e-12)
        # LSE shifts by scale * q_i . c
        shift = 0.5 * np.einsum("bshd,d->bhs", q.reshape(B, S, H, d), c)
        np.testing.assert_allclose(L2 - L1, shift, atol=1e-12)
        g1 = oracle.attn_bwd(q, k, v, do, H, H, 0.5, causal)
        g2 = oracle.attn_bwd(q, k2, v, do, H, H, 0.5, causal)
        for a, b in zip(g1, g2):
            np.testing.assert_allclose(a, b, atol=1e-12)


def test_head_group_and_batch_permutation_equivariance():
    rng = np.random.default_rng(17)
    B, S, Hq, Hkv, d = 3, 10, 4, 2, 5
    G = Hq // Hkv
    q, do = _rand(rng, B, S, Hq, d), _rand(rng, B, S, Hq, d)
    k, v = _rand(rng, B, S, Hkv, d), _rand(rng, B, S, Hkv, d)
    kv_len = np.array([3, 10, 7], dtype=np.int32)
    gperm = np.array([1, 0])                      # permute whole GQA groups
    qperm = np.concatenate([np.arange(g * G, (g + 1) * G) for g in gperm])
    bperm = np.array([2, 0, 1])

    def heads(x, H, perm):
        return x.reshape(B, S, H, d)[:, :, perm, :].reshape(B, S, H * d)

    base_O, base_L = oracle.attn_fwd(q, k, v, Hq, Hkv, 0.4, True, kv_len)
    base_g = oracle.attn_bwd(q, k, v, do, Hq, Hkv, 0.4, True, kv_len)
    O, L = oracle.attn_fwd(heads(q, Hq, qperm), heads(k, Hkv, gperm), heads(v, Hkv, gperm), Hq, Hkv, 0.4, True, kv_len)
    np.testing.assert_allclose(O, heads(base_O, Hq, qperm), atol=1e-13)
    np.testing.assert_allclose(L, base_L[:, qperm, :], atol=1e-13)
    dq, dk, dv = oracle.attn_bwd(heads(q, Hq, qperm), heads(k, Hkv, gperm), heads(v, Hkv, gperm),
                                 heads(do, Hq, qperm), Hq, Hkv, 0.4, True, kv_len)
    np.testing.assert_allclose(dq, heads(base_g[0], Hq, qperm), atol=1e-13)
    np.testing.assert_allclose(dk, heads(base_g[1], Hkv, gperm), atol=1e-13)
    np.testing.assert_allclose(dv, heads(base_g[2], Hkv, gperm), atol=1e-13)
    # batch permutation carries the key lengths along
    O, L = oracle.attn_fwd(q[bperm], k[bperm], v[bperm], Hq, Hkv, 0.4, True, kv_len[bperm])
    np.testing.assert_allclose(O, base_O[bperm], atol=1e-13)
    np.testing.assert_allclose(L, base_L[bperm], atol=1e-13)
    g = oracle.attn_bwd(q[bperm], k[bperm], v[bperm], do[bperm], Hq, Hkv, 0.4, True, kv_len[bperm])
    for a, b in zip(g, base_g):
        np.testing.assert_allclose(a, b[bperm], atol=1e-13)


# ------------------------------------------------- backward structure pins
def test_dv_equals_pt_do_with_brute_force_p():
    rng = np.random.default_rng(29)
    B, S, Hq, Hkv, d = 2, 6, 4, 2, 3
    q, do = _rand(rng, B, S, Hq, d), _rand(rng, B, S, Hq, d)
    k, v = _rand(rng, B, S, Hkv, d), _rand(rng, B, S, Hkv, d)
    kv_len = np.array([6, 4], dtype=np.int32)
    _, _, Pb = brute.fwd(q, k, v, B, S, Hq, Hkv, d, 0.6, True, kv_len)
    Pb = np.array(Pb)                                  # (B, Hq, S, S)
    _, _, dV = oracle.attn_bwd(q, k, v, do, Hq, Hkv, 0.6, True, kv_len)
    G = Hq // Hkv
    for b in range(B):
        for g in range(Hkv):
            want = sum(Pb[b, h].T @ do[b, :, h * d:(h + 1) * d] for h in range(g * G, (g + 1) * G))
            np.testing.assert_allclose(dV[b, :, g * d:(g + 1) * d], want, atol=1e-13)


def test_row_dot_two_ways():
    rng = np.random.default_rng(31)
    B, S, H, d = 2, 12, 3, 4
    q, k, v, do = (_rand(rng, B, S, H, d) for _ in range(4))
    O, _ = oracle.attn_fwd(q, k, v, H, H, 0.5, True)
    D1 = oracle.bwd_row_dot(O, do, H)
    P = oracle.head_probs(q, k, H, H, 0.5, True)
    Vh = v.reshape(B, S, H, d).transpose(0, 2, 1, 3)
    dOh = do.reshape(B, S, H, d).transpose(0, 2, 1, 3)
    dP = dOh @ Vh.transpose(0, 1, 3, 2)
    D2 = np.sum(P * dP, axis=3)
    np.testing.assert_allclose(D1, D2, atol=1e-12)


@pytest.mark.parametrize("causal,keypad", MASKS)
def test_gradient_column_sum_invariants(causal, keypad):
    rng = np.random.default_rng(37)
    B, S, Hq, Hkv, d = 2, 17, 4, 2, 8
    q, do = _rand(rng, B, S, Hq, d), _rand(rng, B, S, Hq, d)
    k, v = _rand(rng, B, S, Hkv, d), _rand(rng, B, S, Hkv, d)
    kv_len = np.array([5, 17], dtype=np.int32) if keypad else None
    _, dK, dV = oracle.attn_bwd(q, k, v, do, Hq, Hkv, 0.35, causal, kv_len)
    G = Hq // Hkv
    for b in range(B):
        for g in range(Hkv):
            # sum_j dS_ij = 0 for every row  =>  sum_j dK_j = 0
            assert np.max(np.abs(dK[b, :, g * d:(g + 1) * d].sum(axis=0))) < 1e-12
            # sum_j P_ij = 1 for every row  =>  sum_j dV_j = sum_i dO_i (over the group)
            want = sum(do[b, :, h * d:(h + 1) * d].sum(axis=0) for h in range(g * G, (g + 1) * G))
            np.testing.assert_allclose(dV[b, :, g * d:(g + 1) * d].sum(axis=0), want, atol=1e-12)


def test_gqa_equals_mha_on_repeated_kv():
    rng = np.random.default_rng(41)
    B, S, Hq, Hkv, d = 2, 9, 6, 2, 4
    G = Hq // Hkv
    q, do = _rand(rng, B, S, Hq, d), _rand(rng, B, S, Hq, d)
    k, v = _rand(rng, B, S, Hkv, d), _rand(rng, B, S, Hkv, d)
    rep = lambda x: np.repeat(x.reshape(B, S, Hkv, d), G, axis=2).reshape(B, S, Hq * d)
    O1, L1 = oracle.attn_fwd(q, k, v, Hq, Hkv, 0.5, True)
    O2, L2 = oracle.attn_fwd(q, rep(k), rep(v), Hq, Hq, 0.5, True)
    np.testing.assert_allclose(O1, O2, atol=1e-14)
    np.testing.assert_allclose(L1, L2, atol=1e-14)
    dq1, dk1, dv1 = oracle.attn_bwd(q, k, v, do, Hq, Hkv, 0.5, True)
    dq2, dk2, dv2 = oracle.attn_bwd(q, rep(k), rep(v), do, Hq, Hq, 0.5, True)
    grp = lambda x: x.reshape(B, S, Hkv, G, d).sum(axis=3).reshape(B, S, Hkv * d)
    np.testing.assert_allclose(dq1, dq2, atol=1e-13)
    np.testing.assert_allclose(dk1, grp(dk2), atol=1e-13)
    np.testing.assert_allclose(dv1, grp(dv2), atol=1e-13)


def test_fully_masked_row_reading():
    """A row with no allowed key: O = 0, LSE = -inf, no gradient (kv_len = 0)."""
    rng = np.random.default_rng(43)
    B, S, H, d = 2, 5, 1, 3
    q, k, v, do = (_rand(rng, B, S, H, d) for _ in range(4))
    kv_len = np.array([0, 5], dtype=np.int32)
    O, L = oracle.attn_fwd(q, k, v, H, H, 1.0, False, kv_len)
    assert np.all(O[0] == 0) and np.all(np.isneginf(L[0]))
    dq, dk, dv = oracle.attn_bwd(q, k, v, do, H, H, 1.0, False, kv_len)
    assert np.all(dq[0] == 0) and np.all(dk[0] == 0) and np.all(dv[0] == 0)


# ------------------------------------------------------- planted mistakes
def _pins_pass():
    """Run a compact subset of the pins; True when all hold."""
    try:
        test_matches_torch_sdpa_float64(True, True, 4, 2, 8)
        test_gradients_match_central_differences(True, False, 2, 1)
        test_single_key_closed_form(4, 2)
        test_gradient_column_sum_invariants(True, True)
    except AssertionError:
        return False
    return True


def test_pins_pass_on_the_real_oracle():
    assert _pins_pass()


REAL_HEAD_BWD = oatt.head_bwd
REAL_ALLOWED = oatt.allowed_mask


def _mut_causal_strict(S_q, S_k, causal, kv_len_b):
    m = REAL_ALLOWED(S_q, S_k, False, kv_len_b)
    if causal:
        m &= np.arange(S_k)[None, :] < np.arange(S_q)[:, None]
    return m


def _mut_no_d(p, qh, kh, vh, doh, s):
    ds = p * (doh @ vh.T)
    return s * (ds @ kh), s * (ds.T @ qh), p.T @ doh


def _mut_dv_untransposed(p, qh, kh, vh, doh, s):
    dq, dk, _ = REAL_HEAD_BWD(p, qh, kh, vh, doh, s)
    return dq, dk, p @ doh


def _mut_dk_unscaled(p, qh, kh, vh, doh, s):
    dq, dk, dv = REAL_HEAD_BWD(p, qh, kh, vh, doh, s)
    return dq, dk / s, dv


def _mut_dq_sign(p, qh, kh, vh, doh, s):
    dq, dk, dv = REAL_HEAD_BWD(p, qh, kh, vh, doh, s)
    return -dq, dk, dv


def _mut_dq_uses_q(p, qh, kh, vh, doh, s):
    dq, dk, dv = REAL_HEAD_BWD(p, qh, kh, vh, doh, s)
    ds = p * (doh @ vh.T - np.sum(doh * (p @ vh), axis=1)[:, None])
    return s * (ds @ qh), dk, dv


MUTANTS = {
    "gqa map h % Hkv": ("kv_head_of", lambda h, Hq, Hkv: h % Hkv),
    "scale dropped from scores": ("masked_scores",
                                  lambda qh, kh, scale, allowed: np.where(allowed, qh @ kh.T, -np.inf)),
    "causal mask off by one": ("allowed_mask", _mut_causal_strict),
    "D term dropped": ("head_bwd", _mut_no_d),
    "dV operand not transposed": ("head_bwd", _mut_dv_untransposed),
    "dK scale dropped": ("head_bwd", _mut_dk_unscaled),
    "dQ sign flipped": ("head_bwd", _mut_dq_sign),
    "dQ multiplies Q instead of K": ("head_bwd", _mut_dq_uses_q),
}


@pytest.mark.parametrize("name", list(MUTANTS))
def test_planted_mistake_is_caught(monkeypatch, name):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(oatt, attr, fn)
    with np.errstate(all="ignore"):
        caught = not _pins_pass()
    assert caught, f"planted mistake '{name}' was not caught by any pin"
