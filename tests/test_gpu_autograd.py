"""The autograd wrappers (paper_2607_21624_amd.autograd): gradients through
torch's autograd equal the oracle's, and a small attention block written with
them gives bit for bit the results of the explicit C ABI calls."""
import math

import numpy as np
import pytest

import oracle
import synth
from parity_util import note, rel_err, to_dev, to_np

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.mark.parametrize("causal,Hq,Hkv,d,S", [(True, 4, 2, 64, 200), (False, 2, 2, 128, 96)])
def test_attention_autograd_matches_oracle(causal, Hq, Hkv, d, S):
    import torch
    from paper_2607_21624_amd import autograd as ag
    B = 2
    rng = np.random.default_rng(S + Hq)
    bf = lambda *s: synth.round_to_bf16(rng.standard_normal(s))
    q, k, v, do = bf(B, S, Hq * d), bf(B, S, Hkv * d), bf(B, S, Hkv * d), bf(B, S, Hq * d)
    note(f"autograd attention causal={causal} Hq={Hq} Hkv={Hkv} d={d} S={S}")
    Q, K, V = (to_dev(t, "bf16").requires_grad_(True) for t in (q, k, v))
    O = ag.attention(Q, K, V, Hq, Hkv, causal=causal)
    (O.float() * to_dev(do, "bf16").float()).sum().backward()
    torch.cuda.synchronize()
    scale = 1.0 / math.sqrt(d)
    O_ref, _ = oracle.attn_fwd(q, k, v, Hq, Hkv, scale, causal)
    dQ, dK, dV = oracle.attn_bwd(q, k, v, do, Hq, Hkv, scale, causal)
    for got, ref in ((O, O_ref), (Q.grad, dQ), (K.grad, dK), (V.grad, dV)):
        assert rel_err(to_np(got), ref) <= TOL


def test_linear_autograd_matches_oracle():
    import torch
    from paper_2607_21624_amd import autograd as ag
    B, S, K, N = 2, 96, 256, 192
    rng = np.random.default_rng(11)
    x, w, dy = (synth.round_to_bf16(rng.standard_normal(s)) for s in ((B, S, K), (K, N), (B, S, N)))
    X, W = to_dev(x, "bf16").requires_grad_(True), to_dev(w, "bf16").requires_grad_(True)
    note("autograd linear")
    Y = ag.linear(X, W)
    assert Y.shape == (B, S, N)
    (Y.float() * to_dev(dy, "bf16").float()).sum().backward()
    torch.cuda.synchronize()
    x2, dy2 = x.reshape(-1, K), dy.reshape(-1, N)
    assert rel_err(to_np(Y).reshape(-1, N), oracle.proj_fwd(x2, w)) <= TOL
    assert rel_err(to_np(X.grad).reshape(-1, K), oracle.proj_bwd_data(dy2, w)) <= TOL
    assert rel_err(to_np(W.grad), oracle.proj_bwd_weight(x2, dy2)) <= TOL


def test_block_through_autograd_equals_explicit_calls():
    """x -> linear(x, Wqkv) -> attention on the packed output -> linear(., Wo):
    forward and every gradient equal the explicit fbl calls bit for bit."""
    import torch
    import paper_2607_21624_amd as fbl
    from paper_2607_21624_amd import autograd as ag
    B, S, Hq, Hkv, d = 2, 128, 4, 2, 64
    Dm, P = Hq * d, (Hq + 2 * Hkv) * d
    g = torch.Generator(device="cpu").manual_seed(3)
    mk = lambda *s, sc=1.0: (sc * torch.randn(*s, generator=g)).to(device="cuda", dtype=torch.bfloat16)
    x, wqkv, wo, dy = mk(B, S, Dm), mk(Dm, P, sc=Dm ** -0.5), mk(Hq * d, Dm, sc=(Hq * d) ** -0.5), mk(B, S, Dm)
    note("autograd block")
    X, Wqkv, Wo = (t.clone().requires_grad_(True) for t in (x, wqkv, wo))
    y = ag.linear(ag.attention_packed(ag.linear(X, Wqkv), Hq, Hkv, causal=True), Wo)
    y.backward(dy)
    # the same chain through explicit calls
    qkv = fbl.proj(fbl.FBL_PROJ_FWD, x.view(B * S, Dm), wqkv).view(B, S, P)
    o, lse = fbl.attn_fwd_packed(qkv, Hq, Hkv, causal=True)
    y_ref = fbl.proj(fbl.FBL_PROJ_FWD, o.view(B * S, -1), wo).view(B, S, Dm)
    do = fbl.proj(fbl.FBL_PROJ_BWD_DATA, dy.view(B * S, Dm), wo)
    dwo = fbl.proj(fbl.FBL_PROJ_BWD_WEIGHT, o.view(B * S, -1), dy.view(B * S, Dm))
    dqkv = fbl.attn_bwd_packed(qkv, o, do.view(B, S, -1), lse, Hq, Hkv, causal=True)
    dx = fbl.proj(fbl.FBL_PROJ_BWD_DATA, dqkv.view(B * S, P), wqkv).view(B, S, Dm)
    dwqkv = fbl.proj(fbl.FBL_PROJ_BWD_WEIGHT, x.view(B * S, Dm), dqkv.view(B * S, P))
    torch.cuda.synchronize()
    for got, ref in ((y, y_ref), (X.grad, dx), (Wqkv.grad, dwqkv), (Wo.grad, dwo)):
        assert torch.equal(got, ref)
