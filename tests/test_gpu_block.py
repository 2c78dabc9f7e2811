"""GPU parity of a whole attention block, forward and backward, with no layout
copy anywhere: the QKV projection writes one packed [B*S, (Hq + 2Hkv) d]
buffer, attention reads Q, K, V from it in place and writes dQ, dK, dV into
one packed gradient buffer, and the output projection and both weight
gradients read the token-major activations as they are (the chain the paper's
tile-based index transformation covers, section 4.3, with the matrix-product
gradients of section 4.1).

Two checks per tensor (tolerance 2e-2 of max|ref|, bf16 storage):
  * stage by stage: the oracle applied to the GPU's own bf16 inputs of that
    stage (isolates each stage's error);
  * end to end: the oracle's fp64 chain from the same X, weights and dY.
"""
import math

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


def _oracle_block(x, wqkv, wo, dy, B, S, Hq, Hkv, d, causal):
    """fp64 chain: projections, attention on the packed columns, and back."""
    scale = 1.0 / math.sqrt(d)
    qkv = oracle.proj_fwd(x, wqkv)
    q3 = qkv[:, :Hq * d].reshape(B, S, Hq * d)
    k3 = qkv[:, Hq * d:(Hq + Hkv) * d].reshape(B, S, Hkv * d)
    v3 = qkv[:, (Hq + Hkv) * d:].reshape(B, S, Hkv * d)
    o3, lse = oracle.attn_fwd(q3, k3, v3, Hq, Hkv, scale, causal)
    o = o3.reshape(B * S, Hq * d)
    y = oracle.proj_fwd(o, wo)
    do = oracle.proj_bwd_data(dy, wo)
    dwo = oracle.proj_bwd_weight(o, dy)
    dq, dk, dv = oracle.attn_bwd(q3, k3, v3, do.reshape(B, S, Hq * d), Hq, Hkv, scale, causal)
    dqkv = np.concatenate([dq.reshape(B * S, -1), dk.reshape(B * S, -1), dv.reshape(B * S, -1)], axis=1)
    dx = oracle.proj_bwd_data(dqkv, wqkv)
    dwqkv = oracle.proj_bwd_weight(x, dqkv)
    return {"qkv": qkv, "o": o, "lse": lse, "y": y, "do": do, "dwo": dwo, "dqkv": dqkv, "dx": dx, "dwqkv": dwqkv}


@pytest.mark.parametrize("B,S,Hq,Hkv,d,causal", [(2, 256, 8, 4, 64, True), (1, 384, 4, 4, 128, False),
                                                 (2, 200, 8, 2, 64, True)])
def test_attention_block_no_copies(B, S, Hq, Hkv, d, causal):
    import torch
    fbl = _lib()
    Dm = Hq * d  # model width
    P = (Hq + 2 * Hkv) * d
    rng = np.random.default_rng(B * 1000 + S + Hq)
    bf = lambda *s, sc=1.0: synth.round_to_bf16(sc * rng.standard_normal(s))
    x = bf(B * S, Dm)
    wqkv = bf(Dm, P, sc=1 / math.sqrt(Dm))
    wo = bf(Hq * d, Dm, sc=1 / math.sqrt(Hq * d))
    dy = bf(B * S, Dm)
    note(f"attention block B={B} S={S} Hq={Hq} Hkv={Hkv} d={d} causal={causal}")
    X, Wqkv, Wo, dY = (to_dev(t, "bf16") for t in (x, wqkv, wo, dy))

    qkv = fbl.proj(fbl.FBL_PROJ_FWD, X, Wqkv)                      # [B*S, P]
    qkv3 = qkv.view(B, S, P)                                      # a view, no copy
    o3, lse = fbl.attn_fwd_packed(qkv3, Hq, Hkv, causal=causal)   # [B, S, Hq d]
    o = o3.view(B * S, Hq * d)
    y = fbl.proj(fbl.FBL_PROJ_FWD, o, Wo)
    do = fbl.proj(fbl.FBL_PROJ_BWD_DATA, dY, Wo)
    dwo = fbl.proj(fbl.FBL_PROJ_BWD_WEIGHT, o, dY)
    dqkv3 = fbl.attn_bwd_packed(qkv3, o3, do.view(B, S, Hq * d), lse, Hq, Hkv, causal=causal)
    dqkv = dqkv3.view(B * S, P)
    dx = fbl.proj(fbl.FBL_PROJ_BWD_DATA, dqkv, Wqkv)
    dwqkv = fbl.proj(fbl.FBL_PROJ_BWD_WEIGHT, X, dqkv)
    torch.cuda.synchronize()
    got = {n: to_np(t) for n, t in (("qkv", qkv), ("o", o), ("lse", lse), ("y", y), ("do", do), ("dwo", dwo),
                                     ("dqkv", dqkv), ("dx", dx), ("dwqkv", dwqkv))}

    # stage by stage, from the GPU's own inputs of each stage
    scale = 1.0 / math.sqrt(d)
    g_qkv = got["qkv"]
    q3, k3, v3 = (g_qkv[:, a:b].reshape(B, S, -1) for a, b in ((0, Hq * d), (Hq * d, (Hq + Hkv) * d),
                                                                ((Hq + Hkv) * d, P)))
    o_ref, lse_ref = oracle.attn_fwd(q3, k3, v3, Hq, Hkv, scale, causal)
    dq, dk, dv = oracle.attn_bwd(q3, k3, v3, got["do"].reshape(B, S, -1), Hq, Hkv, scale, causal)
    stage = {"qkv": oracle.proj_fwd(x, wqkv), "o": o_ref.reshape(B * S, -1), "lse": lse_ref,
             "y": oracle.proj_fwd(got["o"], wo), "do": oracle.proj_bwd_data(dy, wo),
             "dwo": oracle.proj_bwd_weight(got["o"], dy),
             "dqkv": np.concatenate([dq.reshape(B * S, -1), dk.reshape(B * S, -1), dv.reshape(B * S, -1)], axis=1),
             "dx": oracle.proj_bwd_data(got["dqkv"], wqkv), "dwqkv": oracle.proj_bwd_weight(x, got["dqkv"])}
    for n, ref in stage.items():
        e = rel_err(got[n], ref)
        assert e <= TOL, f"stage {n}: rel err {e}"

    # end to end
    chain = _oracle_block(x, wqkv, wo, dy, B, S, Hq, Hkv, d, causal)
    for n, ref in chain.items():
        e = rel_err(got[n], ref)
        assert e <= TOL, f"end to end {n}: rel err {e}"
