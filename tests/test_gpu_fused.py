"""The one-launch backward for key/value sequences of at most 128 tokens (the
statistics, dK, dV and dQ of a (batch, kv head) formed by one workgroup that
holds all its keys), against the fp64 oracle and against the three-pass
backward on the same inputs; and a 128-key shape with few, long (batch, head)
pairs, which keeps the split three-launch path."""
import math

import numpy as np
import pytest

import synth
from parity_util import TOL, compare, note, oracle_fwd_bwd, to_dev, to_np

pytestmark = pytest.mark.gpu

CASES = [  # name, B, S_q, S_kv, Hq, Hkv, d, dtype, mask
    ("causal_gqa", 3, 100, 0, 4, 2, 64, "bf16", synth.MASK_CAUSAL),
    ("cross_d128", 2, 300, 128, 4, 4, 128, "bf16", synth.MASK_NONE),
    ("keypad", 3, 128, 0, 4, 1, 64, "bf16", synth.MASK_KEY_PADDING),
    ("ragged_d32", 2, 77, 0, 2, 2, 32, "bf16", synth.MASK_CAUSAL | synth.MASK_KEY_PADDING),
    ("single_key", 2, 40, 1, 2, 1, 64, "bf16", synth.MASK_NONE),
    ("tiny_f32", 2, 64, 0, 2, 2, 32, "f32", synth.MASK_NONE),
    ("causal_f32_d64", 2, 90, 0, 4, 2, 64, "f32", synth.MASK_CAUSAL),
    ("cross_f32", 1, 200, 50, 2, 2, 64, "f32", synth.MASK_KEY_PADDING),
    # 128 keys, but two (batch, head) pairs of 96 query blocks: the split three-launch path
    ("long_q", 1, 6144, 128, 2, 2, 64, "bf16", synth.MASK_NONE),
]


@pytest.mark.parametrize("name,B,Sq,Skv,Hq,Hkv,d,dt,mask", CASES, ids=[c[0] for c in CASES])
def test_fused_backward(name, B, Sq, Skv, Hq, Hkv, d, dt, mask):
    import torch
    import paper_2607_21624_amd as fbl
    w = synth.Workload(name, B=B, S=Sq, Hq=Hq, Hkv=Hkv, d=d, dtype=dt, mask=mask, seed=Sq + d, len_lo=0,
                       len_hi=Skv or Sq, S_kv=Skv)
    inp = synth.make_inputs(w)
    if inp["kv_len"] is not None:
        inp["kv_len"][0] = 0  # one batch with no allowed key
    note(f"fused {name} B={B} Sq={Sq} Skv={w.Skv} Hq={Hq} Hkv={Hkv} d={d} {dt} mask={mask} kv_len={inp['kv_len']}")
    q, k, v, do = (to_dev(inp[n], dt) for n in ("q", "k", "v", "do"))
    kv_len = None if inp["kv_len"] is None else torch.from_numpy(inp["kv_len"].astype(np.int32)).to("cuda")
    causal = bool(mask & synth.MASK_CAUSAL)
    scale = 1.0 / math.sqrt(d)
    o, lse = fbl.attn_fwd(q, k, v, Hq, Hkv, scale, causal, kv_len)
    ws_full = fbl.fbl_attn_bwd_workspace(fbl.layout_of(q, Hq), fbl.layout_of(k, Hkv))
    n_launch = fbl.attn_bwd_launches(fbl.layout_of(q, Hq), fbl.layout_of(k, Hkv), mask, ws_full)
    assert n_launch == (4 if name == "long_q" else 1), n_launch
    fused = fbl.attn_bwd(q, k, v, o, do, lse, Hq, Hkv, scale, causal, kv_len)
    again = fbl.attn_bwd(q, k, v, o, do, lse, Hq, Hkv, scale, causal, kv_len)
    # the same backward as three passes (statistics, key/value-major, dQ)
    ws = torch.empty(fbl.fbl_attn_bwd_workspace(fbl.layout_of(q, Hq), fbl.layout_of(k, Hkv)), dtype=torch.uint8,
                     device="cuda")
    outs = [torch.full_like(t, float("nan")) for t in (q, k, v)]
    for ph in (fbl.FBL_BWD_PREP, fbl.FBL_BWD_KV, fbl.FBL_BWD_Q):
        fbl.attn_bwd(q, k, v, o, do, lse, Hq, Hkv, scale, causal, kv_len, dq=outs[0], dk=outs[1], dv=outs[2],
                     workspace=ws, phases=ph)
    torch.cuda.synchronize()
    for a_, b_ in zip(fused, again):
        assert torch.equal(a_, b_), "fused backward not repeatable"
    ref = oracle_fwd_bwd(inp)
    for label, res in (("fused", fused), ("three passes", outs)):
        got = {"o": to_np(o), "lse": to_np(lse), "dq": to_np(res[0]), "dk": to_np(res[1]), "dv": to_np(res[2])}
        errs, bad = compare(got, ref, dt)
        note(f"{label} rel errs {errs}")
        assert not bad, f"{name} {label}: {bad} (tol {TOL[dt]})"
