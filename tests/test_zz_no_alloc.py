"""fbl_attn_bwd_noalloc: the backward with the library's own device scratch in
place of a workspace, called through the C ABI.  Its outputs equal those of
fbl_attn_bwd given a workspace of the scratch's size (the same passes run),
bit for bit, and meet the oracle; two calls in a row, the second on a smaller
input, check that nothing left in the shared scratch by the first call leaks
into the second."""
import math

import numpy as np
import pytest

import synth
from parity_util import TOL, compare, note, oracle_fwd_bwd, to_dev, to_np

pytestmark = pytest.mark.gpu


def _run_pair(w, seed):
    import torch
    import paper_2607_21624_amd as fbl
    inp = synth.make_inputs(w, seed=seed)
    dt = w.dtype
    q, k, v, do = (to_dev(inp[n], dt) for n in ("q", "k", "v", "do"))
    kv_len = None if inp["kv_len"] is None else torch.from_numpy(inp["kv_len"].astype(np.int32)).to("cuda")
    causal = bool(w.mask & synth.MASK_CAUSAL)
    scale = 1.0 / math.sqrt(w.d)
    o, lse = fbl.attn_fwd(q, k, v, w.Hq, w.Hkv, scale, causal, kv_len)
    outs = [torch.full_like(t, float("nan")) for t in (q, k, v)]
    fbl.attn_bwd_noalloc(q, k, v, o, do, lse, w.Hq, w.Hkv, *outs, scale=scale, causal=causal, kv_len=kv_len)
    # the existing entry point with a workspace of the scratch's size
    ws = torch.empty(fbl.NOALLOC_SCRATCH_BYTES, dtype=torch.uint8, device="cuda")
    ref = fbl.attn_bwd(q, k, v, o, do, lse, w.Hq, w.Hkv, scale, causal, kv_len, workspace=ws)
    torch.cuda.synchronize()
    for name, a, b in zip(("dq", "dk", "dv"), outs, ref):
        assert torch.equal(a, b), f"{w.name}: {name} differs from fbl_attn_bwd"
    got = {"o": to_np(o), "lse": to_np(lse), "dq": to_np(outs[0]), "dk": to_np(outs[1]), "dv": to_np(outs[2])}
    errs, bad = compare(got, oracle_fwd_bwd(inp), dt)
    note(f"noalloc {w.name} rel errs {errs}")
    assert not bad, f"{w.name}: {bad} (tol {TOL[dt]})"


CASES = [
    # stored-dS path, split key/value pass (GQA, few key blocks), then a smaller causal shape
    (synth.Workload("na_gqa", B=2, S=640, Hq=8, Hkv=2, d=64, dtype="bf16", mask=synth.MASK_CAUSAL, seed=0),
     synth.Workload("na_small", B=1, S=200, Hq=4, Hkv=4, d=128, dtype="bf16", mask=synth.MASK_CAUSAL, seed=1)),
    # dS does not fit the scratch (recompute path), then a smaller key-padding shape that fits it
    (synth.Workload("na_big", B=1, S=4096, Hq=4, Hkv=4, d=128, dtype="bf16", mask=synth.MASK_CAUSAL, seed=2),
     synth.Workload("na_pad", B=3, S=300, Hq=4, Hkv=2, d=64, dtype="bf16", mask=synth.MASK_KEY_PADDING, seed=3,
                    len_lo=100, len_hi=300)),
    # fp32 storage (statistics only), then a smaller fp32 shape
    (synth.Workload("na_f32", B=2, S=160, Hq=4, Hkv=2, d=64, dtype="f32", mask=synth.MASK_CAUSAL, seed=4),
     synth.Workload("na_f32s", B=1, S=40, Hq=2, Hkv=2, d=32, dtype="f32", mask=0, seed=5)),
]


@pytest.mark.parametrize("first,second", CASES, ids=[c[0].name for c in CASES])
def test_noalloc_matches_workspace_entry(first, second):
    note(f"noalloc pair {first.name} then {second.name}")
    _run_pair(first, 0)
    _run_pair(second, 1)

