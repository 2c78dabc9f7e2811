"""HIP graph capture of the hot path: forward + backward (all phases) and the
projection products captured once on a torch CUDA graph and replayed several
times, with unrelated eager launches and synchronisations between the
replays; every replay must equal the eager results bit for bit (the kernels
are deterministic and the step records no memset or allocation)."""
import math

import numpy as np
import pytest

import synth
from parity_util import note

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["bert_base_keypad", "gpt2_medium_causal", "llama32_1b_gqa"])
def test_attention_step_graph_replays_match_eager(name):
    import torch
    import paper_2607_21624_amd as fbl
    w = synth.WORKLOADS[name]
    inp = synth.make_inputs(w)
    note(f"graph replay {name}")
    dev = lambda x: torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda").to(torch.bfloat16)
    q, k, v, do = dev(inp["q"]), dev(inp["k"]), dev(inp["v"]), dev(inp["do"])
    kv_len = None if inp["kv_len"] is None else torch.from_numpy(inp["kv_len"]).to("cuda")
    causal = bool(w.mask & synth.MASK_CAUSAL)
    scale = 1.0 / math.sqrt(w.d)
    o, lse = torch.empty_like(q), torch.empty((w.B, w.Hq, w.S), dtype=torch.float32, device="cuda")
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ws = torch.empty(fbl.fbl_attn_bwd_workspace(fbl.layout_of(q, w.Hq), fbl.layout_of(k, w.Hkv)),
                     dtype=torch.uint8, device="cuda")

    def step():
        fbl.attn_fwd(q, k, v, w.Hq, w.Hkv, scale, causal, kv_len, out=o, lse=lse)
        fbl.attn_bwd(q, k, v, o, do, lse, w.Hq, w.Hkv, scale, causal, kv_len, dq=dq, dk=dk, dv=dv, workspace=ws)

    outs = lambda: [t.clone() for t in (o, lse, dq, dk, dv)]
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):   # warm up off the capture stream (first launches set kernel attributes)
        step()
    torch.cuda.synchronize()
    eager = outs()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    x = torch.randn(1 << 20, device="cuda")
    for rep in range(3):
        for t in (o, lse, dq, dk, dv):   # the replay must rewrite every output
            t.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(outs(), eager):
            assert torch.equal(a, b) or (a.dtype == torch.float32 and torch.equal(torch.nan_to_num(a), torch.nan_to_num(b))), \
                f"replay {rep} differs from the eager step"
        y = (x * 2.0).sum()   # unrelated eager work between replays
        torch.cuda.synchronize()
        assert torch.isfinite(y)


def test_projection_graph_replays_match_eager():
    import torch
    import paper_2607_21624_amd as fbl
    M, K, N = 512, 1024, 768
    g0 = torch.Generator(device="cpu").manual_seed(5)
    mk = lambda r, c: torch.randn(r, c, generator=g0).to(device="cuda", dtype=torch.bfloat16)
    X, W, dY = mk(M, K), mk(K, N), mk(M, N)
    Y, dX, dW = (torch.empty(s, dtype=torch.bfloat16, device="cuda") for s in ((M, N), (M, K), (K, N)))
    note("graph replay projections")

    def step():
        fbl.proj(fbl.FBL_PROJ_FWD, X, W, out=Y)
        fbl.proj(fbl.FBL_PROJ_BWD_DATA, dY, W, out=dX)
        fbl.proj(fbl.FBL_PROJ_BWD_WEIGHT, X, dY, out=dW)

    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        step()
    torch.cuda.synchronize()
    eager = [t.clone() for t in (Y, dX, dW)]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for rep in range(3):
        for t in (Y, dX, dW):
            t.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip((Y, dX, dW), eager):
            assert torch.equal(a, b), f"replay {rep} differs from the eager products"
        torch.cuda.synchronize()
