"""Every attention tile configuration against the fp64 oracle, and the
measured tile selection: the tuned choice meets the oracle and is the tile
the automatic choice then runs, bit for bit equal to the explicit-id run."""
import math

import numpy as np
import pytest

import synth
from parity_util import TOL, compare, note, oracle_fwd_bwd, to_dev, to_np

pytestmark = pytest.mark.gpu


def _inputs(B, S, Hq, Hkv, d, mask, seed, Skv=0):
    w = synth.Workload(f"tile_s{S}", B=B, S=S, Hq=Hq, Hkv=Hkv, d=d, dtype="bf16", mask=mask, seed=seed,
                       len_lo=S // 3, len_hi=S, S_kv=Skv)
    return w, synth.make_inputs(w)


def _dev(inp):
    import torch
    w = inp["workload"]
    q, k, v, do = (to_dev(inp[n], "bf16") for n in ("q", "k", "v", "do"))
    kv_len = None if inp["kv_len"] is None else torch.from_numpy(inp["kv_len"].astype(np.int32)).to("cuda")
    return q, k, v, do, kv_len, bool(w.mask & synth.MASK_CAUSAL), 1.0 / math.sqrt(w.d)


def _legal(pass_, d):
    import paper_2607_21624_amd as fbl
    return [t for t, i in fbl.attn_tiles(d).items() if i["pass"] == pass_ and i["legal"]]


SHAPES = [  # B, S, Hq, Hkv, d, mask: ragged lengths spanning several tiles, every mask kind, GQA
    (2, 300, 4, 2, 128, synth.MASK_CAUSAL), (1, 517, 4, 4, 128, synth.MASK_NONE),
    (2, 300, 4, 1, 64, synth.MASK_CAUSAL), (3, 260, 2, 2, 64, synth.MASK_KEY_PADDING),
    (2, 200, 4, 2, 32, synth.MASK_CAUSAL), (1, 333, 2, 2, 32, synth.MASK_NONE),
]


@pytest.mark.parametrize("B,S,Hq,Hkv,d,mask", SHAPES)
def test_every_forward_tile(B, S, Hq, Hkv, d, mask):
    import torch
    import paper_2607_21624_amd as fbl
    w, inp = _inputs(B, S, Hq, Hkv, d, mask, seed=S + d)
    q, k, v, do, kv_len, causal, scale = _dev(inp)
    ref = oracle_fwd_bwd(inp)
    for t in _legal(fbl.FBL_ATTN_FWD, d):
        note(f"forward tile {t} B={B} S={S} Hq={Hq} Hkv={Hkv} d={d} mask={mask}")
        o, lse = fbl.attn_fwd(q, k, v, Hq, Hkv, scale, causal, kv_len, tile=t)
        o2, lse2 = fbl.attn_fwd(q, k, v, Hq, Hkv, scale, causal, kv_len, tile=t)
        torch.cuda.synchronize()
        assert torch.equal(o, o2) and torch.equal(lse, lse2), f"tile {t} not repeatable"
        errs, bad = compare({"o": to_np(o), "lse": to_np(lse)}, ref, "bf16", names=("o", "lse"))
        assert not bad, f"forward tile {t}: {bad} (tol {TOL['bf16']})"


@pytest.mark.parametrize("B,S,Hq,Hkv,d,mask", SHAPES)
def test_every_backward_tile(B, S, Hq, Hkv, d, mask):
    import torch
    import paper_2607_21624_amd as fbl
    w, inp = _inputs(B, S, Hq, Hkv, d, mask, seed=S + d + 1)
    q, k, v, do, kv_len, causal, scale = _dev(inp)
    ref = oracle_fwd_bwd(inp)
    o, lse = fbl.attn_fwd(q, k, v, Hq, Hkv, scale, causal, kv_len)
    for kt in _legal(fbl.FBL_ATTN_BWD_KV, d):
        for qt in _legal(fbl.FBL_ATTN_BWD_DQ, d):
            note(f"backward tiles kv={kt} dq={qt} B={B} S={S} Hq={Hq} Hkv={Hkv} d={d} mask={mask}")
            dq, dk, dv = fbl.attn_bwd(q, k, v, o, do, lse, Hq, Hkv, scale, causal, kv_len, kv_tile=kt, dq_tile=qt)
            torch.cuda.synchronize()
            got = {"dq": to_np(dq), "dk": to_np(dk), "dv": to_np(dv)}
            errs, bad = compare(got, ref, "bf16", names=("dq", "dk", "dv"))
            assert not bad, f"backward tiles kv={kt} dq={qt}: {bad} (tol {TOL['bf16']})"


def test_llama7b_shape_forward_tiles():
    """The Llama-7B-like causal shape (B=1, H=32, S=4096, d=128) with every
    forward tile, all heads against the oracle's forward."""
    import torch
    import oracle
    import paper_2607_21624_amd as fbl
    w = synth.WORKLOADS["llama7b_causal"]
    inp = synth.make_inputs(w)
    q, k, v, do, kv_len, causal, scale = _dev(inp)
    ro, rlse = oracle.attn_fwd(inp["q"], inp["k"], inp["v"], w.Hq, w.Hkv, scale, causal)
    for t in _legal(fbl.FBL_ATTN_FWD, w.d):
        note(f"llama7b forward tile {t}")
        o, lse = fbl.attn_fwd(q, k, v, w.Hq, w.Hkv, scale, causal, tile=t)
        torch.cuda.synchronize()
        errs, bad = compare({"o": to_np(o), "lse": to_np(lse)}, {"o": ro, "lse": rlse}, "bf16", names=("o", "lse"))
        assert not bad, f"tile {t}: {bad}"


@pytest.mark.parametrize("B,S,Hq,Hkv,d,mask", [(2, 1024, 8, 2, 64, synth.MASK_CAUSAL),
                                                (1, 768, 4, 4, 128, synth.MASK_CAUSAL)])
def test_tuned_tiles_match_oracle_and_explicit_ids(B, S, Hq, Hkv, d, mask):
    import torch
    import paper_2607_21624_amd as fbl
    w, inp = _inputs(B, S, Hq, Hkv, d, mask, seed=7)
    q, k, v, do, kv_len, causal, scale = _dev(inp)
    lq, lk = fbl.layout_of(q, Hq), fbl.layout_of(k, Hkv)
    fbl.attn_tune_reset()
    note(f"tune B={B} S={S} Hq={Hq} Hkv={Hkv} d={d}")
    best, ms, (o, lse, dq, dk, dv) = fbl.attn_tune(q, k, v, do, Hq, Hkv, scale, causal, kv_len, reps=3)
    torch.cuda.synchronize()
    note(f"tuned {best} ms {ms}")
    # the choice is the fastest candidate of each pass
    for p, chosen in zip((fbl.FBL_ATTN_FWD, fbl.FBL_ATTN_BWD_KV, fbl.FBL_ATTN_BWD_DQ), best):
        cands = fbl.attn_candidates(p, lq, lk)
        assert chosen in cands and ms[chosen] == min(ms[t] for t in cands)
        assert fbl.attn_tuned_tile(p, lq, lk, int(causal)) == chosen
    assert fbl.attn_auto_tiles(lq, lk, int(causal)) == best
    got = {"o": to_np(o), "lse": to_np(lse), "dq": to_np(dq), "dk": to_np(dk), "dv": to_np(dv)}
    errs, bad = compare(got, oracle_fwd_bwd(inp), "bf16")
    assert not bad, f"tuned tiles {best}: {bad}"
    # AUTO now runs the tuned tiles: bit for bit the explicit-id results
    oa, lsea = fbl.attn_fwd(q, k, v, Hq, Hkv, scale, causal, kv_len)
    ox, lsex = fbl.attn_fwd(q, k, v, Hq, Hkv, scale, causal, kv_len, tile=best[0])
    ga = fbl.attn_bwd(q, k, v, oa, do, lsea, Hq, Hkv, scale, causal, kv_len)
    gx = fbl.attn_bwd(q, k, v, ox, do, lsex, Hq, Hkv, scale, causal, kv_len, kv_tile=best[1], dq_tile=best[2])
    torch.cuda.synchronize()
    assert torch.equal(oa, ox) and torch.equal(lsea, lsex) and torch.equal(oa, o)
    for a, b, c in zip(ga, gx, (dq, dk, dv)):
        assert torch.equal(a, b) and torch.equal(a, c)
    fbl.attn_tune_reset()
    assert fbl.attn_tuned_tile(fbl.FBL_ATTN_FWD, lq, lk, int(causal)) == -1
