"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on the
same seeded inputs.

Tolerance per output tensor T in {O, LSE, dQ, dK, dV}:
max|T_gpu - T_ref| / max|T_ref| <= 1e-4 for fp32 storage, <= 2e-2 for bf16
storage (over all elements, padded rows included; -inf LSE entries must
match exactly).  Index maps are compared bit-exactly.
"""
import math

import numpy as np
import pytest

import oracle
import synth
from parity_util import (TOL, compare, gpu_fwd_bwd, note, oracle_fwd_bwd, rel_err, select_heads, to_dev,
                         to_np)

pytestmark = pytest.mark.gpu


def _lib():
    import paper_2607_21624_amd as fbl
    return fbl


# ----------------------------------------------------------------- index map
@pytest.mark.parametrize("B,S,H,D,row", [(1, 64, 2, 32, 0), (8, 128, 12, 64, 0), (2, 33, 3, 128, 0),
                                          (2, 9, 4, 64, 10 * 64)])
def test_device_index_map_bit_exact(B, S, H, D, row):
    import torch
    fbl = _lib()
    note(f"index map B={B} S={S} H={H} D={D} row={row}")
    l = fbl.fbl_layout_desc(fbl.FBL_BF16, B, S, H, D, row_stride=row)
    out = torch.full((B * H * S * D,), -7, dtype=torch.int64, device="cuda")
    fbl.fbl_layout_map_device(l, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().reshape(B, H, S, D)
    if row:
        want = oracle.head_split_offsets(B, S, H, D, row_stride=row, batch_stride=S * row)
    else:
        want = oracle.token_major_offsets(B, S, H, D)
    assert np.array_equal(got, want)


# ---------------------------------------------------------- named workloads
def _check_workload(name, kv_heads=None, seed=None):
    w = {**synth.WORKLOADS, **synth.PAPER_MHA_SHAPES}[name]
    inp = synth.make_inputs(w, seed=seed)
    note(f"{name} seed={inp['seed']} B={w.B} S={w.S} Hq={w.Hq} Hkv={w.Hkv} d={w.d} {w.dtype} mask={w.mask}")
    got = select_heads(gpu_fwd_bwd(inp), w, kv_heads)
    ref = oracle_fwd_bwd(inp, kv_heads)
    errs, bad = compare(got, ref, w.dtype)
    note(f"{name} rel errs {errs}")
    assert not bad, f"{name}: {bad} (tol {TOL[w.dtype]})"


def test_tiny_mha_f32():
    _check_workload("tiny_mha_f32")


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_bert_base_keypad(seed):
    _check_workload("bert_base_keypad", seed=seed)


def test_gpt2_medium_causal():
    _check_workload("gpt2_medium_causal")


@pytest.mark.parametrize("name", list(synth.PAPER_MHA_SHAPES))
def test_paper_mha_shapes(name):
    """The three MHA shapes of the paper's own multi-head attention experiment
    (S = 512, bf16): every head checked."""
    _check_workload(name)


def test_llama32_1b_gqa_all_groups():
    # full-size launch, every one of the eight key/value groups checked
    _check_workload("llama32_1b_gqa")


def test_llama7b_causal_all_heads():
    # full-size launch, every one of the 32 heads checked (the oracle takes
    # about 10 s on the host)
    _check_workload("llama7b_causal")


# ------------------------------------------------------- random small shapes
RANDOM_CASES = []
for _d in (32, 64, 128):
    for _dt in ("f32", "bf16"):
        for _i in range(3):
            RANDOM_CASES.append((_d, _dt, 100 * _d + 10 * (_dt == "bf16") + _i))


@pytest.mark.parametrize("d,dt,seed", RANDOM_CASES)
def test_random_shapes(d, dt, seed):
    rng = np.random.default_rng(seed)
    w = synth.random_workload(rng, dtype=dt, d=d, max_s=300, name=f"rand{seed}")
    inp = synth.make_inputs(w)
    note(f"random seed={seed} B={w.B} S={w.S} Hq={w.Hq} Hkv={w.Hkv} d={d} {dt} mask={w.mask} kv_len={inp['kv_len']}")
    errs, bad = compare(gpu_fwd_bwd(inp), oracle_fwd_bwd(inp), dt)
    assert not bad, f"{w}: {bad}"


@pytest.mark.parametrize("S", [1, 2, 31, 32, 33, 64, 65, 127, 128, 129, 191, 257])
@pytest.mark.parametrize("d", [64, 128])
def test_ragged_lengths_causal_gqa(S, d):
    w = synth.Workload(f"ragged{S}", B=2, S=S, Hq=4, Hkv=2, d=d, dtype="bf16", mask=synth.MASK_CAUSAL,
                       seed=S + d)
    inp = synth.make_inputs(w)
    note(f"ragged S={S} d={d}")
    errs, bad = compare(gpu_fwd_bwd(inp), oracle_fwd_bwd(inp), "bf16")
    assert not bad, f"S={S} d={d}: {bad}"


# ------------------------------------------- recompute dQ path (min workspace)
@pytest.mark.parametrize("d,mask,S", [(128, synth.MASK_CAUSAL, 300), (64, synth.MASK_CAUSAL, 129),
                                      (32, synth.MASK_KEY_PADDING, 200), (64, synth.MASK_NONE, 97),
                                      (128, synth.MASK_CAUSAL | synth.MASK_KEY_PADDING, 257)])
def test_recompute_dq_path(d, mask, S):
    """With the smallest workspace the dQ pass recomputes S and dP instead of
    reading stored dS; both ways must meet the oracle."""
    w = synth.Workload(f"recompute{S}", B=2, S=S, Hq=4, Hkv=2, d=d, dtype="bf16", mask=mask, seed=S + d + mask)
    inp = synth.make_inputs(w)
    note(f"recompute dQ S={S} d={d} mask={mask}")
    ref = oracle_fwd_bwd(inp)
    for ws in ("min", "full"):
        errs, bad = compare(gpu_fwd_bwd(inp, workspace=ws), ref, "bf16")
        assert not bad, f"workspace {ws}: {bad}"


# ------------------------------------------- split key/value pass (GQA, few key blocks)
@pytest.mark.parametrize("B,S,Hq,Hkv,d,mask", [(1, 1024, 8, 2, 128, synth.MASK_CAUSAL),
                                               (2, 700, 8, 2, 64, synth.MASK_CAUSAL | synth.MASK_KEY_PADDING),
                                               (1, 513, 4, 1, 128, synth.MASK_NONE),
                                               (2, 2048, 32, 8, 64, synth.MASK_CAUSAL)])
def test_split_kv_pass(B, S, Hq, Hkv, d, mask):
    """Few key blocks per CU: the key/value pass shares each key block's query
    iterations among 2 or 4 workgroups (fp32 partial dK/dV added in a fixed
    order).  The split, the unsplit stored-dS pass and the recompute pass must
    all meet the oracle, and the split run must be bitwise repeatable."""
    w = synth.Workload(f"split{S}", B=B, S=S, Hq=Hq, Hkv=Hkv, d=d, dtype="bf16", mask=mask, seed=S + Hq + d)
    inp = synth.make_inputs(w)
    kv_heads = None if Hkv <= 2 else [0, Hkv - 1]
    note(f"split kv B={B} S={S} Hq={Hq} Hkv={Hkv} d={d} mask={mask}")
    ref = oracle_fwd_bwd(inp, kv_heads)
    full = gpu_fwd_bwd(inp)
    for ws in ("full", "ds", "min"):
        got = full if ws == "full" else gpu_fwd_bwd(inp, workspace=ws)
        errs, bad = compare(select_heads(got, w, kv_heads), ref, "bf16")
        note(f"split kv workspace {ws}: {errs}")
        assert not bad, f"workspace {ws}: {bad}"
    again = gpu_fwd_bwd(inp)
    for n in ("dq", "dk", "dv"):
        assert np.array_equal(again[n], full[n]), n


# ---------------------------------------------------------- cross-attention
@pytest.mark.parametrize("name", list(synth.CROSS_WORKLOADS))
def test_cross_attention_workloads(name):
    """Whisper-large-like decoder cross-attention (448 tokens x 300 frames), all
    heads against the oracle, dQ from stored dS and from the recompute pass."""
    w = synth.CROSS_WORKLOADS[name]
    inp = synth.make_inputs(w)
    note(f"{name} B={w.B} S_q={w.S} S_kv={w.Skv} H={w.Hq} d={w.d} mask={w.mask} kv_len={inp['kv_len']}")
    ref = oracle_fwd_bwd(inp)
    for ws in ("full", "min"):
        errs, bad = compare(gpu_fwd_bwd(inp, workspace=ws), ref, w.dtype)
        note(f"{name} workspace={ws} rel errs {errs}")
        assert not bad, f"{name} workspace {ws}: {bad}"


CROSS_CASES = [
    # (d, dtype, S_q, S_kv, mask, Hq, Hkv)
    (128, "bf16", 300, 77, synth.MASK_NONE, 4, 2),
    (128, "bf16", 65, 257, synth.MASK_KEY_PADDING, 2, 2),
    (64, "bf16", 1, 200, synth.MASK_NONE, 4, 1),
    (64, "bf16", 190, 1, synth.MASK_NONE, 2, 2),
    (64, "bf16", 129, 33, synth.MASK_KEY_PADDING, 8, 2),
    (32, "bf16", 97, 160, synth.MASK_NONE, 3, 3),
    (128, "f32", 70, 130, synth.MASK_KEY_PADDING, 2, 1),
    (64, "f32", 150, 40, synth.MASK_NONE, 4, 2),
    (32, "f32", 33, 95, synth.MASK_NONE, 2, 2),
]


@pytest.mark.parametrize("d,dt,Sq,Skv,mask,Hq,Hkv", CROSS_CASES)
def test_cross_attention_shapes(d, dt, Sq, Skv, mask, Hq, Hkv):
    """Rectangular score matrices: S_q < S_kv and S_q > S_kv, ragged tails on
    both sides, a single query and a single key, MHA and GQA, fp32 and bf16."""
    w = synth.Workload(f"cross{Sq}x{Skv}", B=2, S=Sq, S_kv=Skv, Hq=Hq, Hkv=Hkv, d=d, dtype=dt, mask=mask,
                       len_lo=1, len_hi=Skv, seed=Sq * 1000 + Skv + d)
    inp = synth.make_inputs(w)
    note(f"cross S_q={Sq} S_kv={Skv} d={d} {dt} mask={mask} Hq={Hq} Hkv={Hkv} kv_len={inp['kv_len']}")
    ref = oracle_fwd_bwd(inp)
    for ws in ("full", "min"):
        errs, bad = compare(gpu_fwd_bwd(inp, workspace=ws), ref, dt)
        assert not bad, f"workspace {ws}: {bad}"


# ------------------------------------------------------------- edge cases
def test_zero_and_overlong_key_lengths():
    import torch
    fbl = _lib()
    w = synth.Workload("edge", B=3, S=70, Hq=2, Hkv=1, d=64, dtype="bf16", mask=synth.MASK_KEY_PADDING,
                       len_lo=0, len_hi=0, seed=5)
    inp = synth.make_inputs(w)
    inp["kv_len"] = np.array([0, 70, 1000], dtype=np.int32)  # empty, exact, clamped to S
    note("kv_len 0 / S / >S")
    got = gpu_fwd_bwd(inp)
    ref_in = dict(inp, kv_len=np.array([0, 70, 70], dtype=np.int32))
    ref = oracle_fwd_bwd(ref_in)
    assert np.all(np.isneginf(got["lse"][0])) and np.all(got["o"][0] == 0)
    assert np.all(got["dq"][0] == 0) and np.all(got["dk"][0] == 0) and np.all(got["dv"][0] == 0)
    errs, bad = compare(got, ref, "bf16")
    assert not bad, bad


@pytest.mark.parametrize("mask", [synth.MASK_KEY_PADDING, synth.MASK_KEY_PADDING | synth.MASK_CAUSAL])
@pytest.mark.parametrize("d", [64, 128])
def test_padding_keys_with_overflowing_scores(mask, d):
    """Keys past kv_len carry huge values (their unmasked scores overflow exp):
    the outputs must not see them, and their dK, dV rows must be exact zeros."""
    w = synth.Workload("padinf", B=2, S=200, Hq=4, Hkv=2, d=d, dtype="bf16", mask=mask, len_lo=1, len_hi=1,
                       seed=11 + d + mask)
    inp = synth.make_inputs(w)
    inp["kv_len"] = np.array([100, 37], dtype=np.int32)
    for b, n in enumerate(inp["kv_len"]):
        inp["k"][b, n:] = 300.0
        inp["v"][b, n:] = -300.0
    note(f"padding keys overflow d={d} mask={mask}")
    got = gpu_fwd_bwd(inp)
    for b, n in enumerate(inp["kv_len"]):
        assert np.all(got["dk"][b, n:] == 0) and np.all(got["dv"][b, n:] == 0)
    for name in ("o", "lse", "dq", "dk", "dv"):
        assert np.all(np.isfinite(got[name]) | np.isneginf(got[name])), name
    errs, bad = compare(got, oracle_fwd_bwd(inp), "bf16")
    assert not bad, bad


def test_backward_alone_from_oracle_forward():
    """Feed the oracle's O and LSE (cast to storage) to the GPU backward."""
    import torch
    fbl = _lib()
    w = synth.WORKLOADS["gpt2_medium_causal"]
    w = synth.Workload("bwd_only", B=2, S=384, Hq=8, Hkv=2, d=128, dtype="bf16", mask=synth.MASK_CAUSAL, seed=3)
    inp = synth.make_inputs(w)
    ref = oracle_fwd_bwd(inp)
    scale = 1.0 / math.sqrt(w.d)
    note("bwd only")
    q, k, v, do = (to_dev(inp[n], "bf16") for n in ("q", "k", "v", "do"))
    o = to_dev(synth.round_to_bf16(ref["o"]), "bf16")
    lse = torch.from_numpy(ref["lse"].astype(np.float32)).cuda()
    dq, dk, dv = fbl.attn_bwd(q, k, v, o, do, lse, w.Hq, w.Hkv, scale, True, None)
    torch.cuda.synchronize()
    for n, t in (("dq", dq), ("dk", dk), ("dv", dv)):
        assert rel_err(to_np(t), ref[n]) <= TOL["bf16"], n


def test_strided_views_of_packed_projection():
    """Q, K, V read as column views of one packed [B, S, (Hq+2Hkv)d] tensor and
    dQ/dK/dV written into views of a packed gradient tensor: no copies."""
    import torch
    fbl = _lib()
    B, S, Hq, Hkv, d = 2, 200, 8, 2, 64
    w = synth.Workload("packed", B=B, S=S, Hq=Hq, Hkv=Hkv, d=d, dtype="bf16", mask=synth.MASK_CAUSAL, seed=9)
    inp = synth.make_inputs(w)
    note("packed views")
    packed = to_dev(np.concatenate([inp["q"], inp["k"], inp["v"]], axis=2), "bf16")
    q = packed[:, :, :Hq * d]
    k = packed[:, :, Hq * d:(Hq + Hkv) * d]
    v = packed[:, :, (Hq + Hkv) * d:]
    do = to_dev(inp["do"], "bf16")
    gpacked = torch.zeros_like(packed)
    scale = 1.0 / math.sqrt(d)
    ptrs = [t.data_ptr() for t in (q, k, v)]
    o, lse = fbl.attn_fwd(q, k, v, Hq, Hkv, scale, True)
    dq, dk, dv = fbl.attn_bwd(q, k, v, o, do, lse, Hq, Hkv, scale, True, None,
                              dq=gpacked[:, :, :Hq * d], dk=gpacked[:, :, Hq * d:(Hq + Hkv) * d],
                              dv=gpacked[:, :, (Hq + Hkv) * d:])
    torch.cuda.synchronize()
    assert [t.data_ptr() for t in (q, k, v)] == ptrs
    ref = oracle_fwd_bwd(inp)
    got = {"o": to_np(o), "lse": to_np(lse), "dq": to_np(gpacked[:, :, :Hq * d]),
           "dk": to_np(gpacked[:, :, Hq * d:(Hq + Hkv) * d]), "dv": to_np(gpacked[:, :, (Hq + Hkv) * d:])}
    errs, bad = compare(got, ref, "bf16")
    assert not bad, bad


@pytest.mark.parametrize("d,mask", [(64, synth.MASK_CAUSAL), (128, synth.MASK_KEY_PADDING)])
def test_sequence_sliced_views(d, mask):
    """Q, K, V, dO and the outputs as the first 200 tokens of 300-token buffers
    (batch stride 300 rows, larger than S rows): the tail rows hold NaN and
    must be neither read (a read would bring NaN into the results) nor
    written (they must still hold NaN afterwards)."""
    import torch
    fbl = _lib()
    B, S, S_full, Hq, Hkv = 3, 200, 300, 4, 2
    w = synth.Workload("sliced", B=B, S=S, Hq=Hq, Hkv=Hkv, d=d, dtype="bf16", mask=mask, seed=d + 5)
    inp = synth.make_inputs(w)
    note(f"sequence-sliced views d={d} mask={mask}")

    def view(cols, data=None):
        full = torch.full((B, S_full, cols), float("nan"), dtype=torch.bfloat16, device="cuda")
        if data is not None:
            full[:, :S].copy_(to_dev(data, "bf16"))
        return full, full[:, :S]

    (qf, q), (kf, k), (vf, v), (dof, do) = (view(Hq * d, inp["q"]), view(Hkv * d, inp["k"]),
                                            view(Hkv * d, inp["v"]), view(Hq * d, inp["do"]))
    (of, o), (dqf, dq), (dkf, dk), (dvf, dv) = view(Hq * d), view(Hq * d), view(Hkv * d), view(Hkv * d)
    assert q.stride(0) == S_full * Hq * d and not q.is_contiguous()
    kv_len = None if inp["kv_len"] is None else torch.from_numpy(inp["kv_len"].astype(np.int32)).to("cuda")
    causal = bool(mask & synth.MASK_CAUSAL)
    scale = 1.0 / math.sqrt(d)
    _, lse = fbl.attn_fwd(q, k, v, Hq, Hkv, scale, causal, kv_len, out=o)
    fbl.attn_bwd(q, k, v, o, do, lse, Hq, Hkv, scale, causal, kv_len, dq=dq, dk=dk, dv=dv)
    torch.cuda.synchronize()
    got = {"o": to_np(o), "lse": to_np(lse), "dq": to_np(dq), "dk": to_np(dk), "dv": to_np(dv)}
    errs, bad = compare(got, oracle_fwd_bwd(inp), "bf16")
    assert not bad, bad
    for name, full in (("o", of), ("dq", dqf), ("dk", dkf), ("dv", dvf)):
        assert torch.isnan(full[:, S:].float()).all(), f"{name}: rows past S were written"


@pytest.mark.parametrize("name", ["gpt2_medium_causal", "llama32_1b_gqa", "bert_base_keypad"])
def test_backward_phases_separately(name):
    """fbl_attn_bwd_phases: the preprocessing, key/value and dQ phases as three
    calls -- on one stream, then on two streams ordered by an event -- give the
    bits of the single three-kernel call (the Llama-3.2-1B-like shape with its
    split key/value pass).  The single call names its tiles, which keeps it off
    the one-launch backward that automatic tiles pick for up to 128 keys."""
    import torch
    fbl = _lib()
    w = synth.WORKLOADS[name]
    inp = synth.make_inputs(w)
    note(f"backward phases separately {name}")
    q, k, v, do = (to_dev(inp[n], "bf16") for n in ("q", "k", "v", "do"))
    kv_len = None if inp["kv_len"] is None else torch.from_numpy(inp["kv_len"].astype(np.int32)).to("cuda")
    causal = bool(w.mask & synth.MASK_CAUSAL)
    scale = 1.0 / math.sqrt(w.d)
    o, lse = fbl.attn_fwd(q, k, v, w.Hq, w.Hkv, scale, causal, kv_len)
    ws = torch.empty(fbl.fbl_attn_bwd_workspace(fbl.layout_of(q, w.Hq), fbl.layout_of(k, w.Hkv)),
                     dtype=torch.uint8, device="cuda")
    outs = [torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)]
    run = lambda ph, stream=None, tiles=(-1, -1): fbl.attn_bwd(q, k, v, o, do, lse, w.Hq, w.Hkv, scale, causal,
                                                               kv_len, dq=outs[0], dk=outs[1], dv=outs[2],
                                                               workspace=ws, phases=ph, stream=stream,
                                                               kv_tile=tiles[0], dq_tile=tiles[1])
    mask_kind = int(causal) | (2 if kv_len is not None else 0)
    _, kv_tile, dq_tile = fbl.attn_auto_tiles(fbl.layout_of(q, w.Hq), fbl.layout_of(k, w.Hkv), mask_kind)
    run(fbl.FBL_BWD_ALL, tiles=(kv_tile, dq_tile))
    torch.cuda.synchronize()
    ref = [t.clone() for t in outs]
    for t in outs:
        t.fill_(float("nan"))
    ws.fill_(0xFF)
    for ph in (fbl.FBL_BWD_PREP, fbl.FBL_BWD_KV, fbl.FBL_BWD_Q):
        run(ph)
    torch.cuda.synchronize()
    assert all(torch.equal(a, b) for a, b in zip(outs, ref)), "three calls on one stream"
    for t in outs:
        t.fill_(float("nan"))
    ws.fill_(0xFF)
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(s1):
        run(fbl.FBL_BWD_PREP, stream=s1)
        done = torch.cuda.Event()
        done.record(s1)
    s2.wait_event(done)
    with torch.cuda.stream(s2):
        run(fbl.FBL_BWD_KV, stream=s2)
        run(fbl.FBL_BWD_Q, stream=s2)
    torch.cuda.synchronize()
    assert all(torch.equal(a, b) for a, b in zip(outs, ref)), "phases on two streams"


def test_largest_row_stride():
    """At the largest accepted row stride, (S + 128) * ss * 2 = 2^31 bytes:
    every tensor (inputs, O, dO and the gradients) is a view with 8 MB between
    consecutive tokens, the gaps filled with NaN.  The tiles' row offsets reach
    the top of the 32-bit range; any read of a gap or any wrapped offset would
    bring NaN into the results."""
    import torch
    fbl = _lib()
    B, S, Hq, Hkv, d = 1, 128, 2, 1, 128
    ss = (1 << 31) // ((S + 128) * 2)
    assert ss == 1 << 22
    w = synth.Workload("stride", B=B, S=S, Hq=Hq, Hkv=Hkv, d=d, dtype="bf16", mask=synth.MASK_CAUSAL, seed=77)
    inp = synth.make_inputs(w)
    note(f"largest row stride ss={ss} S={S} d={d}")

    def view(cols, data=None):
        buf = torch.full((S * ss,), float("nan"), dtype=torch.bfloat16, device="cuda")
        t = torch.as_strided(buf, (B, S, cols), (S * ss, ss, 1))
        if data is not None:
            t.copy_(to_dev(data, "bf16"))
        return t

    q, k, v, do = view(Hq * d, inp["q"]), view(Hkv * d, inp["k"]), view(Hkv * d, inp["v"]), view(Hq * d, inp["do"])
    o, dq, dk, dv = view(Hq * d), view(Hq * d), view(Hkv * d), view(Hkv * d)
    assert fbl.layout_of(q, Hq).ss == ss and fbl.layout_of(dk, Hkv).ss == ss
    scale = 1.0 / math.sqrt(d)
    _, lse = fbl.attn_fwd(q, k, v, Hq, Hkv, scale, True, out=o)
    fbl.attn_bwd(q, k, v, o, do, lse, Hq, Hkv, scale, True, None, dq=dq, dk=dk, dv=dv)
    torch.cuda.synchronize()
    got = {"o": to_np(o), "lse": to_np(lse), "dq": to_np(dq), "dk": to_np(dk), "dv": to_np(dv)}
    errs, bad = compare(got, oracle_fwd_bwd(inp), "bf16")
    note(f"largest row stride rel errs {errs}")
    assert not bad, bad
    del q, k, v, do, o, dq, dk, dv
    # one 16-byte step further is refused before any launch
    wide = torch.as_strided(torch.empty(S * (ss + 8), dtype=torch.bfloat16, device="cuda"), (B, S, Hq * d),
                            (S * (ss + 8), ss + 8, 1))
    with pytest.raises(fbl.FblError, match="UNSUPPORTED"):
        fbl.attn_fwd(wide, wide[:, :, :Hkv * d], wide[:, :, :Hkv * d], Hq, Hkv, scale, True)
    torch.cuda.empty_cache()


@pytest.mark.parametrize("causal,Hq,Hkv,d,S", [(True, 8, 2, 64, 200), (False, 4, 4, 128, 131), (True, 6, 3, 32, 97)])
def test_packed_qkv_entry_points(causal, Hq, Hkv, d, S):
    """attn_fwd_packed / attn_bwd_packed: Q, K, V read in place from one packed
    [B, S, (Hq + 2 Hkv) d] projection output through fbl_layout_packed_qkv
    descriptors, gradients written into one packed dQKV tensor; the device
    index map of each descriptor (plus its offset) equals the oracle's split."""
    import torch
    fbl = _lib()
    B = 2
    w = synth.Workload("packedqkv", B=B, S=S, Hq=Hq, Hkv=Hkv, d=d, dtype="bf16",
                       mask=synth.MASK_CAUSAL if causal else synth.MASK_NONE, seed=S + d)
    inp = synth.make_inputs(w)
    note(f"packed qkv causal={causal} Hq={Hq} Hkv={Hkv} d={d} S={S}")
    qkv = to_dev(np.concatenate([inp["q"], inp["k"], inp["v"]], axis=2), "bf16")
    do = to_dev(inp["do"], "bf16")
    o, lse = fbl.attn_fwd_packed(qkv, Hq, Hkv, causal=causal)
    dqkv = fbl.attn_bwd_packed(qkv, o, do, lse, Hq, Hkv, causal=causal)
    torch.cuda.synchronize()
    ref = oracle_fwd_bwd(inp)
    g = to_np(dqkv)
    got = {"o": to_np(o), "lse": to_np(lse), "dq": g[:, :, :Hq * d], "dk": g[:, :, Hq * d:(Hq + Hkv) * d],
           "dv": g[:, :, (Hq + Hkv) * d:]}
    errs, bad = compare(got, ref, "bf16")
    assert not bad, bad
    lq, lk, lv, ko, vo = fbl.fbl_layout_packed_qkv(fbl.FBL_BF16, B, S, Hq, Hkv, d)
    want = oracle.packed_qkv_offsets(B, S, Hq, Hkv, d)
    for l, off, base in ((lq, want[0], 0), (lk, want[1], ko), (lv, want[2], vo)):
        out = torch.full((off.size,), -7, dtype=torch.int64, device="cuda")
        fbl.fbl_layout_map_device(l, out)
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy().reshape(off.shape) + base, off)


def test_repeatability_and_no_allocation():
    """fwd and bwd outputs are bitwise repeatable (no atomics anywhere);
    the calls allocate no device memory when outputs and workspace are given."""
    import torch
    fbl = _lib()
    w = synth.Workload("rep", B=2, S=512, Hq=8, Hkv=4, d=128, dtype="bf16", mask=synth.MASK_CAUSAL, seed=4)
    inp = synth.make_inputs(w)
    note("repeatability")
    q, k, v, do = (to_dev(inp[n], "bf16") for n in ("q", "k", "v", "do"))
    scale = 1.0 / math.sqrt(w.d)
    o = torch.empty_like(q)
    lse = torch.empty((w.B, w.Hq, w.S), dtype=torch.float32, device="cuda")
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    lq, lk = fbl.layout_of(q, w.Hq), fbl.layout_of(k, w.Hkv)
    ws = torch.empty(fbl.fbl_attn_bwd_workspace(lq, lk), dtype=torch.uint8, device="cuda")
    runs = []
    for _ in range(3):
        torch.cuda.synchronize()
        before = torch.cuda.memory_allocated()
        fbl.attn_fwd(q, k, v, w.Hq, w.Hkv, scale, True, None, out=o, lse=lse)
        fbl.attn_bwd(q, k, v, o, do, lse, w.Hq, w.Hkv, scale, True, None, dq=dq, dk=dk, dv=dv, workspace=ws)
        torch.cuda.synchronize()
        assert torch.cuda.memory_allocated() == before
        runs.append([t.clone() for t in (o, lse, dq, dk, dv)])
    for r in runs[1:]:
        for x, y in zip(r, runs[0]):
            assert torch.equal(x, y)


def test_gradient_invariants_on_gpu_outputs():
    """sum_j dK_j = 0 and sum_j dV_j = sum_i dO_i per (batch, kv head), within
    the bf16 tolerance scaled by the number of summed rows."""
    w = synth.Workload("inv", B=2, S=256, Hq=8, Hkv=2, d=64, dtype="bf16", mask=synth.MASK_CAUSAL, seed=6)
    inp = synth.make_inputs(w)
    note("invariants")
    got = gpu_fwd_bwd(inp)
    d, G = w.d, w.Hq // w.Hkv
    for b in range(w.B):
        for g in range(w.Hkv):
            dk = got["dk"][b, :, g * d:(g + 1) * d]
            dv = got["dv"][b, :, g * d:(g + 1) * d]
            want = sum(inp["do"][b, :, h * d:(h + 1) * d].sum(axis=0) for h in range(g * G, (g + 1) * G))
            assert np.max(np.abs(dk.sum(axis=0))) <= 2e-2 * np.max(np.abs(dk)) * math.sqrt(w.S)
            assert np.max(np.abs(dv.sum(axis=0) - want)) <= 2e-2 * np.max(np.abs(want))


@pytest.mark.parametrize("scale", [-0.3, 0.0, 2.5])
def test_unusual_scales(scale):
    """Negative, zero and large softmax scales (the API takes any finite scale)."""
    import torch
    fbl = _lib()
    w = synth.Workload("scale", B=2, S=150, Hq=4, Hkv=2, d=64, dtype="bf16", mask=synth.MASK_CAUSAL, seed=12)
    inp = synth.make_inputs(w)
    note(f"scale={scale}")
    q, k, v, do = (to_dev(inp[n], "bf16") for n in ("q", "k", "v", "do"))
    o, lse = fbl.attn_fwd(q, k, v, w.Hq, w.Hkv, scale, True)
    dq, dk, dv = fbl.attn_bwd(q, k, v, o, do, lse, w.Hq, w.Hkv, scale, True, None)
    torch.cuda.synchronize()
    ro, rl = oracle.attn_fwd(inp["q"], inp["k"], inp["v"], w.Hq, w.Hkv, scale, True)
    rg = oracle.attn_bwd(inp["q"], inp["k"], inp["v"], inp["do"], w.Hq, w.Hkv, scale, True)
    got = {"o": to_np(o), "lse": to_np(lse), "dq": to_np(dq), "dk": to_np(dk), "dv": to_np(dv)}
    ref = {"o": ro, "lse": rl, "dq": rg[0], "dk": rg[1], "dv": rg[2]}
    names = ("o", "lse", "dv") if scale == 0.0 else ("o", "lse", "dq", "dk", "dv")
    errs, bad = compare(got, ref, "bf16", names)
    assert not bad, bad
    if scale == 0.0:
        assert np.max(np.abs(got["dq"])) == 0.0 and np.max(np.abs(got["dk"])) == 0.0


def test_binding_rejects_bad_lse_and_workspace():
    """On the GPU too, a saved log-sum-exp of the wrong type or shape, or a
    strided workspace, is refused by the binding before any launch."""
    import torch
    fbl = _lib()
    B, S, H, d = 2, 64, 2, 64
    q = torch.randn(B, S, H * d, device="cuda").to(torch.bfloat16)
    o, lse = fbl.attn_fwd(q, q, q, H, H, 0.125, False)
    note("binding rejects bad lse / workspace")
    for bad in (lse.to(torch.bfloat16), lse[:, :, :-1], lse.transpose(1, 2).contiguous().transpose(1, 2)):
        with pytest.raises(fbl.FblError):
            fbl.attn_bwd(q, q, q, o, q, bad, H, H, 0.125, False)
        with pytest.raises(fbl.FblError):
            fbl.attn_fwd(q, q, q, H, H, 0.125, False, lse=bad)
    ws = torch.empty(2 * fbl.fbl_attn_bwd_workspace(fbl.layout_of(q, H), fbl.layout_of(q, H)), dtype=torch.uint8,
                     device="cuda")
    with pytest.raises(fbl.FblError):
        fbl.attn_bwd(q, q, q, o, q, lse, H, H, 0.125, False, workspace=ws[::2])
    torch.cuda.synchronize()
