"""Helpers shared by the GPU parity tests: run the HIP path through the C ABI on
seeded inputs and compare with the fp64 oracle."""
import math
import sys

import numpy as np

import oracle
import synth

TOL = {"f32": 1e-4, "bf16": 2e-2}   # max|gpu - ref| / max|ref| per output tensor


def note(msg: str) -> None:
    sys.stderr.write(f"[gpu-case] {msg}\n")
    sys.stderr.flush()


def torch_dtype(dt: str):
    import torch
    return torch.bfloat16 if dt == "bf16" else torch.float32


def to_dev(x: np.ndarray, dt: str):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda").to(torch_dtype(dt))


def to_np(t) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    ninf_ref = np.isneginf(ref)
    if np.any(ninf_ref != np.isneginf(got)):
        return math.inf
    fin = ~ninf_ref
    if not fin.any():
        return 0.0
    denom = np.max(np.abs(ref[fin]))
    diff = np.max(np.abs(got[fin] - ref[fin]))
    if not np.isfinite(diff):
        return math.inf
    return diff / denom if denom > 0 else diff


def gpu_fwd_bwd(inp: dict, stream=None, dO=None, workspace: str = "full"):
    """Run fbl_attn_fwd then fbl_attn_bwd on the inputs of one workload.
    workspace "full" (fbl_attn_bwd_workspace bytes: dQ from the stored dS for
    bf16, and the key/value pass split where the shape calls for it), "ds"
    (statistics and dS only: stored dS, no split) or "min"
    (fbl_attn_bwd_workspace_min bytes: dQ recomputes S and dP).
    Returns a dict of numpy float64 arrays (o, lse, dq, dk, dv)."""
    import torch
    import paper_2607_21624_amd as fbl
    w = inp["workload"]
    dt = w.dtype
    q, k, v = to_dev(inp["q"], dt), to_dev(inp["k"], dt), to_dev(inp["v"], dt)
    do = to_dev(inp["do"] if dO is None else dO, dt)
    kv_len = None
    if inp["kv_len"] is not None:
        kv_len = torch.from_numpy(inp["kv_len"].astype(np.int32)).to("cuda")
    causal = bool(w.mask & synth.MASK_CAUSAL)
    scale = 1.0 / math.sqrt(w.d)
    o, lse = fbl.attn_fwd(q, k, v, w.Hq, w.Hkv, scale, causal, kv_len)
    lq, lk = fbl.layout_of(q, w.Hq), fbl.layout_of(k, w.Hkv)
    if workspace == "full":
        size = fbl.fbl_attn_bwd_workspace(lq, lk)
    elif workspace == "ds":  # statistics and dS blocks only: stored dS, key/value pass not split
        size = fbl.fbl_attn_bwd_workspace_min(lq, lk) + w.B * w.Hq * -(-w.S // 32) * -(-w.Skv // 32) * 2048
    else:
        size = fbl.fbl_attn_bwd_workspace_min(lq, lk)
    ws = torch.empty(size, dtype=torch.uint8, device="cuda")
    dq, dk, dv = fbl.attn_bwd(q, k, v, o, do, lse, w.Hq, w.Hkv, scale, causal, kv_len, workspace=ws)
    torch.cuda.synchronize()
    return {"o": to_np(o), "lse": to_np(lse), "dq": to_np(dq), "dk": to_np(dk), "dv": to_np(dv)}


def oracle_fwd_bwd(inp: dict, kv_heads=None):
    """Oracle outputs, optionally only for a subset of key/value heads (and
    the query heads of their groups); heads are independent, so a subset is
    exactly the oracle's answer for those heads."""
    w = inp["workload"]
    d, G = w.d, w.Hq // w.Hkv
    q, k, v, do = inp["q"], inp["k"], inp["v"], inp["do"]
    Hq, Hkv = w.Hq, w.Hkv
    if kv_heads is not None:
        qh = [g * G + j for g in kv_heads for j in range(G)]
        cols = lambda heads: np.concatenate([np.arange(h * d, (h + 1) * d) for h in heads])
        q, do = q[:, :, cols(qh)], do[:, :, cols(qh)]
        k, v = k[:, :, cols(kv_heads)], v[:, :, cols(kv_heads)]
        Hq, Hkv = len(qh), len(kv_heads)
    causal = bool(w.mask & synth.MASK_CAUSAL)
    scale = 1.0 / math.sqrt(d)
    o, lse = oracle.attn_fwd(q, k, v, Hq, Hkv, scale, causal, inp["kv_len"])
    dq, dk, dv = oracle.attn_bwd(q, k, v, do, Hq, Hkv, scale, causal, inp["kv_len"])
    return {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv}


def select_heads(out: dict, w, kv_heads):
    """Restrict GPU outputs to the heads oracle_fwd_bwd(kv_heads=...) computed."""
    if kv_heads is None:
        return out
    d, G = w.d, w.Hq // w.Hkv
    qh = [g * G + j for g in kv_heads for j in range(G)]
    cols = lambda heads: np.concatenate([np.arange(h * d, (h + 1) * d) for h in heads])
    return {"o": out["o"][:, :, cols(qh)], "lse": out["lse"][:, qh, :], "dq": out["dq"][:, :, cols(qh)],
            "dk": out["dk"][:, :, cols(kv_heads)], "dv": out["dv"][:, :, cols(kv_heads)]}


def compare(got: dict, ref: dict, dt: str, names=("o", "lse", "dq", "dk", "dv")):
    errs = {n: rel_err(got[n], ref[n]) for n in names}
    bad = {n: e for n, e in errs.items() if not e <= TOL[dt]}
    return errs, bad
