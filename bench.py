#!/usr/bin/env python3
"""Attention forward+backward throughput on one MI355X.

One step = the whole hot path on one batch of synthetic token-major input:
fbl_attn_fwd (O, LSE) then the three backward launches (row statistic and
dQ-accumulator reset, main pass, dQ conversion), all through the C ABI on
torch's current stream.  Inputs, outputs and the workspace are resident in
HBM before the timed region; nothing is allocated inside it.

Prints one JSON line.  `value` is algorithmic TFLOP/s of fwd+bwd: 14*d FLOPs
per (query, key) pair the mask allows, per query head (4*d forward: QK^T and
PV; 10*d backward: the QK^T recompute, dO V^T, P^T dO, dS^T Q and dS K).

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # dense MFMA, 256 CU x 4096 flop/clk x 2.4 GHz
PEAK_F32_TFLOPS = 157.3
# bf16 32x32x16 MFMA rate measured by a probe kernel on this part (4+ independent
# accumulators, operands held constant); with random operands the chip's power
# limit lowers the clock (a large library GEMM runs about 30% slower than on zeros)
MEASURED_BF16_TFLOPS = 2450.0
PEAK_HBM_GBS = 8000.0


def allowed_pairs(w, kv_len) -> int:
    """Number of (query, key) pairs the mask allows, summed over batch and query heads."""
    S = w.S
    total = 0
    for b in range(w.B):
        L = w.Skv if kv_len is None else int(min(max(int(kv_len[b]), 0), w.Skv))
        if w.mask & 1:
            # query i sees keys j <= i, j < L
            total += sum(min(i + 1, L) for i in range(S)) if L < S else S * (S + 1) // 2
        else:
            total += S * L
    return total * w.Hq


def ds_blocks(w, kv_len) -> int:
    """32x32 dS blocks the key/value pass stores and the dQ pass reads: per
    (batch, query head), blocks (qb, kb) with kb < ceil(len/32) and, causal,
    kb <= qb (qb < ceil(S/32))."""
    nb = (w.S + 31) // 32
    total = 0
    for b in range(w.B):
        L = w.Skv if kv_len is None else int(min(max(int(kv_len[b]), 0), w.Skv))
        nk = (L + 31) // 32
        total += sum(min(nk, qb + 1) for qb in range(nb)) if w.mask & 1 else nb * nk
    return total * w.Hq


def algorithmic_bytes(w, es: int, kv_len=None) -> dict:
    """Minimum HBM traffic per kernel launch, as the measured metric defines it:
    each tensor of the step read or written once -- the forward reads Q, K, V
    and writes O, LSE; the backward reads Q, K, V, O, dO, LSE and writes dQ,
    dK, dV -- split over the backward's launches by which one touches each
    tensor.  Intermediates of this design (the row statistics, the dS blocks
    the kv pass writes and the dQ pass reads) are not algorithmic; they are
    reported separately by design_bytes."""
    nq = w.B * w.S * w.Hq * w.d * es
    nk = w.B * w.Skv * w.Hkv * w.d * es
    lse = w.B * w.Hq * w.S * 4
    return {"attn_fwd": 2 * nq + 2 * nk + lse,              # read Q K V, write O LSE
            "attn_bwd_stats": 2 * nq + lse,                 # read O dO LSE
            "attn_bwd_kv": 2 * nq + 2 * nk + 2 * nk,        # read Q dO K V, write dK dV
            "attn_bwd_dq": nk + nq,                         # read K, write dQ
            "attn_bwd_q": nk + nq,                          # (fp32: the recomputing dQ pass, same split)
            "attn_bwd_fused": 4 * nq + 4 * nk + lse,        # one launch: read Q O dO LSE K V, write dQ dK dV
            "total": (2 * nq + 2 * nk + lse) + (3 * nq + 2 * nk + lse + nq + 2 * nk)}


def design_bytes(w, es: int, kv_len=None) -> dict:
    """HBM bytes of this design's intermediates per launch: the statistics rows
    (8 bytes per query row, written by the statistics pass and read by the kv
    pass) and the bf16 dS blocks (written by the kv pass, read by the dQ pass)."""
    stats = 2 * w.B * w.Hq * w.S * 4
    ds = ds_blocks(w, kv_len) * 2048 if es == 2 else 0
    return {"attn_bwd_stats": stats, "attn_bwd_kv": stats + ds, "attn_bwd_dq": ds}


KERNEL_SOURCES = ("attn_fwd.hip", "attn_fwd_bf16.hip", "attn_bwd.hip", "attn_bwd_kv.hip", "attn_bwd_q.hip",
                  "attn_bwd_dq.hip", "attn_tiles.hpp", "stage.hpp", "cdna4.hpp", "tokmap.hpp")


def sources_sha() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2607_21624_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _tiles_str(tiles) -> str:
    return "none" if tiles is None else ",".join(str(t) for t in tiles)


def measured_traffic(workload: str, tiles=None):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE/WRITE_SIZE summary,
    only if it was taken on the kernel sources as they are now and with the attention
    tiles this run uses (else None)."""
    path = os.path.join(ROOT, "profiles", f"attn_{workload}_hbm_traffic.txt")
    if not os.path.exists(path):
        return None
    out, sha, rec_tiles = {}, None, None
    for line in open(path):
        line = line.strip()
        if line.startswith("sha="):
            sha = line[4:]
        elif line.startswith("tiles="):
            rec_tiles = line[6:]
        elif line and not line.startswith("#"):
            name, *kv = line.split()
            d = dict(x.split("=") for x in kv)
            out[name] = int(d["fetch_bytes"]) + int(d["write_bytes"])
    return out if sha == sources_sha() and rec_tiles == _tiles_str(tiles) else None


def traced_launch_us(workload: str, tiles=None):
    """Average launch duration (us) per kernel over the timed steps of the
    committed rocprofv3 kernel trace of this workload, only if it was taken on
    the kernel sources as they are now and with the attention tiles this run
    uses (else None)."""
    path = os.path.join(ROOT, "profiles", f"attn_{workload}_kernel_trace.txt")
    if not os.path.exists(path):
        return None
    out, sha, rec_tiles = {}, None, None
    for line in open(path):
        line = line.strip()
        if line.startswith("# kernel sources sha256[:16] = "):
            sha = line.split("= ")[1].split()[0]
        elif line.startswith("# attention tiles (forward, kv, dQ) = "):
            rec_tiles = line.split("= ")[1]
        elif line.startswith("timed "):
            _, name, us = line.split()[:3]
            out[name] = float(us)
    return out if sha == sources_sha() and rec_tiles == _tiles_str(tiles) else None


def cpu_baseline(w, inp, budget_s: float):
    """The fp64 oracle on a bounded sample of the same workload: whole heads of
    batch 0 (full sequence), one at a time, until `budget_s` seconds pass."""
    import numpy as np

    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count()
    d, G = w.d, w.Hq // w.Hkv
    scale = 1.0 / math.sqrt(d)
    kv = inp["kv_len"]
    done_pairs = 0
    heads = 0
    t0 = time.perf_counter()
    for g in range(w.Hkv):
        qh = list(range(g * G, (g + 1) * G))
        qcols = np.concatenate([np.arange(h * d, (h + 1) * d) for h in qh])
        kcols = np.arange(g * d, (g + 1) * d)
        q = inp["q"][:1, :, qcols]
        do = inp["do"][:1, :, qcols]
        k = inp["k"][:1, :, kcols]
        v = inp["v"][:1, :, kcols]
        kl = None if kv is None else kv[:1]
        oracle.attn_fwd(q, k, v, G, 1, scale, bool(w.mask & 1), kl)
        oracle.attn_bwd(q, k, v, do, G, 1, scale, bool(w.mask & 1), kl)
        heads += G
        sub = type(w)(w.name, B=1, S=w.S, Hq=G, Hkv=1, d=d, dtype=w.dtype, mask=w.mask, S_kv=w.S_kv)
        done_pairs += allowed_pairs(sub, kl)
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    flops = 14 * d * done_pairs
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": f"batch 0, query heads 0..{heads - 1} of {w.Hq} (full S={w.S}), fp64 numpy fwd+bwd, "
                      f"{dt:.1f} s, {flops / 1e9:.1f} GFLOP algorithmic",
            "seconds": dt, "host_cpus": os.cpu_count()}


def bench_proj(args, fbl, torch, np):
    """Projection products at one shape: per product and output tile, the
    average of `steps` launches timed with HIP events on the current stream
    (inputs resident, outputs preallocated).  `value` is the three products
    back to back with the automatic tile choice: 3 * 2 M K N flops per step."""
    M, K, N = (int(x) for x in args.proj_shape.split(","))
    g = torch.Generator(device="cpu").manual_seed(0)
    mk = lambda r, c: torch.randn(r, c, generator=g).to(device="cuda", dtype=torch.bfloat16)
    X, W, dY = mk(M, K), mk(K, N), mk(M, N)
    Y, dX, dW = (torch.empty(s, dtype=torch.bfloat16, device="cuda") for s in ((M, N), (M, K), (K, N)))
    ops = {"fwd": (fbl.FBL_PROJ_FWD, X, W, Y), "bwd_data": (fbl.FBL_PROJ_BWD_DATA, dY, W, dX),
           "bwd_weight": (fbl.FBL_PROJ_BWD_WEIGHT, X, dY, dW)}
    info = fbl.gemm_tiles()
    name = lambda g: f"{g['bm']}x{g['bn']}x{g['bk']}/w{g['wm']}{g['wn']}{g['wk']}"
    tiles = {"auto": fbl.FBL_GEMM_TILE_AUTO}
    tiles.update({f"t{t}:{name(g)}": t for t, g in info.items()})
    stream = torch.cuda.current_stream()
    flops = 2.0 * M * K * N
    # half a second of the three products first, so that the first timed
    # entry does not run while the clocks are still ramping up
    t_end = time.perf_counter() + 0.5
    while time.perf_counter() < t_end:
        for op, a, b, c in ops.values():
            fbl.proj(op, a, b, out=c)
        torch.cuda.synchronize()
    res = {}
    for name, (op, a, b, c) in ops.items():
        res[name] = {}
        for tn, t in tiles.items():
            try:
                call = lambda: fbl.proj(op, a, b, out=c, tile=t)
                call()
            except fbl.FblError:
                continue
            for _ in range(args.warmup):
                call()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record(stream)
            for _ in range(args.steps):
                call()
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / args.steps
            res[name][tn] = {"ms": round(ms, 4), "tflops": round(flops / (ms * 1e-3) / 1e12, 1)}
    step_ms = sum(res[n]["auto"]["ms"] for n in ops)
    tf = 3 * flops / (step_ms * 1e-3) / 1e12
    best = max(res[n][t]["tflops"] for n in ops for t in res[n])
    print(json.dumps({
        "metric": "projection products Y = X W, dX = dY W^T, dW = X^T dY: TFLOP/s at 1 GPU",
        "value": round(tf, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(step_ms, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded N(0,1))",
        "config": {"workload": "proj", "M": M, "K": K, "N": N, "layout": "token-major rows, no transposed copies"},
        "pct_peak": round(100 * tf / PEAK_BF16_TFLOPS, 2),
        "roofline": {"bound": "mfma", "achieved": best, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(best / PEAK_BF16_TFLOPS, 4), "traffic": None},
        "per_op": res,
    }), flush=True)


def bench_block(args, fbl, torch, np):
    """A whole attention block, forward and backward, with no layout copy: the
    QKV projection writes one packed [B*S, (Hq + 2Hkv) d] buffer, attention
    reads Q, K, V from it in place and writes dQ, dK, dV into a packed
    gradient buffer, and the output projection and both weight gradients read
    the token-major activations as they are.  Llama-7B-like layer (B=1,
    S=4096, 32 heads of 128, causal) unless --workload names another
    self-attention shape.  value = algorithmic FLOPs of the eight projection
    products and the attention step, over the timed step."""
    import synth
    w = {**synth.WORKLOADS, **synth.PAPER_MHA_SHAPES}[args.workload]
    if w.dtype != "bf16" or w.Skv != w.S or w.mask & synth.MASK_KEY_PADDING:
        raise SystemExit("--op block takes a bf16 self-attention workload without key padding")
    B, S, Hq, Hkv, d = w.B, w.S, w.Hq, w.Hkv, w.d
    causal = bool(w.mask & synth.MASK_CAUSAL)
    Dm, P, M = Hq * d, (Hq + 2 * Hkv) * d, B * S
    g = torch.Generator(device="cpu").manual_seed(0)
    mk = lambda r, c, sc=1.0: (sc * torch.randn(r, c, generator=g)).to(device="cuda", dtype=torch.bfloat16)
    X, dY = mk(M, Dm), mk(M, Dm)
    Wqkv, Wo = mk(Dm, P, 1 / math.sqrt(Dm)), mk(Hq * d, Dm, 1 / math.sqrt(Hq * d))
    qkv = torch.empty(M, P, dtype=torch.bfloat16, device="cuda")
    o3 = torch.empty(B, S, Hq * d, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(B, Hq, S, dtype=torch.float32, device="cuda")
    Y, dO = torch.empty(M, Dm, dtype=torch.bfloat16, device="cuda"), torch.empty(M, Hq * d, dtype=torch.bfloat16, device="cuda")
    dWo, dqkv = torch.empty(Hq * d, Dm, dtype=torch.bfloat16, device="cuda"), torch.empty(M, P, dtype=torch.bfloat16, device="cuda")
    dX, dWqkv = torch.empty(M, Dm, dtype=torch.bfloat16, device="cuda"), torch.empty(Dm, P, dtype=torch.bfloat16, device="cuda")
    qkv3, dqkv3, o = qkv.view(B, S, P), dqkv.view(B, S, P), o3.view(M, Hq * d)
    lq, lk, _, _, _, _ = fbl.fbl._packed(qkv3, Hq, Hkv)
    ws = torch.empty(fbl.fbl_attn_bwd_workspace(lq, lk), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    stages = [
        ("qkv_proj", lambda: fbl.proj(fbl.FBL_PROJ_FWD, X, Wqkv, out=qkv)),
        ("attn_fwd", lambda: fbl.attn_fwd_packed(qkv3, Hq, Hkv, causal=causal, out=o3, lse=lse)),
        ("out_proj", lambda: fbl.proj(fbl.FBL_PROJ_FWD, o, Wo, out=Y)),
        ("out_proj_bwd", lambda: (fbl.proj(fbl.FBL_PROJ_BWD_DATA, dY, Wo, out=dO),
                                  fbl.proj(fbl.FBL_PROJ_BWD_WEIGHT, o, dY, out=dWo))),
        ("attn_bwd", lambda: fbl.attn_bwd_packed(qkv3, o3, dO.view(B, S, Hq * d), lse, Hq, Hkv, causal=causal,
                                                 dqkv=dqkv3, workspace=ws)),
        ("qkv_proj_bwd", lambda: (fbl.proj(fbl.FBL_PROJ_BWD_DATA, dqkv, Wqkv, out=dX),
                                  fbl.proj(fbl.FBL_PROJ_BWD_WEIGHT, X, dqkv, out=dWqkv))),
    ]

    def step(ev=None):
        for i, (_, f) in enumerate(stages):
            if ev is not None:
                ev[i].record(stream)
            f()
        if ev is not None:
            ev[-1].record(stream)

    spin = spin_up(step, args.spinup_s)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    mem_before = torch.cuda.memory_allocated()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(stages) + 1)] for _ in range(args.steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for i in range(args.steps):
        step(evs[i])
    stop.record(stream)
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated() == mem_before, "the timed steps allocated device memory"
    ms_per_step = start.elapsed_time(stop) / args.steps
    stage_ms = {n: round(float(np.mean([e[i].elapsed_time(e[i + 1]) for e in evs])), 4)
                for i, (n, _) in enumerate(stages)}
    pairs = B * Hq * (S * (S + 1) // 2 if causal else S * S)
    proj_flops = 3 * 2.0 * M * Dm * P + 3 * 2.0 * M * (Hq * d) * Dm
    attn_flops = 14.0 * d * pairs
    flops = proj_flops + attn_flops
    tflops = flops / (ms_per_step * 1e-3) / 1e12
    kernels = None if args.no_kernel_list else dispatched_kernels(step)
    foreign = None if kernels is None else [n for n in kernels if not any(t in n for t in ("attn_", "proj_gemm"))]
    print(json.dumps({
        "metric": "attention block fwd+bwd (QKV projection, attention, output projection) TFLOP/s at 1 GPU; "
                  "layout-copy bytes (=0)",
        "value": round(tflops, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "spinup": {"seconds": args.spinup_s, "steps": spin},
        "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded N(0,1) activations and gradients, scaled N(0,1) weights)",
        "config": {"workload": f"attention block, {w.name} shape", "B": B, "S": S, "Hq": Hq, "Hkv": Hkv, "d": d,
                   "model_width": Dm, "qkv_width": P, "mask": "causal" if causal else "none",
                   "layout": "token-major; packed QKV"},
        "pct_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 2),
        "stage_ms": stage_ms,
        "algorithmic_gflop": {"projections": round(proj_flops / 1e9, 2), "attention": round(attn_flops / 1e9, 2)},
        "layout_copy_bytes": 0 if foreign == [] else None,
        "dispatched_kernels": kernels,
    }), flush=True)


def spin_up(step, seconds: float) -> int:
    """Run `step` back to back for `seconds` (untimed, before the warmup steps):
    under sustained load the chip's clocks and the first touches of the
    buffers take some tens of milliseconds to settle, longer than a few warmup
    steps of a sub-millisecond step.  Returns the number of steps run."""
    import torch
    n, t_end = 0, time.perf_counter() + seconds
    while time.perf_counter() < t_end:
        for _ in range(4):
            step()
        n += 4
        torch.cuda.synchronize()
    return n


def dispatched_kernels(step):
    """Kernel names dispatched by one step (torch profiler; None if unavailable)."""
    try:
        import torch
        from torch.profiler import ProfilerActivity, profile
        with profile(activities=[ProfilerActivity.CUDA]) as prof:
            step()
            torch.cuda.synchronize()
        names = sorted({e.key for e in prof.key_averages() if e.device_time_total > 0})
        return names or None
    except Exception:
        return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--spinup-s", type=float, default=0.2,
                    help="seconds of untimed steps before the warmup steps (clock and first-touch settling)")
    ap.add_argument("--workload", default="llama7b_causal")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-list", action="store_true",
                    help="skip the torch-profiler dispatch listing (use under rocprofv3)")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of the step captured in a HIP graph (per-kernel times stay eager)")
    ap.add_argument("--op", default="attention", choices=["attention", "proj", "block"],
                    help="attention: the fwd+bwd step (default); proj: the projection products Y = X W, dX = dY W^T, "
                         "dW = X^T dY on token-major activations, every tile shape; block: a whole attention block "
                         "(QKV projection into a packed buffer, attention in place, output projection) fwd+bwd")
    ap.add_argument("--proj-shape", default="512,2048,8192", help="M,K,N for --op proj")
    ap.add_argument("--tiles", default=None,
                    help="explicit attention tile ids FWD,KV,DQ (bf16; -1 = automatic); default: the automatic choice")
    ap.add_argument("--tune", action="store_true",
                    help="run the measured tile selection (fbl_attn_tune) on the inputs before the warmup; the step "
                         "then runs the tuned tiles")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="instead of attention, run 5 plain device copies of this many MiB (calibrates the HBM "
                         "byte counters FETCH_SIZE / WRITE_SIZE against a kernel of known traffic)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only: the attention path has no multi-GPU mode in this build "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE {world}).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    if args.copy_mib:
        n = args.copy_mib * (1 << 20) // 2
        src = torch.ones(n, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_mib": args.copy_mib, "bytes_read_per_copy": 2 * n, "bytes_written_per_copy": 2 * n}))
        return

    import paper_2607_21624_amd as fbl
    import synth

    if args.op == "proj":
        bench_proj(args, fbl, torch, np)
        return
    if args.op == "block":
        bench_block(args, fbl, torch, np)
        return

    w = {**synth.WORKLOADS, **synth.CROSS_WORKLOADS, **synth.PAPER_MHA_SHAPES}[args.workload]
    inp = synth.make_inputs(w)
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    dev = lambda x: torch.from_numpy(x).to("cuda").to(dt)
    q, k, v, do = dev(inp["q"]), dev(inp["k"]), dev(inp["v"]), dev(inp["do"])
    kv_len = None if inp["kv_len"] is None else torch.from_numpy(inp["kv_len"]).to("cuda")
    causal = bool(w.mask & synth.MASK_CAUSAL)
    scale = 1.0 / math.sqrt(w.d)
    o = torch.empty_like(q)
    lse = torch.empty((w.B, w.Hq, w.S), dtype=torch.float32, device="cuda")
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ws = torch.empty(fbl.fbl_attn_bwd_workspace(fbl.layout_of(q, w.Hq), fbl.layout_of(k, w.Hkv)),
                     dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    tiles = [fbl.FBL_ATTN_TILE_AUTO] * 3
    if args.tiles:
        tiles = [int(x) for x in args.tiles.split(",")]
    lq_, lk_ = fbl.layout_of(q, w.Hq), fbl.layout_of(k, w.Hkv)
    qname = "attn_bwd_dq" if w.dtype == "bf16" else "attn_bwd_q"
    # the backward as the library runs it: one launch up to 128 keys with automatic
    # tiles, else its three phases, each bracketed by events of its own
    fused = fbl.attn_bwd_launches(lq_, lk_, int(w.mask), ws.numel(), kv_tile=tiles[1], dq_tile=tiles[2]) == 1
    if fused:
        bwd_phases = [("attn_bwd_fused", fbl.FBL_BWD_ALL)]
    else:
        bwd_phases = [("attn_bwd_stats", fbl.FBL_BWD_PREP), ("attn_bwd_kv", fbl.FBL_BWD_KV), (qname, fbl.FBL_BWD_Q)]
    n_ev = 2 + len(bwd_phases)

    def bwd(phases):
        fbl.attn_bwd(q, k, v, o, do, lse, w.Hq, w.Hkv, scale, causal, kv_len, dq=dq, dk=dk, dv=dv, workspace=ws,
                     phases=phases, kv_tile=tiles[1], dq_tile=tiles[2])

    def step(ev=None, around=None):
        # ev: events recorded between the launches (n_ev of them), or, with
        # `around` naming a launch, only just before and after that one (2)
        def mark(i, name, after):
            if ev is None:
                return
            if around is None:
                ev[i].record(stream)
            elif around == name:
                ev[1 if after else 0].record(stream)
        mark(0, "attn_fwd", False)
        fbl.attn_fwd(q, k, v, w.Hq, w.Hkv, scale, causal, kv_len, out=o, lse=lse, tile=tiles[0])
        mark(1, "attn_fwd", True)
        for i, (n, ph) in enumerate(bwd_phases):
            if around is not None:
                mark(0, n, False)
            bwd(ph)
            mark(2 + i, n, True)

    spin = spin_up(step, args.spinup_s)
    tune = None
    if args.tune:  # measured at steady clocks (after the spin-up), then the chosen tiles run
        best, tms, _ = fbl.attn_tune(q, k, v, do, w.Hq, w.Hkv, scale, causal, kv_len, o=o, lse=lse, dq=dq, dk=dk,
                                     dv=dv, workspace=ws, reps=5)
        torch.cuda.synchronize()
        tune = {"chosen": list(best), "ms": {str(t): round(x, 4) for t, x in tms.items()}}
    auto = fbl.attn_auto_tiles(lq_, lk_, int(w.mask)) if w.dtype == "bf16" else None
    run_tiles = None if auto is None else [a if t == fbl.FBL_ATTN_TILE_AUTO else t for t, a in zip(tiles, auto)]
    # Algorithmic FLOPs per launch (2*d per allowed pair per matrix product):
    #   attn_fwd        QK^T, PV                                    4*d
    #   attn_bwd_kv     QK^T recompute, dO V^T, P^T dO, dS^T Q      8*d
    #   attn_bwd_dq     dS K from the dS the kv pass stored         2*d
    #   attn_bwd_fused  the kv products and dS K in one launch     10*d
    #   (fp32 storage has no stored-dS path: attn_bwd_q recomputes QK^T and dO V^T, 6*d executed)
    alg = {"attn_fwd": 4, "attn_bwd_kv": 8, "attn_bwd_dq": 2, "attn_bwd_q": 2, "attn_bwd_fused": 10}
    executed = {**alg, "attn_bwd_q": 6}
    # The dominant launch (most algorithmic FLOPs) is timed inside the timed
    # steps with events just around it (for the roofline): each event recorded
    # between two launches adds a gap to the step.  Every launch is timed in as
    # many untimed steps after them.
    dom = max((n for n in ["attn_fwd"] + [n for n, _ in bwd_phases] if n in alg), key=lambda n: alg[n])

    def launch_ms(evs):
        t = {"attn_fwd": float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))}
        for i, (n, _) in enumerate(bwd_phases):
            t[n] = float(np.mean([e[1 + i].elapsed_time(e[2 + i]) for e in evs]))
        return t
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    mem_before = torch.cuda.memory_allocated()

    dom_evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(n_ev)] for _ in range(args.steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(args.steps):
        step(dom_evs[i], around=dom)
    stop.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    ms_per_step = total_ms / args.steps
    eager_ms_per_step = ms_per_step
    t_dom_timed = float(np.mean([e[0].elapsed_time(e[1]) for e in dom_evs]))
    assert torch.cuda.memory_allocated() == mem_before, "the timed steps allocated device memory"
    # every launch, over as many untimed steps
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    k_ms = launch_ms(evs)
    step_each = np.array([e[0].elapsed_time(e[-1]) for e in evs])   # each step, first to last launch
    fwd_each = np.array([e[0].elapsed_time(e[1]) for e in evs])
    bwd_each = step_each - fwd_each
    if args.graph:
        # the step's launches captured once and replayed: no host work per step
        # (capture and its memory pool come after the eager timing and its no-allocation check)
        side = torch.cuda.Stream()
        with torch.cuda.stream(side):
            step()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        spin_up(graph.replay, args.spinup_s)  # the capture left the GPU idle
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
        start.record(stream)
        for _ in range(args.steps):
            graph.replay()
        stop.record(stream)
        torch.cuda.synchronize()
        ms_per_step = start.elapsed_time(stop) / args.steps

    pairs = allowed_pairs(w, inp["kv_len"])
    flops = 14 * w.d * pairs
    tflops = flops / (ms_per_step * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    per_kernel = {n: (t, alg[n]) for n, t in k_ms.items() if n in alg}
    ktf = {n: a * w.d * pairs / (t * 1e-3) / 1e12 for n, (t, a) in per_kernel.items()}
    ktf_exec = {n: executed[n] * w.d * pairs / (per_kernel[n][0] * 1e-3) / 1e12 for n in per_kernel}
    a_dom = alg[dom]
    t_dom = t_dom_timed
    es = 2 if w.dtype == "bf16" else 4
    alg_bytes = algorithmic_bytes(w, es, inp["kv_len"])
    des_bytes = design_bytes(w, es, inp["kv_len"])
    traffic = measured_traffic(w.name, run_tiles)
    trace = traced_launch_us(w.name, run_tiles)
    dom_traffic = None if traffic is None else traffic.get(dom)
    dom_trace_us = None if trace is None else trace.get(dom)
    flops_launch = a_dom * w.d * pairs
    achieved = flops_launch / (t_dom * 1e-3) / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "traffic": dom_traffic, "kernel": dom,
                # achieved = flops_per_launch / avg_launch_ms, the launch timed with HIP events on the
                # stream it runs on, averaged over this run's timed steps
                "frac_source": "HIP events around this launch over the timed steps of this run",
                "avg_launch_ms": round(t_dom, 4), "flops_per_launch": flops_launch,
                # the same figure from the committed rocprofv3 kernel trace (timed steps), when it was
                # taken on the current sources
                "trace_avg_launch_ms": None if dom_trace_us is None else round(dom_trace_us / 1e3, 4),
                "trace_frac": None if dom_trace_us is None else round(flops_launch / (dom_trace_us * 1e-6) / 1e12 / peak, 4),
                "algorithmic_bytes_per_launch": alg_bytes[dom],
                "design_bytes_per_launch": des_bytes.get(dom, 0),
                # the paper's MemEfficiency (section 4.2): algorithmic over counted HBM bytes
                # (FETCH_SIZE + WRITE_SIZE, calibrated), when the counters match the sources
                "mem_efficiency": None if dom_traffic is None else round(alg_bytes[dom] / dom_traffic, 3),
                "hbm_gbs_measured": None if dom_traffic is None else round(dom_traffic / (t_dom * 1e-3) / 1e9, 1)}
    stat = lambda x: {"median": round(float(np.median(x)), 4), "min": round(float(np.min(x)), 4),
                      "max": round(float(np.max(x)), 4)}

    kernels = None if args.no_kernel_list else dispatched_kernels(step)
    foreign = None
    if kernels is not None:
        foreign = [n for n in kernels if not any(t in n for t in ("attn_fwd", "attn_bwd"))]

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, inp, args.cpu_budget)

    line = {
        "metric": "attn fwd+bwd TFLOP/s & % bf16 MFMA peak at 1 GPU; layout-copy bytes (=0)",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "spinup": {"seconds": args.spinup_s, "steps": spin},
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "launch": "hip graph replay" if args.graph else "eager (one host call per launch)",
        "eager_ms_per_step": round(eager_ms_per_step, 4),
        "dtype": w.dtype,
        "data": "synthetic (seeded N(0,1) token-major Q,K,V,dO)",
        "config": {"workload": w.name, "B": w.B, "S": w.S, "S_kv": w.Skv, "Hq": w.Hq, "Hkv": w.Hkv, "d": w.d,
                   "mask": {0: "none", 1: "causal", 2: "key_padding", 3: "causal+key_padding"}[w.mask],
                   "layout": "token-major [B,S,H*d]", "parallelism": "single GPU"},
        "pct_peak": round(100 * tflops / peak, 2),
        # against the bf16 MFMA rate a probe kernel reaches on this part (operands held constant)
        "pct_measured_mfma_peak": round(100 * tflops / MEASURED_BF16_TFLOPS, 2) if w.dtype == "bf16" else None,
        "ms": {"step": stat(step_each), "fwd": stat(fwd_each), "bwd": stat(bwd_each)},
        "layout_copy_bytes": 0 if foreign == [] else None,
        "dispatched_kernels": kernels,
        "bwd_launches": len(bwd_phases),
        # every launch, timed with events between the launches in as many untimed steps after the timed ones
        "kernel_ms": {n: round(t, 4) for n, t in k_ms.items()},
        # the HBM-bound launches: algorithmic bytes over their time
        "kernel_gbs_algorithmic": None if fused else {
            "attn_bwd_stats": round(alg_bytes["attn_bwd_stats"] / (k_ms["attn_bwd_stats"] * 1e-3) / 1e9, 1),
            qname: round(alg_bytes["attn_bwd_dq"] / (k_ms[qname] * 1e-3) / 1e9, 1)},
        "kernel_tflops_algorithmic": {n: round(v, 2) for n, v in ktf.items()},
        "kernel_tflops_executed": {n: round(v, 2) for n, v in ktf_exec.items()},
        "algorithmic_gflop": round(flops / 1e9, 3),
        "algorithmic_bytes": alg_bytes["total"],
        "roofline": roofline,
        "attn_tiles": run_tiles,
        "tune": tune,
        "cpu_baseline": cpu,
        "gpu_over_oracle": None if cpu is None else round(tflops / cpu["value"], 1),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
