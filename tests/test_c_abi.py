"""The C ABI called from plain C11 (tests/c_abi/fbl_c_caller.c), no PyTorch
in the caller.  CPU: the header compiles as strict C11 and the host-only
entry points behave (index map against the token-major closed form, packed
QKV, workspace sizes, tile table).  GPU: attention forward and backward run
through hipMalloc'd buffers and the null stream, and the results meet the
oracle and equal, bit for bit, those of the Python binding on the same
inputs."""
import math
import os
import subprocess
import sys

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "c_abi"))

import cbuild as c_build  # noqa: E402  (tests/c_abi/cbuild.py)
import synth  # noqa: E402
from parity_util import compare, note, oracle_fwd_bwd  # noqa: E402

LIB = os.path.join(os.path.dirname(HERE), "paper_2607_21624_amd", "libfbl.so")


def test_header_is_c11_and_host_entry_points(tmp_path):
    if not os.path.exists(LIB):
        pytest.fail("libfbl.so is not built (run __graft_entry__.build())")
    exe = c_build.build(out=str(tmp_path / "fbl_c_caller"))
    r = subprocess.run([exe, "host"], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "host checks passed" in r.stdout


def _bf16_bits(x: np.ndarray) -> np.ndarray:
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).view(torch.int16).numpy()


def _from_bits(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


@pytest.mark.gpu
def test_attention_from_plain_c(tmp_path):
    import torch
    import paper_2607_21624_amd as fbl
    exe = c_build.OUT
    assert os.path.exists(exe), "the C caller is not built (run __graft_entry__.build())"
    w = synth.Workload("c_abi", B=2, S=200, Hq=4, Hkv=2, d=128, dtype="bf16", mask=synth.MASK_CAUSAL, seed=31)
    inp = synth.make_inputs(w)
    scale = 1.0 / math.sqrt(w.d)
    note("plain-C caller: attention B=2 S=200 Hq=4 Hkv=2 d=128 causal")
    bits = {n: _bf16_bits(inp[n]) for n in ("q", "k", "v", "do")}
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(src, "wb") as f:
        f.write(np.array([w.B, w.S, w.Hq, w.Hkv, w.d, 1], dtype=np.int32).tobytes())
        f.write(np.array([scale], dtype=np.float32).tobytes())
        for n in ("q", "k", "v", "do"):
            f.write(bits[n].tobytes())
    r = subprocess.run([exe, "attn", str(src), str(dst)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    raw = open(dst, "rb").read()
    nq, nk = w.B * w.S * w.Hq * w.d, w.B * w.S * w.Hkv * w.d
    off, got = 0, {}
    for n, cnt, shape in (("o", nq, inp["q"].shape), ("dq", nq, inp["q"].shape), ("dk", nk, inp["k"].shape),
                          ("dv", nk, inp["k"].shape)):
        got[n] = np.frombuffer(raw, dtype=np.int16, count=cnt, offset=off).reshape(shape)
        off += 2 * cnt
    got["lse"] = np.frombuffer(raw, dtype=np.float32, count=w.B * w.Hq * w.S, offset=off).reshape(w.B, w.Hq, w.S)
    assert off + 4 * w.B * w.Hq * w.S == len(raw)
    c_out = {n: (_from_bits(v) if n != "lse" else v.astype(np.float64)) for n, v in got.items()}
    errs, bad = compare(c_out, oracle_fwd_bwd(inp), "bf16")
    note(f"plain-C caller rel errs {errs}")
    assert not bad, bad
    # the same kernels through the Python binding: identical bits
    dev = {n: torch.from_numpy(bits[n]).view(torch.bfloat16).to("cuda") for n in bits}
    o, lse = fbl.attn_fwd(dev["q"], dev["k"], dev["v"], w.Hq, w.Hkv, scale, True)
    dq, dk, dv = fbl.attn_bwd(dev["q"], dev["k"], dev["v"], o, dev["do"], lse, w.Hq, w.Hkv, scale, True)
    torch.cuda.synchronize()
    for n, t in (("o", o), ("dq", dq), ("dk", dk), ("dv", dv)):
        assert np.array_equal(t.view(torch.int16).cpu().numpy(), got[n]), n
    assert np.array_equal(lse.cpu().numpy(), got["lse"])


@pytest.mark.gpu
def test_projection_products_from_plain_c(tmp_path):
    """Y = X W, dX = dY W^T and dW = X^T dY through fbl_proj from plain C
    (automatic tile, extents ragged against every tile): they meet the oracle
    and equal, bit for bit, the Python binding's products on the same inputs."""
    import torch
    import oracle
    import paper_2607_21624_amd as fbl
    exe = c_build.OUT
    assert os.path.exists(exe), "the C caller is not built (run __graft_entry__.build())"
    M, K, N = 304, 520, 264
    rng = np.random.default_rng(17)
    mats = {"x": rng.standard_normal((M, K)), "w": rng.standard_normal((K, N)), "dy": rng.standard_normal((M, N))}
    bits = {n: _bf16_bits(m) for n, m in mats.items()}
    vals = {n: _from_bits(b) for n, b in bits.items()}  # the bf16-rounded operands, as the GPU sees them
    note(f"plain-C caller: projection products M={M} K={K} N={N}")
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(src, "wb") as f:
        f.write(np.array([M, K, N], dtype=np.int32).tobytes())
        for n in ("x", "w", "dy"):
            f.write(bits[n].tobytes())
    r = subprocess.run([exe, "proj", str(src), str(dst)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    raw = open(dst, "rb").read()
    assert len(raw) == 2 * (M * N + M * K + K * N)
    y = np.frombuffer(raw, dtype=np.int16, count=M * N).reshape(M, N)
    dx = np.frombuffer(raw, dtype=np.int16, count=M * K, offset=2 * M * N).reshape(M, K)
    dw = np.frombuffer(raw, dtype=np.int16, count=K * N, offset=2 * (M * N + M * K)).reshape(K, N)
    refs = {"y": oracle.proj_fwd(vals["x"], vals["w"]), "dx": oracle.proj_bwd_data(vals["dy"], vals["w"]),
            "dw": oracle.proj_bwd_weight(vals["x"], vals["dy"])}
    for n, got in (("y", y), ("dx", dx), ("dw", dw)):
        err = float(np.max(np.abs(_from_bits(got) - refs[n])) / np.max(np.abs(refs[n])))
        assert err <= 2e-2, (n, err)
    dev = {n: torch.from_numpy(b).view(torch.bfloat16).to("cuda") for n, b in bits.items()}
    py = {"y": fbl.proj(fbl.FBL_PROJ_FWD, dev["x"], dev["w"]),
          "dx": fbl.proj(fbl.FBL_PROJ_BWD_DATA, dev["dy"], dev["w"]),
          "dw": fbl.proj(fbl.FBL_PROJ_BWD_WEIGHT, dev["x"], dev["dy"])}
    torch.cuda.synchronize()
    for n, got in (("y", y), ("dx", dx), ("dw", dw)):
        assert np.array_equal(py[n].view(torch.int16).cpu().numpy(), got), n
