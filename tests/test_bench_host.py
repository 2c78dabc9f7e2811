"""Host-side logic of bench.py (CPU): the one-GPU guard, and the algorithmic
work counts that `value` and the roofline are computed from -- pinned by
closed forms, by the oracle's own mask (counted element by element), and by
the figures of the Llama-7B-like workload."""
import math
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import synth  # noqa: E402
from oracle import attention as oatt  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_llama7b_work_counts():
    w = synth.WORKLOADS["llama7b_causal"]
    pairs = bench.allowed_pairs(w, None)
    assert pairs == 32 * 4096 * 4097 // 2 == 268_500_992
    assert abs(14 * w.d * pairs / 1e9 - 481.154) < 1e-3
    nb = 4096 // 32
    assert bench.ds_blocks(w, None) == 32 * nb * (nb + 1) // 2          # 8256 blocks per head
    ab = bench.algorithmic_bytes(w, 2)
    assert ab["total"] == 403_701_760
    nq = 4096 * 32 * 128 * 2   # bytes of Q (and of K, V, O, dO, dQ, dK, dV) at this shape
    # per launch, each tensor it must touch once: the kv pass reads Q, dO, K, V and writes dK, dV;
    # the dQ pass reads K and writes dQ; the statistics pass reads O, dO and LSE
    lse = 32 * 4096 * 4
    assert ab["attn_bwd_kv"] == 6 * nq and ab["attn_bwd_dq"] == 2 * nq and ab["attn_bwd_stats"] == 2 * nq + lse
    assert ab["attn_fwd"] == 4 * nq + lse and ab["total"] == ab["attn_fwd"] + 8 * nq + lse
    # the one-launch backward touches each backward tensor once: the whole backward's share of the total
    assert ab["attn_bwd_fused"] == ab["total"] - ab["attn_fwd"]
    db = bench.design_bytes(w, 2)
    assert db["attn_bwd_dq"] == 32 * 8256 * 2048 and db["attn_bwd_kv"] == db["attn_bwd_dq"] + 2 * 32 * 4096 * 4


@pytest.mark.parametrize("name", ["bert_base_keypad", "gpt2_medium_causal", "tiny_mha_f32",
                                  "whisper_large_cross", "whisper_large_cross_keypad"])
def test_allowed_pairs_match_the_oracle_mask(name):
    w = {**synth.WORKLOADS, **synth.CROSS_WORKLOADS}[name]
    kv_len = None
    if w.mask & synth.MASK_KEY_PADDING:
        kv_len = synth.make_inputs(w)["kv_len"]
    want = 0
    for b in range(w.B):
        m = oatt._mask_for(b, w.S, w.Skv, bool(w.mask & synth.MASK_CAUSAL), kv_len)
        want += int(np.count_nonzero(m))
    assert bench.allowed_pairs(w, kv_len) == want * w.Hq


def test_ds_blocks_count_blocks_with_an_allowed_pair():
    """A 32 x 32 block is stored iff it holds at least one allowed pair (keys
    past kv_len need no block; causal blocks wholly above the diagonal none)."""
    for name in ("bert_base_keypad", "gpt2_medium_causal", "whisper_large_cross_keypad"):
        w = {**synth.WORKLOADS, **synth.CROSS_WORKLOADS}[name]
        kv_len = synth.make_inputs(w)["kv_len"] if w.mask & synth.MASK_KEY_PADDING else None
        want = 0
        for b in range(w.B):
            m = oatt._mask_for(b, w.S, w.Skv, bool(w.mask & synth.MASK_CAUSAL), kv_len)
            nq, nk = math.ceil(w.S / 32), math.ceil(w.Skv / 32)
            for qb in range(nq):
                for kb in range(nk):
                    want += bool(m[32 * qb:32 * qb + 32, 32 * kb:32 * kb + 32].any())
        assert bench.ds_blocks(w, kv_len) == want * w.Hq, name
