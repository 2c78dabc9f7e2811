"""Seeded synthetic inputs for the attention forward/backward workloads.

This module is shared by the oracle-side tests and the HIP-side tests and bench.
It holds workload shapes and random draws only, none of the attention
arithmetic: every tensor it returns is an input (Q, K, V, dO, key lengths).

Draw recipe (one ``numpy.random.default_rng(seed)`` PCG64 stream per workload;
S is the query length, S_kv the key/value length, equal to S for
self-attention):
  Q  (B, S, Hq*d)      standard normal, fp64
  K  (B, S_kv, Hkv*d)  standard normal, fp64
  V  (B, S_kv, Hkv*d)  standard normal, fp64
  dO (B, S, Hq*d)      standard normal, fp64
  kv_len (B,)       integers uniform on [len_lo, len_hi] inclusive, only for
                    key-padding workloads, drawn after dO
Values are then rounded to the storage type: fp32 by IEEE round-to-nearest-even,
bf16 by rounding to fp32 first and then to bf16 with round-to-nearest-even on
the bit pattern.  The arrays handed out are float32 arrays whose values are
exactly representable in the storage type, so both the oracle (which upcasts to
fp64) and the GPU path (which casts to its storage type) see identical numbers.

All tensors are token-major: element (b, s, h, i) of a tensor with H heads of
width d sits at flat index ((b*S + s)*H + h)*d + i, i.e. the layout a QKV
projection writes, before any head split.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

MASK_NONE = 0
MASK_CAUSAL = 1
MASK_KEY_PADDING = 2


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    S: int
    Hq: int
    Hkv: int
    d: int
    dtype: str            # "f32" or "bf16": storage type of Q, K, V, O, dO, dQ, dK, dV
    mask: int             # bit 0 causal, bit 1 key padding
    seed: int = 0
    len_lo: int = 0       # key-padding length range (inclusive), used when mask & 2
    len_hi: int = 0
    note: str = field(default="", compare=False)
    S_kv: int = 0         # key/value tokens; 0 means S (self-attention)

    @property
    def Skv(self) -> int:
        return self.S_kv or self.S


# The five workload shapes measured and checked.  Names say what
# each one stands in for; the pretrained models themselves are not used.
WORKLOADS = {
    "tiny_mha_f32": Workload("tiny_mha_f32", B=1, S=64, Hq=2, Hkv=2, d=32, dtype="f32",
                             mask=MASK_NONE,
                             note="tiny MHA, fp32, no mask"),
    "bert_base_keypad": Workload("bert_base_keypad", B=8, S=128, Hq=12, Hkv=12, d=64, dtype="bf16",
                                 mask=MASK_KEY_PADDING, len_lo=32, len_hi=128,
                                 note="BERT-base-like encoder, key-padding lengths U[32,128]"),
    "gpt2_medium_causal": Workload("gpt2_medium_causal", B=4, S=1024, Hq=16, Hkv=16, d=64, dtype="bf16",
                                   mask=MASK_CAUSAL,
                                   note="GPT-2-medium-like causal decoder"),
    "llama32_1b_gqa": Workload("llama32_1b_gqa", B=2, S=2048, Hq=32, Hkv=8, d=64, dtype="bf16",
                               mask=MASK_CAUSAL,
                               note="Llama-3.2-1B-like causal GQA, 4 query heads per KV head"),
    "llama7b_causal": Workload("llama7b_causal", B=1, S=4096, Hq=32, Hkv=32, d=128, dtype="bf16",
                               mask=MASK_CAUSAL,
                               note="Llama-7B-like causal MHA, the headline workload"),
}

# Extra shapes from the paper's multi-head-attention layout experiment
# ([seq, heads, hidden] triples in the tile-based index transformation study).
PAPER_MHA_SHAPES = {
    "paper_mha_c1": Workload("paper_mha_c1", B=1, S=512, Hq=32, Hkv=32, d=64, dtype="bf16", mask=MASK_CAUSAL),
    "paper_mha_c2": Workload("paper_mha_c2", B=1, S=512, Hq=16, Hkv=16, d=64, dtype="bf16", mask=MASK_NONE),
    "paper_mha_c3": Workload("paper_mha_c3", B=1, S=512, Hq=8, Hkv=8, d=128, dtype="bf16", mask=MASK_CAUSAL),
}


# Cross-attention (S_kv != S): the decoder-side attention of the encoder-decoder
# models in the paper's evaluation, here Whisper-large-like (20 heads of 64;
# decoder tokens attend to the encoder's audio frames, 300 as in the paper's
# model table).  Not one of the five measured shapes above.
CROSS_WORKLOADS = {
    "whisper_large_cross": Workload("whisper_large_cross", B=2, S=448, S_kv=300, Hq=20, Hkv=20, d=64,
                                    dtype="bf16", mask=MASK_NONE,
                                    note="Whisper-large-like decoder cross-attention, 448 tokens x 300 frames"),
    "whisper_large_cross_keypad": Workload("whisper_large_cross_keypad", B=4, S=448, S_kv=300, Hq=20, Hkv=20,
                                           d=64, dtype="bf16", mask=MASK_KEY_PADDING, len_lo=100, len_hi=300,
                                           note="as above with padded encoder frames, lengths U[100,300]"),
}


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bf16 value (ties to even), returned as float32."""
    x32 = np.ascontiguousarray(x, dtype=np.float32)
    bits = x32.view(np.uint32).astype(np.uint64)
    rounded = ((bits + 0x7FFF + ((bits >> 16) & 1)) >> 16) << 16
    out = rounded.astype(np.uint32).view(np.float32)
    # keep NaN/Inf untouched (the draws never produce them)
    special = ~np.isfinite(x32)
    if special.any():
        out = out.copy()
        out[special] = x32[special]
    return out


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Bit patterns (uint16) of float32 values that are exactly representable in bf16."""
    x32 = np.ascontiguousarray(x, dtype=np.float32)
    return (x32.view(np.uint32) >> 16).astype(np.uint16)


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32)
    if dtype == "bf16":
        return round_to_bf16(x)
    raise ValueError(f"unknown dtype {dtype}")


def make_inputs(w: Workload, seed: Optional[int] = None, zero_q: bool = False) -> dict:
    """Draw the seeded inputs of workload ``w``.

    Returns a dict with float32 arrays ``q``, ``k``, ``v``, ``do`` (token-major,
    values exactly representable in ``w.dtype``), ``kv_len`` (int32 (B,) or
    None) and the workload under ``w``.
    """
    s = w.seed if seed is None else seed
    rng = np.random.default_rng(s)
    q = rng.standard_normal((w.B, w.S, w.Hq * w.d))
    k = rng.standard_normal((w.B, w.Skv, w.Hkv * w.d))
    v = rng.standard_normal((w.B, w.Skv, w.Hkv * w.d))
    do = rng.standard_normal((w.B, w.S, w.Hq * w.d))
    kv_len = None
    if w.mask & MASK_KEY_PADDING:
        kv_len = rng.integers(w.len_lo, w.len_hi + 1, size=w.B).astype(np.int32)
    if zero_q:
        q = np.zeros_like(q)
    return {
        "q": to_storage(q, w.dtype),
        "k": to_storage(k, w.dtype),
        "v": to_storage(v, w.dtype),
        "do": to_storage(do, w.dtype),
        "kv_len": kv_len,
        "workload": w,
        "seed": s,
    }


def random_workload(rng: np.random.Generator, *, dtype: str, d: int, max_s: int = 200,
                    name: str = "random") -> Workload:
    """A small random shape (ragged S, random mask, MHA or GQA) for parity sweeps."""
    B = int(rng.integers(1, 4))
    S = int(rng.integers(1, max_s + 1))
    Hkv = int(rng.integers(1, 4))
    G = int(rng.choice([1, 2, 4]))
    mask = int(rng.integers(0, 4))
    return Workload(name, B=B, S=S, Hq=Hkv * G, Hkv=Hkv, d=d, dtype=dtype, mask=mask,
                    seed=int(rng.integers(0, 2**31 - 1)), len_lo=1, len_hi=S)
