"""Seeded synthetic workloads for the FOCUS hot path.

This module is shared by the HIP path (through its tests and the benchmark) and
by the CPU oracle.  It holds shapes, seeds and random draws only: no part of the
FOCUS method (summary layout, compaction, attention, decode state) is computed
here, so that neither side can inherit a mistake from the other through it.
Every count that depends on the method (number of augmented tokens, cache
lengths) is passed in by the caller, which derives it on its own side.

The paper evaluates on human and viral DNA pushed through Evo-2 7B; neither the
sequences nor the weights are available, and the attention kernels' cost does
not depend on the values, so seeded N(0, 1) projections of one Evo-2-scale
attention layer (32 heads x 128) stand in for them.  The base seed 42 is the
seed of the paper's training recipe (hyper-parameter table).
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Sequence, Tuple

import numpy as np

BASE_SEED = 42

# Tensor tags folded into the seed so that Q, K, V and the per-step decode
# tensors of one workload never share a random stream.
_TENSOR_TAG = {"q": 1, "k": 2, "v": 3, "cache_k": 4, "cache_v": 5,
               "win_k": 6, "win_v": 7, "step_q": 8, "step_k": 9, "step_v": 10,
               "bases": 11}


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: batch of sequences plus one attention layer's shape.

    kmer: a single cadence for every window, or None when per-window cadences
    are drawn from kmer_choices (see kmer_draw).  kmer == 0 means no summary
    tokens (plain causal attention inside each window).
    """
    name: str
    index: int
    batch: int
    seq_nt: int
    window_nt: int
    kmer: Optional[int]
    heads: int
    kv_heads: int
    head_dim: int
    dtype: str                      # "f32" or "bf16"
    kmer_choices: Tuple[int, ...] = ()
    # decode only
    decode_steps: int = 0
    decode_cache_rows: int = 0
    decode_pos_max: int = 0
    extra: dict = field(default_factory=dict)


# The five workloads: tiny oracle check, 100 kb and 1 Mb single-layer prefill,
# a batch-8 ragged-cadence prefill and a batch-16 decode at ~1 Mb.
WORKLOADS = {
    "tiny_4kb_f32": Workload("tiny_4kb_f32", 0, batch=1, seq_nt=4_000, window_nt=1_000,
                             kmer=100, heads=1, kv_heads=1, head_dim=64, dtype="f32"),
    "prefill_100kb": Workload("prefill_100kb", 1, batch=1, seq_nt=100_000, window_nt=1_000,
                              kmer=100, heads=32, kv_heads=32, head_dim=128, dtype="bf16"),
    "prefill_1mb": Workload("prefill_1mb", 2, batch=1, seq_nt=1_000_000, window_nt=1_000,
                            kmer=100, heads=32, kv_heads=32, head_dim=128, dtype="bf16"),
    "ragged_b8_256kb": Workload("ragged_b8_256kb", 3, batch=8, seq_nt=256_000, window_nt=1_000,
                                kmer=None, heads=32, kv_heads=32, head_dim=128, dtype="bf16",
                                kmer_choices=(50, 100, 200, 500)),
    "decode_b16_1mb": Workload("decode_b16_1mb", 4, batch=16, seq_nt=1_000_000, window_nt=1_000,
                               kmer=100, heads=32, kv_heads=32, head_dim=128, dtype="bf16",
                               decode_steps=1_000, decode_cache_rows=10_000, decode_pos_max=1_000),
    # Dense causal comparison point: one 32 kb window with no summary tokens.
    "dense_32kb": Workload("dense_32kb", 5, batch=1, seq_nt=32_000, window_nt=32_000,
                           kmer=0, heads=32, kv_heads=32, head_dim=128, dtype="bf16"),
}


def seed_for(workload_index: int, tensor: str, seq: int = 0) -> int:
    """Deterministic seed for one tensor of one workload (and one sequence)."""
    return (BASE_SEED * 1_000_003 + workload_index * 10_007 + _TENSOR_TAG[tensor] * 101
            + seq) & 0x7FFF_FFFF


def windows_per_seq(seq_nt: int, window_nt: int) -> int:
    """Number of base-domain windows covering seq_nt bases (a plain ceiling)."""
    return -(-seq_nt // window_nt) if seq_nt > 0 else 0


def kmer_draw(w: Workload) -> np.ndarray:
    """Per-window cadences, int32 [batch * windows_per_seq], sequence-major.

    Uniform workloads repeat w.kmer; the ragged workload draws each window's
    cadence uniformly from w.kmer_choices with numpy's PCG64 seeded from the
    base seed and the workload index.
    """
    nw = windows_per_seq(w.seq_nt, w.window_nt)
    if w.kmer is not None:
        return np.full(w.batch * nw, w.kmer, dtype=np.int32)
    rng = np.random.default_rng(BASE_SEED + w.index)
    return rng.choice(np.asarray(w.kmer_choices, dtype=np.int32),
                      size=(w.batch, nw)).reshape(-1).astype(np.int32)


def decode_positions(w: Workload) -> np.ndarray:
    """Per-sequence starting position inside the current window (decode workload).

    p_b ~ U{1..decode_pos_max}: the number of augmented tokens of the current
    window that precede the first decode step.
    """
    rng = np.random.default_rng(BASE_SEED + w.index)
    return rng.integers(1, w.decode_pos_max + 1, size=w.batch).astype(np.int64)


def random_bases(n: int, seed: int) -> np.ndarray:
    """n random nucleotides as byte codes of 'A', 'C', 'G', 'T' (uint8)."""
    rng = np.random.default_rng(seed)
    return np.frombuffer(b"ACGT", dtype=np.uint8)[rng.integers(0, 4, size=n)]


def randn(shape: Sequence[int], dtype: str, seed: int, device="cpu"):
    """i.i.d. N(0, 1) tensor from torch's generator on `device`, cast to dtype.

    bf16 values are the round-to-nearest-even images of fp32 draws.  The CPU
    and GPU generators produce different streams for one seed; a test uses one
    device and hands the very same values to both sides.
    """
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    t = torch.randn(tuple(shape), generator=g, dtype=torch.float32, device=device)
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    elif dtype != "f32":
        raise ValueError(f"unknown dtype {dtype}")
    return t


def qkv(n_rows: int, w: Workload, device="cpu", seed_offset: int = 0):
    """Q [n_rows, H, D], K and V [n_rows, H_kv, D] for workload w.

    n_rows is the number of augmented tokens, which the caller derives from its
    own layout.
    """
    q = randn((n_rows, w.heads, w.head_dim), w.dtype, seed_for(w.index, "q") + seed_offset, device)
    k = randn((n_rows, w.kv_heads, w.head_dim), w.dtype, seed_for(w.index, "k") + seed_offset, device)
    v = randn((n_rows, w.kv_heads, w.head_dim), w.dtype, seed_for(w.index, "v") + seed_offset, device)
    return q, k, v


# Next-base distributions for the fidelity metrics: the base model's logits are
# N(0, scale^2) and the FOCUS model's are the same logits plus an independent
# N(0, noise^2) perturbation (a compressed model close to its base).  Two
# shapes: the four nucleotides, and a byte-level vocabulary of 512 entries.
FIDELITY = {
    # name: (positions, vocab, dtype)
    "fidelity_1mb_acgt": (1_000_000, 4, "f32"),
    "fidelity_1mb_vocab512": (1_000_000, 512, "bf16"),
}


def fidelity_logits(n_pos: int, vocab: int, dtype: str, seed: int, device="cpu",
                    scale: float = 2.0, noise: float = 0.5):
    """(p_logits, q_logits) [n_pos, vocab] as described above FIDELITY."""
    base = randn((n_pos, vocab), "f32", seed, device) * scale
    q = base + randn((n_pos, vocab), "f32", seed + 1, device) * noise
    import torch
    if dtype == "bf16":
        return base.to(torch.bfloat16), q.to(torch.bfloat16)
    return base, q
