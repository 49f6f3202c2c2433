"""The benchmark's algorithmic pair counts (the FLOP numerators of its
roofline figures) equal the number of visible (query, key) pairs of the
oracle's visibility matrices, window by window."""

import numpy as np
import pytest

import bench
from oracle import attention as A
from oracle.layout import build_layout


@pytest.mark.parametrize("seed", range(6))
def test_pair_counts_match_oracle_visibility(seed):
    rng = np.random.default_rng(seed)
    seq = [int(x) for x in rng.integers(1, 300, int(rng.integers(1, 4)))]
    W = int(rng.integers(5, 120))
    nw = sum(-(-L // W) for L in seq)
    kmer = rng.choice([0, 1, 3, 7, 50, 200], nw).astype(np.int32)
    lay = build_layout(seq, W, kmer)
    ct = sum(int(A.window_visibility(int(T), int(C)).sum())
             for T, C in zip(lay["win_ntok"], lay["win_cache_off"]))
    kl = sum(int(A.kmer_local_window_visibility(lay, w).sum()) for w in range(lay["n_windows"]))
    assert bench.visible_pairs(lay["win_ntok"], lay["win_cache_off"]) == ct
    assert bench.kmer_local_pairs(lay["win_ntok"], lay["win_cache_off"], kmer) == kl


def test_one_mb_counts():
    lay = build_layout([1_000_000], 1000, 100)
    assert bench.visible_pairs(lay["win_ntok"], lay["win_cache_off"]) == 5_555_505_000
    # per window of 1 010 tokens: ten 101-token k-mers, plus the boundary after the first
    per_win = 10 * (101 * 102 // 2) + 101 * (10 * 9 // 2)
    assert bench.kmer_local_pairs(lay["win_ntok"], lay["win_cache_off"], 100) == 1000 * per_win + 999 * 1010


def test_traffic_record_keyed_to_code_not_comments(tmp_path, monkeypatch):
    """The counter record's source hash covers the attention's code: a comment
    or whitespace edit keeps it, any code edit changes it."""
    src = tmp_path / "k.hip"
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    src.write_text("int f(int x) {\n  return x + 1;  // one\n}\n/* block */\n")
    h0 = bench.source_hash(["k.hip"])
    src.write_text("// header\nint f(int x) {\n    return x + 1;  /* other */\n}\n")
    assert bench.source_hash(["k.hip"]) == h0
    src.write_text("int f(int x) {\n  return x + 2;  // one\n}\n")
    assert bench.source_hash(["k.hip"]) != h0
