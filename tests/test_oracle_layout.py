"""Pins for the layout oracle: facts fixed by the paper, not by the oracle itself.

* hand-worked examples (tests/golden/layout_worked_examples.txt), derived from
  Appendix A's window and B_w definitions and Section 3.2's insertion rule;
* closed forms of Appendix A: ceil(L/W) windows, |I_w| bases, B_w = ceil(|I_w|/k);
* Section 3.2: M = ceil(L/k) summaries in total when k divides W;
* eq. kv-budget / eq. kv-ratio: retained rows <= sum_w ceil(W/k) + W, and
  gamma = 1/k exactly at 1 Mb with W = 1000, k = 100;
* literal string insertion built independently with Python slicing;
* the workload sizes the benchmark configurations state (cache of 40, 1 000
  and 10 000 rows).
"""

import math
import os

import numpy as np
import pytest

from oracle.layout import BASE, SUMMARY, build_layout, token_string
import focus_workloads as fw

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "layout_worked_examples.txt")


def _golden_cases():
    cases = []
    for line in open(GOLDEN):
        if not line.strip() or line.startswith("#"):
            continue
        # the stream itself contains '|' (window boundaries): split on the
        # first and on the last bar only
        head, rest = line.split("|", 1)
        stream, offs = rest.rsplit("|", 1)
        head, stream, offs = head.strip(), stream.strip(), offs.strip()
        L, W, k = (int(x) for x in head.split())
        cases.append((L, W, k, stream, [int(x) for x in offs.split()]))
    return cases


@pytest.mark.parametrize("L,W,k,stream,offs", _golden_cases())
def test_worked_examples(L, W, k, stream, offs):
    lay = build_layout([L], W, k)
    assert token_string(lay, 0) == stream
    assert lay["win_cache_off"].tolist() == offs


def _random_case(rng):
    B = int(rng.integers(1, 4))
    seq = [int(x) for x in rng.integers(0, 60, B)]
    W = int(rng.integers(1, 20))
    nw = sum(-(-L // W) for L in seq)
    kmer = rng.integers(0, 9, nw).astype(np.int32)
    return seq, W, kmer


@pytest.mark.parametrize("seed", range(40))
def test_appendix_a_closed_forms(seed):
    """Window count, window sizes and B_w follow Appendix A's formulas."""
    rng = np.random.default_rng(seed)
    seq, W, kmer = _random_case(rng)
    lay = build_layout(seq, W, kmer)
    gw = 0
    for b, L in enumerate(seq):
        n_win = math.ceil(L / W) if L else 0
        assert lay["cu_windows"][b + 1] - lay["cu_windows"][b] == n_win
        cache = 0
        for w in range(n_win):
            size = len(range(w * W + 1, min((w + 1) * W, L) + 1))     # |I_w|
            k = int(kmer[gw])
            B_w = math.ceil(size / k) if k else 0
            assert lay["win_nt"][gw] == size
            assert lay["win_nsum"][gw] == B_w
            assert lay["win_ntok"][gw] == size + B_w
            assert lay["win_cache_off"][gw] == cache
            assert lay["win_seq"][gw] == b
            cache += B_w
            gw += 1
        # cache length of the sequence equals its summed summary count
        assert lay["cu_summaries"][b + 1] - lay["cu_summaries"][b] == cache
    assert lay["n_windows"] == gw
    assert lay["n_tokens"] == sum(seq) + lay["n_summaries"]


@pytest.mark.parametrize("L,W,k", [(4000, 1000, 100), (100_000, 1000, 100), (997, 100, 10),
                                   (12, 4, 2), (1, 3, 3), (30, 6, 3)])
def test_total_summaries_is_ceil_L_over_k(L, W, k):
    """Section 3.2: M = ceil(L/k) summary tokens when k divides W."""
    assert W % k == 0
    lay = build_layout([L], W, k)
    assert lay["n_summaries"] == math.ceil(L / k)


@pytest.mark.parametrize("seed", range(10))
def test_literal_string_insertion(seed):
    """Token ids equal the stream built by cutting each window's text into
    k-base pieces and appending the summary symbol to each piece."""
    rng = np.random.default_rng(100 + seed)
    seq, W, kmer = _random_case(rng)
    bases = fw.random_bases(sum(seq), seed)
    SID = 999
    lay = build_layout(seq, W, kmer, bases=bases, summary_token_id=SID)
    expect = []
    off = 0
    gw = 0
    for L in seq:
        text = bases[off:off + L].tolist()
        for w0 in range(0, L, W):
            chunk = text[w0:w0 + W]
            k = int(kmer[gw])
            gw += 1
            if k == 0:
                expect += chunk
                continue
            for p in range(0, len(chunk), k):
                expect += chunk[p:p + k] + [SID]
        off += L
    assert lay["token_ids"].tolist() == expect
    # dropping the summaries gives the bases back in order
    assert (lay["tok_base"][lay["tok_kind"] == BASE] == np.arange(sum(seq))).all()
    assert (lay["tok_base"][lay["tok_kind"] == SUMMARY] == -1).all()


@pytest.mark.parametrize("seed", range(20))
def test_kmer_membership_and_positions(seed):
    """Each summary closes a run of 1..k bases of its own window that carry its
    cache row; positions count up inside each sequence; window ids match."""
    rng = np.random.default_rng(200 + seed)
    seq, W, kmer = _random_case(rng)
    lay = build_layout(seq, W, kmer)
    for b in range(len(seq)):
        t0, t1 = lay["cu_tokens"][b], lay["cu_tokens"][b + 1]
        assert (lay["tok_pos"][t0:t1] == np.arange(t1 - t0)).all()
        s0 = lay["cu_summaries"][b]
        for row, t in enumerate(lay["sum_tok"][s0:lay["cu_summaries"][b + 1]]):
            assert lay["tok_kind"][t] == SUMMARY and lay["tok_kmer"][t] == row
            w = lay["tok_win"][t]
            k = lay["window_kmer"][w]
            u = t - 1
            run = 0
            while u >= lay["win_tok_off"][w] and lay["tok_kind"][u] == BASE:
                assert lay["tok_kmer"][u] == row
                run += 1
                u -= 1
            assert 1 <= run <= k
    for w in range(lay["n_windows"]):
        t0 = lay["win_tok_off"][w]
        assert (lay["tok_win"][t0:t0 + lay["win_ntok"][w]] == w).all()
        if lay["window_kmer"][w] == 0:
            assert (lay["tok_kmer"][t0:t0 + lay["win_ntok"][w]] == -1).all()
        else:   # a window with summaries always ends on one (right boundary)
            assert lay["tok_kind"][t0 + lay["win_ntok"][w] - 1] == SUMMARY


@pytest.mark.parametrize("L,W,k", [(1_000_000, 1000, 100), (256_000, 1000, 50), (1024 * 7 + 5, 1024, 100)])
def test_kv_budget_and_ratio(L, W, k):
    """eq. kv-budget: R_kept <= sum_w ceil(W/k) + W; eq. kv-ratio: gamma ~ 1/k."""
    lay = build_layout([L], W, k)
    kept = lay["n_summaries"]
    M = math.ceil(L / W)
    assert kept <= M * math.ceil(W / k) + W
    assert abs(kept / L - 1 / k) <= 1 / k * 0.05 + W / L
    if L % W == 0 and W % k == 0:
        assert kept * k == L        # gamma = 1/k exactly


@pytest.mark.parametrize("name,windows,tokens,cache", [
    ("tiny_4kb_f32", 4, 4_040, 40),
    ("prefill_100kb", 100, 101_000, 1_000),
    ("prefill_1mb", 1000, 1_010_000, 10_000),
    ("dense_32kb", 1, 32_000, 0),
])
def test_workload_sizes(name, windows, tokens, cache):
    """Sizes stated by the workloads: 4 windows with a 40-row cache, 100 and
    1 000 windows with 1 000 and 10 000 cache rows; the dense point has none."""
    w = fw.WORKLOADS[name]
    lay = build_layout([w.seq_nt] * w.batch, w.window_nt, fw.kmer_draw(w))
    assert lay["n_windows"] == windows
    assert lay["n_tokens"] == tokens
    assert lay["n_summaries"] == cache


def test_ragged_workload_counts():
    """Batch 8 x 256 kb with per-window cadence in {50, 100, 200, 500}: each
    window holds 1000/k_w summaries (2..20) and the caches are ragged."""
    w = fw.WORKLOADS["ragged_b8_256kb"]
    kmer = fw.kmer_draw(w)
    lay = build_layout([w.seq_nt] * w.batch, w.window_nt, kmer)
    assert lay["n_windows"] == 8 * 256
    assert (lay["win_nsum"] == 1000 // kmer).all()
    assert set(np.unique(lay["win_nsum"]).tolist()) <= {2, 5, 10, 20}
    per_seq = np.diff(lay["cu_summaries"])
    assert len(set(per_seq.tolist())) > 1
    assert per_seq.sum() == lay["n_summaries"] == int((1000 // kmer).sum())


# ---- target map pi(t) (Appendix A.1, eq. loss) ----

def _next_base_cases():
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "next_base_worked_examples.txt")
    cases = []
    for line in open(path):
        if line.startswith("#") or not line.strip():
            continue
        head, stream, pi = (x.strip() for x in line.split("|"))
        lens, W, k = head.split()
        cases.append(([int(x) for x in lens.split(",")], int(W), int(k), stream, [int(x) for x in pi.split()]))
    return cases


@pytest.mark.parametrize("seq,W,k,stream,pi", _next_base_cases())
def test_next_base_worked_examples(seq, W, k, stream, pi):
    lay = build_layout(seq, W, k)
    toks = stream.replace("/", " ").replace(";", " ").split()
    assert len(toks) == lay["n_tokens"]
    for t, s in enumerate(toks):
        assert (lay["tok_kind"][t] == SUMMARY) == (s == "S")
        if s != "S":
            assert lay["tok_base"][t] == int(s[1:])
    assert lay["tok_next_base"].tolist() == pi


@pytest.mark.parametrize("seed", range(6))
def test_next_base_brute_force(seed):
    """pi(t) = min{u > t : u a real base} by literal search over the stream,
    on random batches with per-window cadences (k = 0 windows included)."""
    rng = np.random.default_rng(100 + seed)
    seq = [int(x) for x in rng.integers(0, 40, 3)]
    W = int(rng.integers(1, 12))
    nw = sum(-(-L // W) for L in seq)
    km = rng.integers(0, 6, nw).astype(np.int32)
    lay = build_layout(seq, W, km)
    kind, base, cu = lay["tok_kind"], lay["tok_base"], lay["cu_tokens"]
    for b in range(len(seq)):
        for t in range(cu[b], cu[b + 1]):
            later = [u for u in range(t + 1, cu[b + 1]) if kind[u] == BASE]
            want = base[min(later)] if later else -1
            assert lay["tok_next_base"][t] == want
    # a real base's target is the next base of its sequence
    for t in np.nonzero(kind == BASE)[0]:
        b = int(np.searchsorted(cu, t, side="right") - 1)
        last = sum(seq[:b + 1]) - 1
        assert lay["tok_next_base"][t] == (base[t] + 1 if base[t] < last else -1)
