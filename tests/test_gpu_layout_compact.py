"""GPU parity of the integer steps: focus_layout and focus_compact_kv are
compared bit for bit with the oracle (oracle.layout, oracle.attention.compact)
on random small batches (ragged lengths, empty sequences, k = 0 windows, a
partial last window and k-mer), the hand-worked examples, and every workload
at its full size.  The optional target map pi(t) (tok_next_base) is part of
every comparison."""

import numpy as np
import pytest
import torch

import focus_workloads as fw
import paper_2511_14694_amd as F
from gpu_util import DEV, announce
from oracle.layout import build_layout

pytestmark = pytest.mark.gpu

FIELDS = ["cu_windows", "cu_tokens", "cu_summaries", "win_seq", "win_nt", "win_nsum", "win_ntok",
          "win_tok_off", "win_cache_off", "win_sum_off", "win_base_off", "tok_pos", "tok_kind",
          "tok_base", "tok_kmer", "tok_win", "sum_tok", "tok_next_base"]
SID = 260   # the reserved summary token id (outside the byte range of bases)


def run_layout(seq, W, kmer, with_bases=True):
    totals = F.focus_layout_plan(seq, W, kmer)
    bases = fw.random_bases(int(sum(seq)), 7) if with_bases else None
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    lay = F.focus_layout(totals, seq, W, kmer, bases=bases, summary_token_id=SID, err=err, next_base=True)
    torch.cuda.synchronize()
    return lay, bases, int(err.item())


def check_layout(seq, W, kmer, with_bases=True):
    lay, bases, err = run_layout(seq, W, kmer, with_bases)
    assert err == 0
    ref = build_layout(seq, W, kmer, bases=bases, summary_token_id=SID)
    got = lay.to_numpy()
    for f in FIELDS + (["token_ids"] if with_bases else []):
        np.testing.assert_array_equal(got[f], ref[f], err_msg=f)
    return lay, ref


def random_case(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 6))
    seq = [int(x) for x in rng.integers(0, 3000, B)]
    if B > 2:
        seq[1] = 0                                   # an empty sequence in the middle
    W = int(rng.choice([1, 7, 100, 257, 1000, 1024]))
    nw = sum(-(-L // W) for L in seq)
    kmer = rng.choice([0, 1, 3, 50, 100, 2000], nw).astype(np.int32)
    return seq, W, kmer


@pytest.mark.parametrize("seed", range(12))
def test_layout_random(seed):
    seq, W, kmer = random_case(seed)
    announce(f"layout random seed={seed} seq={seq} W={W}")
    check_layout(seq, W, kmer)


def test_layout_edge_cases():
    announce("layout edge cases")
    check_layout([], 10, np.zeros(0, np.int32), with_bases=False)          # empty batch
    check_layout([0, 0], 10, np.zeros(0, np.int32), with_bases=False)      # only empty sequences
    check_layout([1], 1, np.array([1], np.int32))                           # one base, one summary
    check_layout([1024], 1024, np.array([100], np.int32))                   # 24-base last k-mer
    check_layout([5000], 1000, np.array([0] * 5, np.int32))                # no summaries
    check_layout([3], 10, np.array([100], np.int32))                        # k larger than window


@pytest.mark.parametrize("name", ["tiny_4kb_f32", "prefill_100kb", "prefill_1mb",
                                  "ragged_b8_256kb", "decode_b16_1mb", "dense_32kb"])
def test_layout_workloads(name):
    w = fw.WORKLOADS[name]
    announce(f"layout workload {name}")
    check_layout([w.seq_nt] * w.batch, w.window_nt, fw.kmer_draw(w), with_bases=False)


def test_layout_plan_mismatch_raises_device_error():
    """Totals planned for one cadence, device given another: the device reports
    FOCUS_ERR_PLAN and writes no token metadata."""
    announce("layout plan mismatch")
    totals = F.focus_layout_plan([5000], 1000, None, 100)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    lay = F.focus_layout(totals, [5000], 1000, np.full(5, 50, np.int32), err=err)
    torch.cuda.synchronize()
    assert int(err.item()) & F.FOCUS_ERR_PLAN
    assert (lay["win_ntok"].cpu().numpy() == 0).all()


# ------------------------------------------------------------------ compaction

def _kv(n, hkv, d, dtype, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    k = torch.randn(n, hkv, d, generator=g, device=DEV).to(dtype)
    v = torch.randn(n, hkv, d, generator=g, device=DEV).to(dtype)
    return k, v


def _expected_cache(ref, k, v, B, cap):
    ek = torch.zeros(B, cap, *k.shape[1:], dtype=k.dtype, device=DEV)
    ev = torch.zeros_like(ek)
    for b in range(B):
        idx = ref["sum_tok"][ref["cu_summaries"][b]:ref["cu_summaries"][b + 1]]
        t = torch.as_tensor(idx, device=DEV)
        ek[b, :len(idx)] = k[t]
        ev[b, :len(idx)] = v[t]
    return ek, ev


@pytest.mark.parametrize("seed,dtype,hkv,d", [(0, torch.bfloat16, 4, 128), (1, torch.float32, 2, 64),
                                              (2, torch.bfloat16, 1, 64), (3, torch.float32, 8, 128)])
def test_compact_bulk_and_listed(seed, dtype, hkv, d):
    seq, W, kmer = random_case(100 + seed)
    announce(f"compact seed={seed} {dtype} hkv={hkv} d={d}")
    lay, ref = check_layout(seq, W, kmer, with_bases=False)
    B = len(seq)
    k, v = _kv(lay.totals.n_tokens, hkv, d, dtype, seed)
    cap = max(lay.totals.max_cache_per_seq, 1) + 3
    ek, ev = _expected_cache(ref, k, v, B, cap)
    # bulk (every window in one launch)
    ck = torch.zeros(B, cap, hkv, d, dtype=dtype, device=DEV)
    cv = torch.zeros_like(ck)
    clen = torch.zeros(B, dtype=torch.int32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    F.focus_compact_kv(lay, k, v, ck, cv, clen, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    assert torch.equal(ck, ek) and torch.equal(cv, ev)
    n_b = np.diff(ref["cu_summaries"])
    assert clen.cpu().numpy().tolist() == n_b.tolist()
    # one window per call, in a shuffled order, with the window's rows only
    ck2, cv2 = torch.zeros_like(ck), torch.zeros_like(cv)
    clen2 = torch.zeros_like(clen)
    order = np.random.default_rng(seed).permutation(lay.totals.n_windows)
    for w in order:
        t0, T = int(ref["win_tok_off"][w]), int(ref["win_ntok"][w])
        ids = torch.tensor([w], dtype=torch.int32, device=DEV)
        F.focus_compact_kv(lay, k[t0:t0 + T].contiguous(), v[t0:t0 + T].contiguous(), ck2, cv2, clen2,
                           win_ids=ids, kv_tok_base=t0, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    assert torch.equal(ck2, ek) and torch.equal(cv2, ev)
    assert clen2.cpu().numpy().tolist() == n_b.tolist()


def test_compact_capacity_and_bounds_are_device_errors():
    """Rows beyond cache_cap and sources outside the k/v buffer are skipped
    with an error bit; nothing beyond the cache is written."""
    announce("compact capacity/bounds")
    seq, W = [3000], 1000
    kmer = np.full(3, 100, np.int32)
    lay, ref = check_layout(seq, W, kmer, with_bases=False)
    k, v = _kv(lay.totals.n_tokens, 2, 64, torch.bfloat16, 5)
    cap = 15                                        # 30 summaries planned
    store_k = torch.full((1, cap + 8, 2, 64), 7.0, dtype=torch.bfloat16, device=DEV)
    store_v = store_k.clone()
    ck, cv = store_k[:, :cap], store_v[:, :cap]     # leading rows: a contiguous view
    assert ck.is_contiguous()
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    ids = torch.arange(3, dtype=torch.int32, device=DEV)
    F.focus_compact_kv(lay, k, v, ck, cv, None, win_ids=ids, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) & F.FOCUS_ERR_CAPACITY
    assert (store_k[0, cap:].float() == 7.0).all() and (store_v[0, cap:].float() == 7.0).all()
    ek, _ = _expected_cache(ref, k, v, 1, 30)
    assert torch.equal(ck[0], ek[0, :cap])
    # a k/v buffer that does not hold window 2's rows
    err.zero_()
    t0 = int(ref["win_tok_off"][2])
    ck3 = torch.zeros(1, 40, 2, 64, dtype=torch.bfloat16, device=DEV)
    F.focus_compact_kv(lay, k[:t0].contiguous(), v[:t0].contiguous(), ck3, ck3.clone(), None,
                       win_ids=ids, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) & F.FOCUS_ERR_BOUNDS
    assert (ck3[0, 20:].float() == 0).all()


@pytest.mark.parametrize("name", ["prefill_1mb", "ragged_b8_256kb"])
def test_compact_workloads_full_size(name):
    """Bulk compaction at the full workload size, in the launch the benchmark
    times, bit-exact against the oracle's retained rows."""
    w = fw.WORKLOADS[name]
    announce(f"compact workload {name}")
    seq = [w.seq_nt] * w.batch
    kmer = fw.kmer_draw(w)
    totals = F.focus_layout_plan(seq, w.window_nt, kmer)
    lay = F.focus_layout(totals, seq, w.window_nt, kmer)
    ref = build_layout(seq, w.window_nt, kmer)
    k, v = _kv(totals.n_tokens, w.kv_heads, w.head_dim, torch.bfloat16, 11)
    cap = totals.max_cache_per_seq
    ck = torch.empty(w.batch, cap, w.kv_heads, w.head_dim, dtype=torch.bfloat16, device=DEV)
    cv = torch.empty_like(ck)
    clen = torch.zeros(w.batch, dtype=torch.int32, device=DEV)
    F.focus_compact_kv(lay, k, v, ck, cv, clen)
    torch.cuda.synchronize()
    n_b = np.diff(ref["cu_summaries"])
    assert clen.cpu().numpy().tolist() == n_b.tolist()
    for b in range(w.batch):
        idx = torch.as_tensor(ref["sum_tok"][ref["cu_summaries"][b]:ref["cu_summaries"][b + 1]], device=DEV)
        assert torch.equal(ck[b, :len(idx)], k[idx]) and torch.equal(cv[b, :len(idx)], v[idx])
    del k, v, ck, cv
    torch.cuda.empty_cache()
