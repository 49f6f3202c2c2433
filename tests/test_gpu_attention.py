"""GPU parity of focus_window_attn against the float64 oracle.

Small cases compare every output row (several 128-row query tiles and 64-key
tiles, ragged tails, GQA, head_dim 64 and 128, k = 0 windows, empty
sequences, cache lengths on and around the key-tile edges); the workloads at full size run the very launch the benchmark times
(every window of every sequence in one masked-parallel launch) and compare
sampled windows and heads; the dense 32 kb point compares sampled rows.
Properties checked on the device output: streaming (one window per call, the
cache filled as it goes) equals masked-parallel bit for bit when neither splits
keys, two runs are bitwise equal, every softmax row sums to one through the
returned LSE.  Launches with few (window, head, query tile) items split each
item's keys over several workgroups (merged by log-sum-exp): those are checked
against the oracle directly, including splits left without a key tile.
"""

import numpy as np
import pytest
import torch

import focus_workloads as fw
import paper_2511_14694_amd as F
from gpu_util import DEV, announce, assert_parity, gather_rows, to64, torch_dtype
from oracle import attention as A
from oracle.layout import build_layout

pytestmark = pytest.mark.gpu


def _randn(shape, dtype, seed):
    return fw.randn(shape, dtype, seed, device=DEV)


class Prefill:
    """Layout + bulk compaction + masked-parallel attention on the device."""

    def __init__(self, seq, W, kmer, H, Hkv, D, dtype, seed, scale=0.0, run=True):
        self.seq, self.W, self.kmer = seq, W, kmer
        self.H, self.Hkv, self.D, self.dtype = H, Hkv, D, dtype
        self.scale = scale
        self.totals = F.focus_layout_plan(seq, W, kmer)
        self.lay = F.focus_layout(self.totals, seq, W, kmer)
        n = self.totals.n_tokens
        self.q = _randn((n, H, D), dtype, seed)
        self.k = _randn((n, Hkv, D), dtype, seed + 1)
        self.v = _randn((n, Hkv, D), dtype, seed + 2)
        B = len(seq)
        self.cap = max(self.totals.max_cache_per_seq, 1)
        self.ck = torch.zeros(B, self.cap, Hkv, D, dtype=torch_dtype(dtype), device=DEV)
        self.cv = torch.zeros_like(self.ck)
        self.clen = torch.zeros(B, dtype=torch.int32, device=DEV)
        self.err = torch.zeros(1, dtype=torch.int32, device=DEV)
        F.focus_compact_kv(self.lay, self.k, self.v, self.ck, self.cv, self.clen, err=self.err)
        if run:
            self.o, self.lse = self.attn()

    def attn(self, **kw):
        o, lse = F.focus_window_attn(self.lay, self.q, self.k, self.v, self.ck, self.cv,
                                     softmax_scale=self.scale, err=self.err, **kw)
        torch.cuda.synchronize()
        assert int(self.err.item()) == 0
        return o, lse


def oracle_window(ref, p: Prefill, w, heads):
    """Oracle outputs of window w for the given query heads (fetching only the
    input rows the window reads)."""
    t0, T = int(ref["win_tok_off"][w]), int(ref["win_ntok"][w])
    grp = p.H // p.Hkv
    kvh = [h // grp for h in heads]
    idx = A.cache_token_indices(ref, w)
    q = to64(p.q[t0:t0 + T][:, heads])
    kw = to64(p.k[t0:t0 + T][:, kvh])
    vw = to64(p.v[t0:t0 + T][:, kvh])
    ck = gather_rows(p.k, idx)[:, kvh] if len(idx) else np.zeros((0, len(heads), p.D))
    cv = gather_rows(p.v, idx)[:, kvh] if len(idx) else np.zeros((0, len(heads), p.D))
    scale = p.scale if p.scale > 0 else None
    return A.window_attention(q, kw, vw, ck, cv, scale)


def compare_windows(ref, p: Prefill, windows, heads, what):
    worst = (0.0, 0.0)
    for w in windows:
        t0, T = int(ref["win_tok_off"][w]), int(ref["win_ntok"][w])
        o_ref, lse_ref = oracle_window(ref, p, w, heads)
        got = to64(p.o[t0:t0 + T][:, heads])
        lse = p.lse[t0:t0 + T][:, heads].cpu().numpy().astype(np.float64)
        e = assert_parity(got, o_ref, p.dtype, f"{what} window {w}", lse, lse_ref)
        worst = max(worst, e)
    return worst


SMALL = [
    # seq lengths, W, kmer (None: per-window draw), H, Hkv, D
    ([2500], 1000, 100, 4, 4, 128),
    ([1000, 0, 2345], 700, None, 4, 2, 128),
    ([3000], 257, 7, 2, 1, 128),
    ([777, 1500], 1000, 0, 2, 2, 64),
    ([4096], 1024, 100, 8, 2, 64),
    ([1], 1000, 100, 4, 4, 128),
    ([130, 129, 64], 1000, 1, 2, 2, 128),
]


def _kmer_for(seq, W, kmer, seed):
    nw = sum(-(-L // W) for L in seq)
    if kmer is None:
        return np.random.default_rng(seed).choice([0, 5, 50, 100, 500], nw).astype(np.int32)
    return np.full(nw, kmer, np.int32)


@pytest.mark.parametrize("case", range(len(SMALL)))
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_small_all_rows(case, dtype):
    seq, W, kmer, H, Hkv, D = SMALL[case]
    km = _kmer_for(seq, W, kmer, case)
    announce(f"attn small case={case} dtype={dtype} seq={seq} W={W} H={H}/{Hkv} D={D}")
    p = Prefill(seq, W, km, H, Hkv, D, dtype, seed=1000 + case)
    ref = build_layout(seq, W, km)
    compare_windows(ref, p, range(ref["n_windows"]), list(range(H)), f"case {case} {dtype}")


# Per-window cadences whose cache lengths C_w land on and around the 64-key
# tile edges (0, 1, 32, 33, 63, 64, 65, 124-126): the partial cache tile is the
# first key tile, masked below its first cache row, and every full tile after
# it up to the block's diagonal takes the branch-free path.  One window has no
# summaries (k = 0) and the last is truncated.
EDGE_W = 640
EDGE_KMER = [640, 21, 640, 22, 640, 640, 11, 640, 640, 9, 0, 100]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_cache_lengths_at_tile_edges(dtype):
    seq = [EDGE_W * len(EDGE_KMER) - 37]
    km = np.array(EDGE_KMER, np.int32)
    ref = build_layout(seq, EDGE_W, km)
    assert [int(c) for c in ref["win_cache_off"][:10]] == [0, 1, 32, 33, 63, 64, 65, 124, 125, 126]
    announce(f"attn cache lengths at tile edges dtype={dtype}")
    p = Prefill(seq, EDGE_W, km, 2, 1, 128, dtype, seed=77)
    compare_windows(ref, p, range(ref["n_windows"]), [0, 1], f"tile edges {dtype}")


def test_tiny_workload_f32_full():
    """The tiny 4 kb workload (1 head x 64, float32) against the sequential
    oracle over every token."""
    w = fw.WORKLOADS["tiny_4kb_f32"]
    announce("attn tiny_4kb_f32")
    km = fw.kmer_draw(w)
    p = Prefill([w.seq_nt], w.window_nt, km, w.heads, w.kv_heads, w.head_dim, "f32", seed=fw.seed_for(0, "q"))
    ref = build_layout([w.seq_nt], w.window_nt, km)
    o_ref, lse_ref = A.prefill_sequential(ref, to64(p.q), to64(p.k), to64(p.v))
    assert_parity(to64(p.o), o_ref, "f32", "tiny workload", p.lse.cpu().numpy().astype(np.float64), lse_ref)
    assert p.clen.item() == 40


def test_custom_scale():
    announce("attn custom scale")
    seq, W = [1500], 500
    km = np.full(3, 50, np.int32)
    p = Prefill(seq, W, km, 2, 2, 128, "bf16", seed=77, scale=0.3)
    ref = build_layout(seq, W, km)
    compare_windows(ref, p, range(3), [0, 1], "scale 0.3")


def _no_split():
    return torch.empty(0, dtype=torch.uint8, device=DEV)


def test_streaming_equals_masked_parallel_bitwise():
    """One window per call, in order, compacting each window right after its
    attention and passing only the window's rows, reproduces the single
    masked-parallel launch bit for bit (both without the key split)."""
    announce("attn streaming vs masked-parallel")
    seq, W = [3000, 1200], 500
    km = _kmer_for(seq, W, None, 3)
    p = Prefill(seq, W, km, 4, 2, 128, "bf16", seed=5, run=False)
    p.o, p.lse = p.attn(workspace=_no_split())
    ref = build_layout(seq, W, km)
    ck = torch.zeros_like(p.ck)
    cv = torch.zeros_like(p.cv)
    o = torch.full_like(p.o, float("nan"))
    lse = torch.full_like(p.lse, float("nan"))
    for w in range(ref["n_windows"]):
        t0, T = int(ref["win_tok_off"][w]), int(ref["win_ntok"][w])
        ids = torch.tensor([w], dtype=torch.int32, device=DEV)
        sl = slice(t0, t0 + T)
        ow, lw = F.focus_window_attn(p.lay, p.q[sl].contiguous(), p.k[sl].contiguous(), p.v[sl].contiguous(),
                                     ck, cv, win_ids=ids, qkv_tok_base=t0, err=p.err, workspace=_no_split())
        o[sl], lse[sl] = ow, lw
        F.focus_compact_kv(p.lay, p.k[sl].contiguous(), p.v[sl].contiguous(), ck, cv, win_ids=ids,
                           kv_tok_base=t0, err=p.err)
    torch.cuda.synchronize()
    assert int(p.err.item()) == 0
    assert torch.equal(o, p.o) and torch.equal(lse, p.lse)


@pytest.mark.parametrize("seq,H,Hkv,D,wins", [
    ([300_000], 2, 1, 128, [299, 0]),   # 7 splits; window 0's first tile: 4 key tiles
    ([100_000], 4, 2, 64, [99]),        # 4 splits, head_dim 64
])
def test_key_split_against_oracle(seq, H, Hkv, D, wins):
    """Few items per launch: each item's key tiles are split over several
    workgroups and merged; every row of the listed windows against the
    oracle, and against the unsplit launch to float32 rounding."""
    announce(f"attn key split seq={seq} H={H}/{Hkv} D={D} windows={wins}")
    W = 1000
    km = np.full(-(-seq[0] // W), 100, np.int32)
    p = Prefill(seq, W, km, H, Hkv, D, "bf16", seed=31, run=False)
    ids = torch.tensor(wins, dtype=torch.int32, device=DEV)
    assert F.focus_window_attn_workspace(p.lay, p.q, p.k, p.v, p.ck, p.cv, ids) > 0
    p.o, p.lse = p.attn(win_ids=ids)
    ref = build_layout(seq, W, km)
    compare_windows(ref, p, wins, list(range(H)), "key split")
    o1, lse1 = p.attn(win_ids=ids, workspace=_no_split())
    for w in wins:
        sl = slice(int(ref["win_tok_off"][w]), int(ref["win_tok_off"][w] + ref["win_ntok"][w]))
        assert (p.o[sl].float() - o1[sl].float()).abs().max().item() < 2e-2
        assert (p.lse[sl] - lse1[sl]).abs().max().item() < 1e-4
    o2, lse2 = p.attn(win_ids=ids)
    for w in wins:  # deterministic (rows of unlisted windows are not written)
        sl = slice(int(ref["win_tok_off"][w]), int(ref["win_tok_off"][w] + ref["win_ntok"][w]))
        assert torch.equal(o2[sl], p.o[sl]) and torch.equal(lse2[sl], p.lse[sl])


def test_side_stream_scratch():
    """A key-split launch on a side stream while the current stream keeps
    allocating and writing: the call's scratch belongs to the side stream, so
    the result equals the same launch on the current stream bit for bit."""
    announce("attn key split on a side stream")
    seq, W, H, D = [300_000], 1000, 2, 128
    km = np.full(300, 100, np.int32)
    p = Prefill(seq, W, km, H, 1, D, "bf16", seed=41, run=False)
    ids = torch.tensor([299], dtype=torch.int32, device=DEV)
    n = F.focus_window_attn_workspace(p.lay, p.q, p.k, p.v, p.ck, p.cv, ids)
    assert n > 0
    o_ref, lse_ref = p.attn(win_ids=ids)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    o = torch.zeros_like(o_ref)
    lse = torch.zeros_like(lse_ref)
    F.focus_window_attn(p.lay, p.q, p.k, p.v, p.ck, p.cv, o=o, lse=lse, win_ids=ids, stream=side)
    # the current stream allocates blocks of the scratch's size and scribbles on them
    junk = [torch.full((n,), 0xFF, dtype=torch.uint8, device=DEV) for _ in range(4)]
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    del junk
    ref = build_layout(seq, W, km)
    sl = slice(int(ref["win_tok_off"][299]), int(ref["win_tok_off"][299] + ref["win_ntok"][299]))
    assert torch.equal(o[sl], o_ref[sl]) and torch.equal(lse[sl], lse_ref[sl])


def test_window_subset_any_order_and_determinism():
    announce("attn window subset / determinism")
    seq, W = [5000], 1000
    km = np.full(5, 100, np.int32)
    p = Prefill(seq, W, km, 4, 4, 128, "bf16", seed=9)
    o2, lse2 = p.attn()
    assert torch.equal(o2, p.o) and torch.equal(lse2, p.lse)
    ids = torch.tensor([3, 0, 4], dtype=torch.int32, device=DEV)
    o = torch.full_like(p.o, 5.0)
    lse = torch.full_like(p.lse, 5.0)
    p.attn(win_ids=ids, o=o, lse=lse)
    ref = build_layout(seq, W, km)
    for w in range(5):
        sl = slice(int(ref["win_tok_off"][w]), int(ref["win_tok_off"][w] + ref["win_ntok"][w]))
        if w in (3, 0, 4):
            assert torch.equal(o[sl], p.o[sl]) and torch.equal(lse[sl], p.lse[sl])
        else:
            assert (o[sl].float() == 5.0).all() and (lse[sl] == 5.0).all()


def test_lse_rows_sum_to_one():
    """sum_j exp(s_ij - lse_i) = 1 over each row's visible keys, with s from
    the inputs in float64 and lse from the device."""
    announce("attn lse row sums")
    seq, W = [2000], 1000
    km = np.full(2, 100, np.int32)
    p = Prefill(seq, W, km, 2, 2, 128, "bf16", seed=21)
    ref = build_layout(seq, W, km)
    w = 1
    t0, T = int(ref["win_tok_off"][w]), int(ref["win_ntok"][w])
    idx = A.cache_token_indices(ref, w)
    keys = np.concatenate([gather_rows(p.k, idx), to64(p.k[t0:t0 + T])], axis=0)
    q = to64(p.q[t0:t0 + T])
    lse = p.lse[t0:t0 + T].cpu().numpy().astype(np.float64)
    vis = A.window_visibility(T, len(idx))
    for h in range(2):
        s = (q[:, h] @ keys[:, h].T) / np.sqrt(128)
        tot = np.where(vis, np.exp(s - lse[:, h:h + 1]), 0.0).sum(axis=1)
        assert np.abs(tot - 1).max() < 2e-4


def test_bounds_error_writes_nothing():
    announce("attn bounds error")
    seq, W = [3000], 1000
    km = np.full(3, 100, np.int32)
    p = Prefill(seq, W, km, 2, 2, 64, "bf16", seed=4, run=False)
    ref = build_layout(seq, W, km)
    t0 = int(ref["win_tok_off"][2])
    o = torch.full((t0, 2, 64), 3.0, dtype=torch.bfloat16, device=DEV)
    ids = torch.tensor([2], dtype=torch.int32, device=DEV)
    F.focus_window_attn(p.lay, p.q[:t0].contiguous(), p.k[:t0].contiguous(), p.v[:t0].contiguous(),
                        p.ck, p.cv, o=o, win_ids=ids, err=p.err)
    torch.cuda.synchronize()
    assert int(p.err.item()) & F.FOCUS_ERR_BOUNDS
    assert (o.float() == 3.0).all()


def _sample_windows(ref, seed, n_random=2):
    nw = ref["n_windows"]
    cu = ref["cu_windows"]
    picks = {0, 1, nw // 2, nw - 1}
    for b in (0, len(cu) - 2):
        picks |= {int(cu[b]), int(cu[b + 1]) - 1}
    picks |= set(np.random.default_rng(seed).integers(0, nw, n_random).tolist())
    return sorted(w for w in picks if 0 <= w < nw)


@pytest.mark.parametrize("name", ["prefill_100kb", "prefill_1mb", "ragged_b8_256kb"])
def test_workload_full_size_sampled(name):
    """Full-size masked-parallel launch (the benchmark's), sampled windows and
    heads against the oracle; compaction of the whole cache bit-exact."""
    w = fw.WORKLOADS[name]
    announce(f"attn workload {name}")
    seq = [w.seq_nt] * w.batch
    km = fw.kmer_draw(w)
    p = Prefill(seq, w.window_nt, km, w.heads, w.kv_heads, w.head_dim, w.dtype, seed=fw.seed_for(w.index, "q"))
    ref = build_layout(seq, w.window_nt, km)
    assert p.clen.cpu().numpy().tolist() == np.diff(ref["cu_summaries"]).tolist()
    heads = [0, 13, w.heads - 1]
    worst = compare_windows(ref, p, _sample_windows(ref, w.index), heads, name)
    print(f"[parity] {name}: worst max-abs {worst[0]:.3e} rel-L2 {worst[1]:.3e}", flush=True)
    if name == "prefill_1mb":
        # the streaming launch the benchmark times: one window per call (key split)
        last = ref["n_windows"] - 1
        ids = torch.tensor([last], dtype=torch.int32, device=DEV)
        assert F.focus_window_attn_workspace(p.lay, p.q, p.k, p.v, p.ck, p.cv, ids) > 0
        p.attn(win_ids=ids, o=p.o, lse=p.lse)
        e = compare_windows(ref, p, [last], heads, f"{name} streaming")
        print(f"[parity] {name} streaming: max-abs {e[0]:.3e} rel-L2 {e[1]:.3e}", flush=True)
    del p
    torch.cuda.empty_cache()


def test_dense_32kb_sampled_rows():
    """k = 0, one 32 000-token window: textbook causal attention, rows sampled
    across the whole window (first, last, tile edges, random)."""
    w = fw.WORKLOADS["dense_32kb"]
    announce("attn dense_32kb")
    p = Prefill([w.seq_nt], w.window_nt, fw.kmer_draw(w), w.heads, w.kv_heads, w.head_dim, w.dtype,
                seed=fw.seed_for(w.index, "q"))
    n = w.seq_nt
    rows = sorted({0, 1, 127, 128, 4095, 16000, n - 129, n - 1} |
                  set(np.random.default_rng(5).integers(0, n, 8).tolist()))
    heads = [0, 17, 31]
    last = max(rows) + 1
    keys = to64(p.k[:last][:, heads])
    vals = to64(p.v[:last][:, heads])
    q = to64(p.q[rows][:, heads])
    vis = np.arange(last)[None, :] <= np.asarray(rows)[:, None]
    for i, h in enumerate(heads):
        o_ref, lse_ref, _ = A.attend(q[:, i], keys[:, i], vals[:, i], vis, 1 / np.sqrt(w.head_dim))
        got = to64(p.o[rows][:, h])
        assert_parity(got, o_ref, "bf16", f"dense head {h}",
                      p.lse[rows][:, h].cpu().numpy().astype(np.float64), lse_ref)
    del p
    torch.cuda.empty_cache()
