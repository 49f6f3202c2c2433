"""GPU parity of focus_decode_step against the oracle's streaming state machine
(oracle.decode.DecodeSequence).

The device derives every step's kind itself (DecodeSchedule:
focus_decode_sched_start places each sequence part-way into its window,
focus_decode_next_kind gives the next token's kind); the oracle decides every
token's kind on its own.  Both start from the same random cache/window contents
and the same start position inside the window, and each derives its own
initial lengths.  Cadences are uniform or drawn per window.
"""

import numpy as np
import pytest
import torch

import focus_workloads as fw
import paper_2511_14694_amd as F
from gpu_util import DEV, announce, assert_parity, to64, torch_dtype
from oracle.decode import DecodeSequence

pytestmark = pytest.mark.gpu


class DecodeRun:
    """k: one cadence for every window, or [B, n] cadences of each sequence's
    current window and the ones after it."""

    def __init__(self, B, H, Hkv, D, dtype, W, k, cache_rows0, starts, steps, seed,
                 split=0, cache_slack=None):
        self.B, self.H, self.Hkv, self.D, self.dtype = B, H, Hkv, D, dtype
        self.W, self.k, self.steps = W, k, steps
        self.starts = np.asarray(starts, np.int64)
        self.cache_rows0 = cache_rows0
        # device schedule: place every sequence start[b] tokens into its window
        uniform = np.ndim(k) == 0
        self.sched = F.DecodeSchedule(B, W, None if uniform else np.asarray(k, np.int32),
                                      int(k) if uniform else 0, device=DEV)
        n_sum0 = self.sched.start(self.starts).clone()
        n_base0 = self.sched.bases_in_window.clone()
        kmin = int(k) if uniform else int(np.min(k))
        per_window = -(-W // kmin) if kmin else 0
        slack = cache_slack if cache_slack is not None else per_window * (2 + steps // max(W, 1))
        self.cap_c = cache_rows0 + slack
        self.cap_w = W
        td = torch_dtype(dtype)
        g = seed
        self.cache_k = fw.randn((B, self.cap_c, Hkv, D), dtype, g + 1, DEV)
        self.cache_v = fw.randn((B, self.cap_c, Hkv, D), dtype, g + 2, DEV)
        self.win_k = fw.randn((B, self.cap_w, Hkv, D), dtype, g + 3, DEV)
        self.win_v = fw.randn((B, self.cap_w, Hkv, D), dtype, g + 4, DEV)
        self.sq = fw.randn((steps, B, H, D), dtype, g + 5, DEV)
        self.sk = fw.randn((steps, B, Hkv, D), dtype, g + 6, DEV)
        self.sv = fw.randn((steps, B, Hkv, D), dtype, g + 7, DEV)
        self.init_k = (self.cache_k.clone(), self.win_k.clone())
        self.init_v = (self.cache_v.clone(), self.win_v.clone())
        self.cache_len = (n_sum0 + cache_rows0).to(torch.int32)
        self.win_len = n_base0.clone()
        self.kinds = torch.empty(steps, B, dtype=torch.uint8, device=DEV)     # [steps, B], as derived
        self.o = torch.empty(steps, B, H, D, dtype=td, device=DEV)
        self.lse = torch.empty(steps, B, H, dtype=torch.float32, device=DEV)
        self.len_hist = torch.empty(steps, 2, B, dtype=torch.int32, device=DEV)
        self.err = torch.zeros(1, dtype=torch.int32, device=DEV)
        ws = F.focus_decode_workspace(self.sq[0], self.sk[0], self.cache_k, self.win_k, split)
        self.ws = torch.empty(ws, dtype=torch.uint8, device=DEV)
        for i in range(steps):
            self.kinds[i].copy_(self.sched.next_kind())
            F.focus_decode_step(self.sq[i], self.sk[i], self.sv[i], self.sched.kind, self.cache_k, self.cache_v,
                                self.cache_len, self.win_k, self.win_v, self.win_len, o=self.o[i],
                                lse=self.lse[i], workspace=self.ws, split_keys=split, err=self.err)
            self.len_hist[i, 0].copy_(self.cache_len)
            self.len_hist[i, 1].copy_(self.win_len)
        torch.cuda.synchronize()

    def oracle(self, b, sample_steps):
        """Run the oracle over every step of sequence b; compare at sample_steps."""
        k_b = self.k if np.ndim(self.k) == 0 else [int(x) for x in self.k[b]]
        n_bases, n_sum, open_kmer = DecodeSequence.replay_counters(
            self.W, k_b if np.ndim(k_b) == 0 else k_b[0], int(self.starts[b]))
        c0 = self.cache_rows0 + n_sum
        ck = to64(self.init_k[0][b, :c0]).astype(np.float32)
        cv = to64(self.init_v[0][b, :c0]).astype(np.float32)
        wk = to64(self.init_k[1][b, :n_bases]).astype(np.float32)
        wv = to64(self.init_v[1][b, :n_bases]).astype(np.float32)
        st = DecodeSequence(self.W, k_b, ck, cv, wk, wv, n_bases, open_kmer)
        q = to64(self.sq[:, b])
        k = to64(self.sk[:, b]).astype(np.float32)
        v = to64(self.sv[:, b]).astype(np.float32)
        hist = self.len_hist.cpu().numpy()
        worst = (0.0, 0.0)
        for i in range(self.steps):
            o, lse, kind, end = st.step(q[i], k[i], v[i], compute=i in sample_steps)
            assert kind == (int(self.kinds[i, b]) & F.FOCUS_STEP_SUMMARY)
            assert end == bool(int(self.kinds[i, b]) & F.FOCUS_STEP_WINDOW_END)
            assert hist[i, 0, b] == st.cache_len and hist[i, 1, b] == st.win_len, f"lengths at step {i}"
            if o is not None:
                e = assert_parity(to64(self.o[i, b]), o, self.dtype, f"seq {b} step {i}",
                                  self.lse[i, b].cpu().numpy().astype(np.float64), lse)
                worst = max(worst, e)
        return worst


@pytest.mark.parametrize("dtype,D,Hkv", [("bf16", 128, 4), ("bf16", 64, 2), ("f32", 128, 1), ("f32", 64, 4)])
def test_decode_small_every_step(dtype, D, Hkv):
    announce(f"decode small {dtype} D={D} Hkv={Hkv}")
    r = DecodeRun(B=3, H=4, Hkv=Hkv, D=D, dtype=dtype, W=40, k=6, cache_rows0=37,
                  starts=[1, 17, 45], steps=70, seed=300 + D)
    assert int(r.err.item()) == 0
    for b in range(3):
        r.oracle(b, set(range(70)))


def test_decode_per_window_cadence():
    """Every window draws its own cadence from {50, 100, 200, 500} (the ragged
    schedule): the device schedule switches cadence at each window end, and
    every step matches the oracle, which switches on its own."""
    announce("decode per-window cadence")
    B, W, steps = 4, 1000, 2600
    rng = np.random.default_rng(11)
    km = rng.choice([50, 100, 200, 500], (B, 4)).astype(np.int32)
    starts = rng.integers(1, 900, B)
    r = DecodeRun(B=B, H=4, Hkv=2, D=128, dtype="bf16", W=W, k=km, cache_rows0=40, starts=starts,
                  steps=steps, seed=19)
    assert int(r.err.item()) == 0
    kinds = r.kinds.cpu().numpy()
    assert ((kinds & F.FOCUS_STEP_WINDOW_END) > 0).sum(0).min() >= 2    # every sequence crosses two windows
    for b in range(B):
        ends = np.nonzero(kinds[:, b] & F.FOCUS_STEP_WINDOW_END)[0]
        sample = set(range(0, steps, 97)) | {int(e) for e in ends} | {int(e) + 1 for e in ends}
        r.oracle(b, {i for i in sample if i < steps})


def test_decode_mixed_cadences_every_step():
    """Small windows whose cadences include k = 0 (no summaries: the window
    ends at its W-th base) and k = W (one summary per window); every step
    against the oracle."""
    announce("decode mixed cadences")
    km = np.array([[0, 5, 3, 0, 12, 1], [4, 0, 12, 1, 0, 5]], np.int32)
    r = DecodeRun(B=2, H=4, Hkv=2, D=64, dtype="bf16", W=12, k=km, cache_rows0=9, starts=[3, 0],
                  steps=70, seed=23, cache_slack=70)
    assert int(r.err.item()) == 0
    for b in range(2):
        r.oracle(b, set(range(70)))


def test_decode_split_invariance():
    announce("decode split invariance")
    runs = [DecodeRun(B=2, H=4, Hkv=4, D=128, dtype="bf16", W=100, k=10, cache_rows0=300,
                      starts=[5, 90], steps=30, seed=7, split=s) for s in (16, 64, 0)]
    for r in runs[1:]:
        assert torch.equal(r.len_hist, runs[0].len_hist)
        assert_parity(to64(r.o), to64(runs[0].o), "bf16", "split vs split")
        assert float((r.lse - runs[0].lse).abs().max()) < 1e-5
    rerun = DecodeRun(B=2, H=4, Hkv=4, D=128, dtype="bf16", W=100, k=10, cache_rows0=300,
                      starts=[5, 90], steps=30, seed=7, split=0)
    assert torch.equal(rerun.o, runs[2].o) and torch.equal(rerun.lse, runs[2].lse)


def test_decode_capacity_error():
    """A summary step into a full cache is skipped with FOCUS_ERR_CAPACITY; the
    step still attends over what is there and the length stays put."""
    announce("decode capacity")
    r = DecodeRun(B=1, H=2, Hkv=2, D=64, dtype="bf16", W=10, k=5, cache_rows0=8,
                  starts=[5], steps=1, seed=3, cache_slack=1)
    # start 5: [b b b b b] -> next token is the first summary; cache 8 + 0 -> 9 == cap
    assert r.cap_c == 9 and int(r.cache_len.item()) == 9 and int(r.err.item()) == 0
    o2 = torch.empty_like(r.o[0])
    kinds = torch.tensor([F.FOCUS_STEP_SUMMARY], dtype=torch.uint8, device=DEV)
    F.focus_decode_step(r.sq[0], r.sk[0], r.sv[0], kinds, r.cache_k, r.cache_v, r.cache_len, r.win_k, r.win_v,
                        r.win_len, o=o2, workspace=r.ws, err=r.err)
    torch.cuda.synchronize()
    assert int(r.err.item()) & F.FOCUS_ERR_CAPACITY
    assert int(r.cache_len.item()) == 9
    assert torch.isfinite(o2.float()).all()


def test_decode_workload_full_size():
    """Batch 16 at ~1 Mb: 10 000 cached summaries plus a partial window, 1 000
    steps with summaries and a window rollover; sampled steps of sampled
    sequences against the oracle, lengths after every step for those."""
    w = fw.WORKLOADS["decode_b16_1mb"]
    announce("decode workload decode_b16_1mb")
    starts = fw.decode_positions(w)
    r = DecodeRun(B=w.batch, H=w.heads, Hkv=w.kv_heads, D=w.head_dim, dtype=w.dtype, W=w.window_nt,
                  k=w.kmer, cache_rows0=w.decode_cache_rows, starts=starts, steps=w.decode_steps,
                  seed=fw.seed_for(w.index, "cache_k"))
    assert int(r.err.item()) == 0
    kinds = r.kinds.cpu().numpy()
    for b in (0, int(np.argmax(starts)), w.batch - 1):
        summ = np.nonzero(kinds[:, b] & F.FOCUS_STEP_SUMMARY)[0]
        ends = np.nonzero(kinds[:, b] & F.FOCUS_STEP_WINDOW_END)[0]
        assert len(ends) >= 1 and len(summ) >= 9
        sample = {0, 1, 2, int(summ[0]), int(ends[0]), int(ends[0]) + 1, w.decode_steps - 1}
        worst = r.oracle(b, sample)
        print(f"[parity] decode seq {b}: worst max-abs {worst[0]:.3e} rel-L2 {worst[1]:.3e}", flush=True)
    del r
    torch.cuda.empty_cache()
