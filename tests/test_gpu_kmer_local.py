"""GPU parity of focus_window_attn under FOCUS_MASK_KMER_LOCAL (the Section 3.2
visibility rule) against the float64 oracle.

Small cases compare every output row (several query tiles, ragged tails, GQA,
head_dim 64 and 128, k = 0 windows, k = 1, partial k-mers, windows with more
than 64 summaries, a summary list that exactly fills one 32-row tile, query
tiles of exactly four window tiles); the 1 Mb and ragged workloads at full size run one
masked-parallel launch and compare sampled windows and heads.  Properties on
the device output: every softmax row sums to one over the k-mer-local visible
set through the returned LSE, streaming equals masked-parallel bit for bit, and
a per-window k array and a uniform k give the same result.
"""

import numpy as np
import pytest
import torch

import focus_workloads as fw
import paper_2511_14694_amd as F
from gpu_util import DEV, announce, assert_parity, gather_rows, to64
from oracle import attention as A
from oracle.layout import build_layout
from test_gpu_attention import Prefill, _kmer_for, _sample_windows

pytestmark = pytest.mark.gpu

KL = F.FOCUS_MASK_KMER_LOCAL


def oracle_window_kl(ref, p: Prefill, w, heads):
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
    return A.window_attention_masked(q, kw, vw, ck, cv, A.kmer_local_window_visibility(ref, w), scale)


def compare_windows_kl(ref, p: Prefill, o, lse, windows, heads, what):
    worst = (0.0, 0.0)
    for w in windows:
        t0, T = int(ref["win_tok_off"][w]), int(ref["win_ntok"][w])
        o_ref, lse_ref = oracle_window_kl(ref, p, w, heads)
        got = to64(o[t0:t0 + T][:, heads])
        lg = lse[t0:t0 + T][:, heads].cpu().numpy().astype(np.float64)
        worst = max(worst, assert_parity(got, o_ref, p.dtype, f"{what} window {w}", lg, lse_ref))
    return worst


SMALL_KL = [
    # seq lengths, W, kmer (None: per-window draw), H, Hkv, D
    ([2500], 1000, 100, 4, 4, 128),
    ([1000, 0, 2345], 700, None, 4, 2, 128),
    ([3000], 257, 7, 2, 1, 128),        # ~33 summaries per window
    ([777, 1500], 1000, 0, 2, 2, 64),   # no summaries: causal windows + boundary
    ([4096], 1024, 100, 8, 2, 64),      # partial last k-mer of every window
    ([1], 1000, 100, 4, 4, 128),
    ([130, 129, 64], 1000, 1, 2, 2, 128),   # k = 1: 2-token k-mers, > 64 summaries
    ([2600], 1300, 9, 2, 2, 128),       # 130 summaries per window: three list tiles
    ([2000], 1000, 127, 2, 2, 128),     # k-mers of 128 rows: four window tiles per query tile
    ([1000, 1000], 1000, 33, 2, 1, 128),  # 31 summaries: the boundary and list fill one tile
]


@pytest.mark.parametrize("case", range(len(SMALL_KL)))
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_kmer_local_small_all_rows(case, dtype):
    seq, W, kmer, H, Hkv, D = SMALL_KL[case]
    km = _kmer_for(seq, W, kmer, case)
    announce(f"kmer-local small case={case} dtype={dtype} seq={seq} W={W} H={H}/{Hkv} D={D}")
    p = Prefill(seq, W, km, H, Hkv, D, dtype, seed=2000 + case, run=False)
    o, lse = p.attn(mask=KL)
    ref = build_layout(seq, W, km)
    compare_windows_kl(ref, p, o, lse, range(ref["n_windows"]), list(range(H)), f"kl case {case} {dtype}")


def test_kmer_local_uniform_k_equals_per_window_array():
    announce("kmer-local uniform k vs per-window array")
    seq, W = [3000, 700], 500
    km = np.full(sum(-(-L // W) for L in seq), 50, np.int32)
    p = Prefill(seq, W, km, 4, 2, 128, "bf16", seed=31, run=False)
    o1, l1 = p.attn(mask=KL)
    lay_u = F.focus_layout(p.totals, seq, W, None, 50)
    o2, l2 = F.focus_window_attn(lay_u, p.q, p.k, p.v, p.ck, p.cv, mask=KL, err=p.err)
    torch.cuda.synchronize()
    assert int(p.err.item()) == 0
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_kmer_local_lse_rows_sum_to_one():
    announce("kmer-local lse row sums")
    seq, W = [2000], 1000
    km = np.full(2, 100, np.int32)
    p = Prefill(seq, W, km, 2, 2, 128, "bf16", seed=22, run=False)
    _, lse_all = p.attn(mask=KL)
    ref = build_layout(seq, W, km)
    w = 1
    t0, T = int(ref["win_tok_off"][w]), int(ref["win_ntok"][w])
    idx = A.cache_token_indices(ref, w)
    keys = np.concatenate([gather_rows(p.k, idx), to64(p.k[t0:t0 + T])], axis=0)
    q = to64(p.q[t0:t0 + T])
    lse = lse_all[t0:t0 + T].cpu().numpy().astype(np.float64)
    vis = A.kmer_local_window_visibility(ref, w)
    for h in range(2):
        s = (q[:, h] @ keys[:, h].T) / np.sqrt(128)
        tot = np.where(vis, np.exp(s - lse[:, h:h + 1]), 0.0).sum(axis=1)
        assert np.abs(tot - 1).max() < 2e-4


def test_kmer_local_streaming_equals_masked_parallel_bitwise():
    announce("kmer-local streaming vs masked-parallel")
    seq, W = [3000, 1200], 500
    km = _kmer_for(seq, W, None, 3)
    p = Prefill(seq, W, km, 4, 2, 128, "bf16", seed=6, run=False)
    o_all, lse_all = p.attn(mask=KL)
    ref = build_layout(seq, W, km)
    ck, cv = torch.zeros_like(p.ck), torch.zeros_like(p.cv)
    o = torch.full_like(o_all, float("nan"))
    lse = torch.full_like(lse_all, float("nan"))
    for w in range(ref["n_windows"]):
        t0, T = int(ref["win_tok_off"][w]), int(ref["win_ntok"][w])
        ids = torch.tensor([w], dtype=torch.int32, device=DEV)
        sl = slice(t0, t0 + T)
        ow, lw = F.focus_window_attn(p.lay, p.q[sl].contiguous(), p.k[sl].contiguous(), p.v[sl].contiguous(),
                                     ck, cv, win_ids=ids, qkv_tok_base=t0, mask=KL, err=p.err)
        o[sl], lse[sl] = ow, lw
        F.focus_compact_kv(p.lay, p.k[sl].contiguous(), p.v[sl].contiguous(), ck, cv, win_ids=ids,
                           kv_tok_base=t0, err=p.err)
    torch.cuda.synchronize()
    assert int(p.err.item()) == 0
    assert torch.equal(o, o_all) and torch.equal(lse, lse_all)


@pytest.mark.parametrize("name", ["prefill_1mb", "ragged_b8_256kb"])
def test_kmer_local_workload_full_size_sampled(name):
    """Every window in one launch at full size; sampled windows and heads."""
    w = fw.WORKLOADS[name]
    announce(f"kmer-local workload {name}")
    seq = [w.seq_nt] * w.batch
    km = fw.kmer_draw(w)
    p = Prefill(seq, w.window_nt, km, w.heads, w.kv_heads, w.head_dim, w.dtype,
                seed=fw.seed_for(w.index, "q"), run=False)
    o, lse = p.attn(mask=KL)
    ref = build_layout(seq, w.window_nt, km)
    worst = compare_windows_kl(ref, p, o, lse, _sample_windows(ref, w.index + 7), [0, 13, w.heads - 1], name)
    print(f"[parity] kmer-local {name}: worst max-abs {worst[0]:.3e} rel-L2 {worst[1]:.3e}", flush=True)
    del p, o, lse
    torch.cuda.empty_cache()
