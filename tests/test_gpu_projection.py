"""GPU parity of focus_qkv_project (Q/K/V projection, rotary positions at the
augmented-stream index, summary K/V written straight to the cache) against
the float64 oracle that stores bf16 as the device does.

Every row of small layouts (ragged k, k = 0 windows, GQA, head_dim 64 / 128);
sampled rows of the 1 Mb layout with an Evo-2-scale projection (d_model 4096,
32 + 2 x 32 heads of 128), including positions near 1 M where the rotation
angle (in revolutions) must keep its fraction to ~2^-32.  Outputs that are not
4-byte aligned are refused.  The fused cache write is checked
bit for bit against focus_compact_kv applied to the projected K / V, and
cache_len against the summary counts.  Window-by-window calls reproduce the
whole-layout call bit for bit.  Tolerance: the bf16 bar (max-abs 2e-2, rel-L2
5e-3) on outputs of unit scale.
"""

import numpy as np
import pytest
import torch

import focus_workloads as fw
import paper_2511_14694_amd as F
from gpu_util import DEV, announce, assert_parity, to64
from oracle import projection as P
from oracle.layout import build_layout
from test_gpu_attention import _kmer_for

pytestmark = pytest.mark.gpu


def _w(d, n, seed):
    return (fw.randn((d, n), "f32", seed, DEV) / np.sqrt(d)).to(torch.bfloat16)


def _setup(seq, W, kmer, H, Hkv, D, d, seed):
    km = _kmer_for(seq, W, kmer, seed)
    tot = F.focus_layout_plan(seq, W, km)
    lay = F.focus_layout(tot, seq, W, km)
    hid = fw.randn((tot.n_tokens, d), "bf16", seed, DEV)
    w = _w(d, (H + 2 * Hkv) * D, seed + 1)
    return km, tot, lay, hid, w


@pytest.mark.parametrize("seq,W,kmer,H,Hkv,D,d", [
    ([2500], 1000, 100, 2, 2, 128, 256),
    ([1300, 0, 700], 500, None, 4, 2, 64, 192),
    ([777, 1500], 1000, 0, 2, 2, 64, 128),
])
def test_projection_all_rows_and_fused_cache(seq, W, kmer, H, Hkv, D, d):
    announce(f"qkv project seq={seq} H={H}/{Hkv} D={D} d={d}")
    km, tot, lay, hid, w = _setup(seq, W, kmer, H, Hkv, D, d, 41)
    cap = max(tot.max_cache_per_seq, 1)
    ck = torch.zeros(len(seq), cap, Hkv, D, dtype=torch.bfloat16, device=DEV)
    cv = torch.zeros_like(ck)
    clen = torch.zeros(len(seq), dtype=torch.int32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    q, k, v = F.focus_qkv_project(lay, hid, w, H, Hkv, 10000.0, cache_k=ck, cache_v=cv, cache_len=clen, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    ref = build_layout(seq, W, km)
    rq, rk, rv = P.qkv_project(ref, to64(hid), to64(w), H, Hkv, 10000.0, store_bf16=True)
    assert_parity(to64(q), rq, "bf16", "q")
    assert_parity(to64(k), rk, "bf16", "k")
    assert_parity(to64(v), rv, "bf16", "v")
    # the fused cache write equals compacting the projected K / V afterwards
    ck2, cv2 = torch.zeros_like(ck), torch.zeros_like(cv)
    F.focus_compact_kv(lay, k, v, ck2, cv2)
    torch.cuda.synchronize()
    assert torch.equal(ck, ck2) and torch.equal(cv, cv2)
    assert clen.cpu().numpy().tolist() == np.diff(ref["cu_summaries"]).tolist()


def test_window_by_window_equals_whole_layout():
    announce("qkv project streaming")
    seq, W, H, Hkv, D, d = [3000, 1200], 500, 2, 1, 128, 256
    km, tot, lay, hid, w = _setup(seq, W, None, H, Hkv, D, d, 43)
    cap = max(tot.max_cache_per_seq, 1)
    ck = torch.zeros(len(seq), cap, Hkv, D, dtype=torch.bfloat16, device=DEV)
    cv = torch.zeros_like(ck)
    q, k, v = F.focus_qkv_project(lay, hid, w, H, Hkv, 5000.0, cache_k=ck, cache_v=cv)
    ref = build_layout(seq, W, km)
    ck2, cv2 = torch.zeros_like(ck), torch.zeros_like(cv)
    q2, k2, v2 = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    for x in range(ref["n_windows"]):
        t0, T = int(ref["win_tok_off"][x]), int(ref["win_ntok"][x])
        sl = slice(t0, t0 + T)
        a, b_, c = F.focus_qkv_project(lay, hid[sl].contiguous(), w, H, Hkv, 5000.0, tok_base=t0,
                                       cache_k=ck2, cache_v=cv2)
        q2[sl], k2[sl], v2[sl] = a, b_, c
    torch.cuda.synchronize()
    assert torch.equal(q, q2) and torch.equal(k, k2) and torch.equal(v, v2)
    assert torch.equal(ck, ck2) and torch.equal(cv, cv2)


def test_evo2_scale_projection_1mb_sampled():
    w_ = fw.WORKLOADS["prefill_1mb"]
    H, Hkv, D, d = w_.heads, w_.kv_heads, w_.head_dim, 4096
    announce("qkv project 1 Mb, d_model 4096")
    seq = [w_.seq_nt]
    km = fw.kmer_draw(w_)
    tot = F.focus_layout_plan(seq, w_.window_nt, km)
    lay = F.focus_layout(tot, seq, w_.window_nt, km)
    hid = fw.randn((tot.n_tokens, d), "bf16", 44, DEV)
    w = _w(d, (H + 2 * Hkv) * D, 45)
    q, k, v = F.focus_qkv_project(lay, hid, w, H, Hkv, 10000.0)
    torch.cuda.synchronize()
    ref = build_layout(seq, w_.window_nt, km)
    n = tot.n_tokens
    rows = np.unique(np.concatenate([[0, 1, 100, 101, n - 1], np.arange(n - 40, n - 1),
                                     np.random.default_rng(3).integers(0, n, 40)]))
    fetch = lambda r: to64(hid[torch.as_tensor(np.asarray(r, np.int64), device=DEV)])   # noqa: E731
    rq, rk, rv = P.qkv_project(ref, fetch, to64(w), H, Hkv, 10000.0, store_bf16=True, rows=rows)
    idx = torch.as_tensor(rows, device=DEV)
    assert_parity(to64(q[idx]), rq, "bf16", "q 1 Mb")
    assert_parity(to64(k[idx]), rk, "bf16", "k 1 Mb")
    assert_parity(to64(v[idx]), rv, "bf16", "v 1 Mb")
    del q, k, v, hid
    torch.cuda.empty_cache()


def test_projection_rejects_misaligned_outputs():
    """Pairs of bf16 columns are stored as 4-byte words: q, k, v and the
    caches must be 4-byte aligned."""
    announce("projection misaligned q")
    seq, W, kmer, H, Hkv, D, d = [1000], 500, 100, 2, 2, 64, 128
    km, tot, lay, hid, w = _setup(seq, W, kmer, H, Hkv, D, d, 11)
    rows = tot.n_tokens
    buf = torch.empty(rows * H * D + 1, dtype=torch.bfloat16, device=DEV)
    q_bad = buf[1:].view(rows, H, D)                # 2-byte offset
    with pytest.raises(F.FocusError):
        F.focus_qkv_project(lay, hid, w, H, Hkv, q=q_bad)
    q_ok, _, _ = F.focus_qkv_project(lay, hid, w, H, Hkv)
    torch.cuda.synchronize()
    assert torch.isfinite(q_ok.float()).all()
