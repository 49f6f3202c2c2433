"""GPU parity of the FOCUS adapter (Appendix A eq. focus-attn) against the
float64 oracle.

focus_adapter_attn: every summary of small ragged cases (k = 0 windows, more
than 32 summaries per window, GQA, head_dim 64 / 128) under both visibility
rules, and sampled windows of the 1 Mb layout.  focus_adapter_layer (the
projections, the adapter's retained K/V, the attention and W_O): every summary
of small layers, and sampled windows of an Evo-2-scale layer (d_model 4096,
32 x 128) at 100 kb, against the oracle layer that stores its intermediates
in bf16 as the device does, and against the plain float64 layer.  Tolerances:
the bf16 bar of the workloads for the attention; for the layer rel-L2 5e-3 and
max-abs 5e-2 of the output's RMS against the bf16-storing oracle, rel-L2 1e-2
and max-abs 6e-2 against the float64 one (derivations at _layer_parity and
_layer_parity_fp64).
"""

import numpy as np
import pytest
import torch

import focus_workloads as fw
import paper_2511_14694_amd as F
from gpu_util import DEV, announce, assert_parity, to64
from oracle import adapter as AD
from oracle.layout import build_layout
from test_gpu_attention import Prefill, _kmer_for, _sample_windows

pytestmark = pytest.mark.gpu

MASKS = {"ct": F.FOCUS_MASK_CT, "kmer_local": F.FOCUS_MASK_KMER_LOCAL}

CASES = [
    # seq lengths, W, kmer (None: per-window draw), H, Hkv, D
    ([2500], 1000, 100, 4, 4, 128),
    ([1000, 0, 2345], 700, None, 4, 2, 128),
    ([3000], 257, 7, 2, 1, 128),        # 33 summaries per window: two query tiles
    ([777, 1500], 1000, 0, 2, 2, 64),   # no summaries at all
    ([4096], 1024, 100, 8, 2, 64),
    ([130, 129, 64], 1000, 1, 2, 2, 128),
    ([20000], 100, 10, 2, 2, 128),      # 200 windows: 25 per workgroup, windows across waves
    ([3000, 1500, 2200], 100, 25, 2, 1, 64),  # 64 windows per workgroup, spanning sequences
    ([600], 1000, 2, 2, 2, 128),        # 300 summaries per window: one workgroup per window
]


def _sum_rows(p: Prefill):
    return p.q[p.lay["sum_tok"]].contiguous()


@pytest.mark.parametrize("mask", list(MASKS))
@pytest.mark.parametrize("case", range(len(CASES)))
def test_adapter_attention_all_summaries(case, mask):
    seq, W, kmer, H, Hkv, D = CASES[case]
    km = _kmer_for(seq, W, kmer, case)
    announce(f"adapter attn case={case} mask={mask}")
    p = Prefill(seq, W, km, H, Hkv, D, "bf16", seed=3000 + case, run=False)
    qs = _sum_rows(p)
    o, lse = F.focus_adapter_attn(p.lay, qs, p.k, p.v, p.ck, p.cv, mask=MASKS[mask], err=p.err)
    torch.cuda.synchronize()
    assert int(p.err.item()) == 0
    ref = build_layout(seq, W, km)
    if ref["n_summaries"] == 0:
        return
    o_ref, lse_ref = AD.adapter_attention(ref, to64(qs), to64(p.k), to64(p.v), mask)
    assert_parity(to64(o), o_ref, "bf16", f"adapter case {case} {mask}", lse.cpu().numpy().astype(np.float64),
                  lse_ref)


@pytest.mark.parametrize("mask", list(MASKS))
def test_adapter_attention_listed_windows(mask):
    """A shuffled subset of the windows of a 200-window sequence and of a
    second sequence (win_ids): only those windows' summaries are written, each
    against its own cache prefix; the other rows keep what was there."""
    seq, W, kmer, H, Hkv, D = [12000, 8000], 100, 10, 2, 2, 128
    km = _kmer_for(seq, W, kmer, 0)
    announce(f"adapter attn listed windows mask={mask}")
    p = Prefill(seq, W, km, H, Hkv, D, "bf16", seed=3100, run=False)
    ref = build_layout(seq, W, km)
    rng = np.random.default_rng(3101)
    wins = rng.permutation(ref["n_windows"])[:77].astype(np.int32)
    qs = _sum_rows(p)
    o = torch.full_like(qs, 7.0)
    lse = torch.full((qs.shape[0], H), 7.0, dtype=torch.float32, device=DEV)
    F.focus_adapter_attn(p.lay, qs, p.k, p.v, p.ck, p.cv, o_sum=o, lse_sum=lse, mask=MASKS[mask],
                         win_ids=torch.as_tensor(wins, device=DEV), err=p.err)
    torch.cuda.synchronize()
    assert int(p.err.item()) == 0
    listed = np.zeros(ref["n_summaries"], dtype=bool)
    for x in wins:
        listed[ref["win_sum_off"][x]:ref["win_sum_off"][x] + ref["win_nsum"][x]] = True
    o_ref, lse_ref = AD.adapter_attention(ref, to64(qs), to64(p.k), to64(p.v), mask, windows=wins)
    got, got_lse = to64(o), lse.cpu().numpy().astype(np.float64)
    assert_parity(got[listed], o_ref[listed], "bf16", f"adapter listed {mask}", got_lse[listed], lse_ref[listed])
    assert np.all(got[~listed] == 7.0) and np.all(got_lse[~listed] == 7.0)


@pytest.mark.parametrize("mask", list(MASKS))
def test_adapter_attention_1mb_sampled(mask):
    w = fw.WORKLOADS["prefill_1mb"]
    announce(f"adapter attn 1mb mask={mask}")
    seq = [w.seq_nt]
    km = fw.kmer_draw(w)
    p = Prefill(seq, w.window_nt, km, w.heads, w.kv_heads, w.head_dim, w.dtype,
                seed=fw.seed_for(w.index, "q"), run=False)
    qs = _sum_rows(p)
    o, lse = F.focus_adapter_attn(p.lay, qs, p.k, p.v, p.ck, p.cv, mask=MASKS[mask], err=p.err)
    torch.cuda.synchronize()
    ref = build_layout(seq, w.window_nt, km)
    wins = _sample_windows(ref, 11)
    heads = [0, 31]
    sums = np.concatenate([np.arange(ref["win_sum_off"][x], ref["win_sum_off"][x] + ref["win_nsum"][x]) for x in wins])
    # the oracle reads only the rows these windows see
    need = np.unique(np.concatenate([np.arange(ref["win_tok_off"][x], ref["win_tok_off"][x] + ref["win_ntok"][x])
                                     for x in wins] + [ref["sum_tok"]]))
    k64 = np.zeros((ref["n_tokens"], w.kv_heads, w.head_dim))
    v64 = np.zeros_like(k64)
    idx = torch.as_tensor(need, device=DEV)
    k64[need], v64[need] = to64(p.k[idx]), to64(p.v[idx])
    q64 = np.zeros((ref["n_summaries"], len(heads), w.head_dim))
    q64[sums] = to64(qs[torch.as_tensor(sums, device=DEV)][:, heads])
    o_ref, lse_ref = AD.adapter_attention(ref, q64, k64[:, heads], v64[:, heads], mask, windows=wins)
    got = to64(o[torch.as_tensor(sums, device=DEV)][:, heads])
    assert_parity(got, o_ref[sums], "bf16", f"adapter 1mb {mask}",
                  lse[torch.as_tensor(sums, device=DEV)][:, heads].cpu().numpy().astype(np.float64), lse_ref[sums])
    del p
    torch.cuda.empty_cache()


def _weights(d, H, Hkv, D, seed):
    s = 1.0 / np.sqrt(d)
    wq = (fw.randn((d, H * D), "f32", seed, DEV) * s).to(torch.bfloat16)
    wk = (fw.randn((d, Hkv * D), "f32", seed + 1, DEV) * s).to(torch.bfloat16)
    wv = (fw.randn((d, Hkv * D), "f32", seed + 2, DEV) * s).to(torch.bfloat16)
    wo = (fw.randn((H * D, d), "f32", seed + 3, DEV) / np.sqrt(H * D)).to(torch.bfloat16)
    return wq, wk, wv, wo


def _layer_parity(got, ref, what):
    """Layer bar: rel-L2 <= 5e-3 (as every bf16 output) and max-abs <= 5e-2 of
    the output's RMS.  The max-abs bar is looser than the attention's 2e-2
    because the layer's largest outputs reach ~4 RMS, where one bf16 ulp of the
    output is 2^-8 * 4 RMS = 1.6e-2 RMS, and each of the four bf16-stored
    intermediates (Q, K, V, attention output) may round to the other neighbour
    of a float32 sum than the float64 reference does (one ulp, 2^-8 relative)."""
    rms = float(np.sqrt(np.mean(ref ** 2)))
    g, r = got / rms, ref / rms
    err = float(np.abs(g - r).max())
    rl2 = float(np.linalg.norm(g - r) / np.linalg.norm(r))
    assert err <= 5e-2 and rl2 <= 5e-3, f"{what}: max-abs {err:.3e} RMS (<= 5e-2), rel-L2 {rl2:.3e} (<= 5e-3)"


def _layer_parity_fp64(got, ref, what):
    """Bar against the plain float64 layer (no intermediate rounding).  The
    device stores five values in bf16: Q, K, V, the attention output and the
    layer output.  Each rounding leaves a relative error of RMS u / sqrt(3)
    (u = 2^-9, half a bf16 ulp, errors uniform over +-u); five independent ones
    add to sqrt(5) u / sqrt(3) = 2.5e-3 relative.  The softmax turns a relative
    error e of Q or K into an error of about e |s| on the probabilities (scores s
    of a few units here), so the total stays near 5e-3: the bar is rel-L2 <= 1e-2.
    The largest outputs reach ~7 RMS, where the final rounding alone is up to
    u 7 RMS = 1.4e-2 RMS; the propagated part, roughly Gaussian with sigma
    ~5e-3 RMS, stays below 5 sigma over ~1e5 outputs: max-abs <= 6e-2 RMS.
    (float32 accumulation over d_model <= 4096 terms adds ~1e-5, negligible.)"""
    rms = float(np.sqrt(np.mean(ref ** 2)))
    g, r = got / rms, ref / rms
    err = float(np.abs(g - r).max())
    rl2 = float(np.linalg.norm(g - r) / np.linalg.norm(r))
    assert err <= 6e-2 and rl2 <= 1e-2, f"{what}: max-abs {err:.3e} RMS (<= 6e-2), rel-L2 {rl2:.3e} (<= 1e-2)"


@pytest.mark.parametrize("mask", list(MASKS))
@pytest.mark.parametrize("seq,W,kmer,H,Hkv,D,d", [
    ([2500], 1000, 100, 2, 2, 128, 256),
    ([1300, 700], 500, None, 4, 2, 64, 384),
])
def test_adapter_layer_small(seq, W, kmer, H, Hkv, D, d, mask):
    announce(f"adapter layer seq={seq} d={d} mask={mask}")
    km = _kmer_for(seq, W, kmer, 5)
    tot = F.focus_layout_plan(seq, W, km)
    lay = F.focus_layout(tot, seq, W, km)
    hid = fw.randn((tot.n_tokens, d), "bf16", 91, DEV)
    ws = _weights(d, H, Hkv, D, 17)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = F.focus_adapter_layer(lay, hid, *ws, H, Hkv, mask=MASKS[mask], err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    ref = build_layout(seq, W, km)
    o_ref = AD.adapter_layer(ref, to64(hid), *[to64(x) for x in ws], H, Hkv, mask, store_bf16=True)
    _layer_parity(to64(out), o_ref, f"adapter layer {mask}")
    o64 = AD.adapter_layer(ref, to64(hid), *[to64(x) for x in ws], H, Hkv, mask, store_bf16=False)
    _layer_parity_fp64(to64(out), o64, f"adapter layer {mask} vs float64")


def test_adapter_layer_evo2_scale_100kb_sampled():
    w = fw.WORKLOADS["prefill_100kb"]
    d, H, Hkv, D = 4096, w.heads, w.kv_heads, w.head_dim
    announce("adapter layer 100 kb, d_model 4096")
    seq = [w.seq_nt]
    km = fw.kmer_draw(w)
    tot = F.focus_layout_plan(seq, w.window_nt, km)
    lay = F.focus_layout(tot, seq, w.window_nt, km)
    hid = fw.randn((tot.n_tokens, d), "bf16", 92, DEV)
    ws = _weights(d, H, Hkv, D, 23)
    out = F.focus_adapter_layer(lay, hid, *ws, H, Hkv)
    torch.cuda.synchronize()
    ref = build_layout(seq, w.window_nt, km)
    wins = [0, ref["n_windows"] - 1]
    fetch = lambda r: to64(hid[torch.as_tensor(np.asarray(r, np.int64), device=DEV)])   # noqa: E731
    o_ref = AD.adapter_layer(ref, fetch, *[to64(x) for x in ws], H, Hkv, "ct", store_bf16=True, windows=wins)
    sums = np.concatenate([np.arange(ref["win_sum_off"][x], ref["win_sum_off"][x] + ref["win_nsum"][x]) for x in wins])
    got = to64(out[torch.as_tensor(sums, device=DEV)])
    _layer_parity(got, o_ref[sums], "adapter layer 100 kb")
    o64 = AD.adapter_layer(ref, fetch, *[to64(x) for x in ws], H, Hkv, "ct", store_bf16=False, windows=wins)
    _layer_parity_fp64(got, o64[sums], "adapter layer 100 kb vs float64")
