"""CPU checks of the C ABI: the library loads, exports every symbol the header
declares, the binding's struct mirrors match, the host-side plan agrees with
the oracle's layout, and host validation rejects bad descriptors before any
launch (no GPU is touched: every call here returns before enqueueing work)."""

import ctypes as C
import os
import re

import numpy as np
import pytest

import focus_workloads as fw
import paper_2511_14694_amd as F
from paper_2511_14694_amd import _abi
from oracle.layout import build_layout

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "focus.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(focus_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = _abi.lib()
    declared = header_functions()
    assert set(declared) == set(_abi.SYMBOLS), "binding and header disagree"
    for name in declared:
        assert hasattr(lib, name), name
    nm = os.popen(f"nm -D --defined-only {_abi.LIB_PATH}").read()
    for name in declared:
        assert re.search(rf"\bT {name}\b", nm), f"{name} not exported"


def test_struct_mirrors_and_version():
    lib = _abi.lib()
    for i, st in enumerate(_abi.STRUCTS):
        assert lib.focus_struct_size(i) == C.sizeof(st)
    assert lib.focus_struct_size(99) == -1
    assert F.focus_abi_version() == 3
    assert lib.focus_status_str(0) == b"ok"
    assert lib.focus_status_str(5) == b"unsupported configuration"


def _oracle_totals(seq, W, kmer):
    lay = build_layout(seq, W, kmer)
    cache_per_seq = [int(lay["win_nsum"][lay["win_seq"] == b].sum()) for b in range(len(seq))]
    return {
        "n_windows": lay["n_windows"], "n_tokens": lay["n_tokens"], "n_summaries": lay["n_summaries"],
        "max_window_tokens": int(lay["win_ntok"].max(initial=0)),
        "max_window_summaries": int(lay["win_nsum"].max(initial=0)),
        "max_cache_per_seq": max(cache_per_seq, default=0),
        "max_window_cache": int(lay["win_cache_off"].max(initial=0)),
    }


@pytest.mark.parametrize("seed", range(25))
def test_plan_matches_oracle_random(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(0, 5))
    seq = [int(x) for x in rng.integers(0, 300, B)]
    W = int(rng.integers(1, 80))
    nw = sum(-(-L // W) for L in seq)
    kmer = rng.integers(0, 30, nw).astype(np.int32)
    got = F.focus_layout_plan(seq, W, kmer).as_dict()
    assert got == _oracle_totals(seq, W, kmer)
    if nw:
        got_u = F.focus_layout_plan(seq, W, None, int(kmer[0])).as_dict()
        assert got_u == _oracle_totals(seq, W, int(kmer[0]))


@pytest.mark.parametrize("name", ["tiny_4kb_f32", "prefill_100kb", "prefill_1mb",
                                  "ragged_b8_256kb", "dense_32kb"])
def test_plan_matches_oracle_workloads(name):
    w = fw.WORKLOADS[name]
    seq = [w.seq_nt] * w.batch
    kmer = fw.kmer_draw(w)
    assert F.focus_layout_plan(seq, w.window_nt, kmer).as_dict() == _oracle_totals(seq, w.window_nt, kmer)


def test_plan_rejects_bad_arguments():
    with pytest.raises(F.FocusError) as e:
        F.focus_layout_plan([10], 0, None, 3)
    assert e.value.status == 2
    with pytest.raises(F.FocusError):
        F.focus_layout_plan([-1], 4, None, 3)
    with pytest.raises(F.FocusError):
        F.focus_layout_plan([10], 4, None, -1)
    with pytest.raises(F.FocusError):
        F.focus_layout_plan([10, 5], 4, np.array([1, 1, 1, -2, 1], np.int32))
    assert F.focus_layout_plan([], 4, None, 3).n_windows == 0


# ---- host validation: each descriptor below is rejected before any launch ----

def _call(fn, desc):
    return getattr(_abi.lib(), fn)(C.byref(desc), None)


def _attn_ok():
    d = _abi.AttnDesc()
    d.totals = F.focus_layout_plan([100], 50, None, 10)
    d.dtype, d.n_heads, d.n_kv_heads, d.head_dim = 0, 4, 2, 128
    d.batch = 1
    fake = 1 << 20   # aligned, never dereferenced: every case below fails validation first
    for f in ("win_seq", "win_ntok", "win_cache_off", "win_tok_off", "q", "k", "v", "o",
              "cache_k", "cache_v"):
        setattr(d, f, fake)
    d.qkv_rows = 110
    d.cache_cap = 10
    return d


@pytest.mark.parametrize("mutate,status", [
    (lambda d: setattr(d, "dtype", 7), 4),
    (lambda d: setattr(d, "head_dim", 96), 5),
    (lambda d: setattr(d, "kmer_uniform", -1) or setattr(d, "mask", 1), 2),
    (lambda d: setattr(d, "mask", 9), 2),
    (lambda d: setattr(d, "n_kv_heads", 3), 3),
    (lambda d: setattr(d, "n_heads", 0), 2),
    (lambda d: setattr(d, "q", None), 1),
    (lambda d: setattr(d, "o", (1 << 20) + 8), 2),
    (lambda d: setattr(d, "cache_cap", 1), 7),
    (lambda d: setattr(d, "softmax_scale", float("nan")), 2),
])
def test_window_attn_host_validation(mutate, status):
    d = _attn_ok()
    mutate(d)
    assert _call("focus_window_attn", d) == status
    assert _abi.lib().focus_window_attn(None, None) == 1


def _decode_ok():
    d = _abi.DecodeDesc()
    d.dtype, d.batch, d.n_heads, d.n_kv_heads, d.head_dim = 0, 2, 4, 4, 128
    fake = 1 << 20
    for f in ("q", "k_new", "v_new", "kind", "cache_k", "cache_v", "cache_len", "win_k", "win_v",
              "win_len", "o"):
        setattr(d, f, fake)
    d.cache_cap, d.win_cap = 100, 10
    return d


@pytest.mark.parametrize("mutate,status", [
    (lambda d: setattr(d, "dtype", 3), 4),
    (lambda d: setattr(d, "head_dim", 80), 5),
    (lambda d: setattr(d, "split_keys", 24), 2),
    (lambda d: setattr(d, "n_kv_heads", 3), 3),
    (lambda d: setattr(d, "win_len", None), 1),
    (lambda d: None, 6),                      # no workspace
])
def test_decode_host_validation(mutate, status):
    d = _decode_ok()
    mutate(d)
    assert _call("focus_decode_step", d) == status


def test_decode_workspace_size_formula():
    d = _decode_ok()
    d.split_keys = 32
    n_split = -(-(100 + 10) // 32)
    # partials (o, max, sum) per (sequence, split, head) + one key count per sequence
    assert _abi.lib().focus_decode_workspace(C.byref(d)) == 2 * n_split * 4 * (128 + 2) * 4 + 16
    d.head_dim = 80
    assert _abi.lib().focus_decode_workspace(C.byref(d)) == 0


@pytest.mark.parametrize("mutate,status", [
    (lambda d: setattr(d, "dtype", 5), 4),
    (lambda d: setattr(d, "head_dim", 32), 5),
    (lambda d: setattr(d, "k", None), 1),
    (lambda d: setattr(d, "cache_cap", 3), 7),
    (lambda d: setattr(d, "cache_k", (1 << 20) + 4), 2),
])
def test_compact_host_validation(mutate, status):
    d = _abi.CompactDesc()
    d.totals = F.focus_layout_plan([100], 50, None, 10)
    d.dtype, d.n_kv_heads, d.head_dim, d.batch = 0, 2, 64, 1
    fake = 1 << 20
    for f in ("win_seq", "win_nsum", "win_cache_off", "win_sum_off", "sum_tok", "k", "v",
              "cache_k", "cache_v"):
        setattr(d, f, fake)
    d.kv_rows, d.cache_cap = 110, 10
    mutate(d)
    assert _call("focus_compact_kv", d) == status


@pytest.mark.parametrize("mutate,status", [
    (lambda d: setattr(d, "window_nt", 0), 2),
    (lambda d: setattr(d, "batch", -1), 2),
    (lambda d: setattr(d, "cu_tokens", None), 1),
    (lambda d: setattr(d, "sum_tok", None), 1),
    (lambda d: setattr(d, "token_ids", None), 1),
])
def test_layout_host_validation(mutate, status):
    d = _abi.LayoutDesc()
    d.totals = F.focus_layout_plan([100], 50, None, 10)
    d.batch, d.window_nt, d.kmer_uniform = 1, 50, 10
    fake = 1 << 20
    for f, _ in _abi.LayoutDesc._fields_[5:-1]:
        setattr(d, f, fake)
    mutate(d)
    assert _call("focus_layout", d) == status


def _fid_ok():
    d = _abi.FidelityDesc()
    d.dtype, d.input_kind, d.n_pos, d.vocab = 1, 0, 10, 4
    fake = 1 << 20
    d.p, d.q, d.out = fake, fake, fake
    return d


@pytest.mark.parametrize("mutate,status", [
    (lambda d: setattr(d, "dtype", 9), 4),
    (lambda d: setattr(d, "input_kind", 3), 2),
    (lambda d: setattr(d, "vocab", 0), 2),
    (lambda d: setattr(d, "vocab", 1025), 5),
    (lambda d: setattr(d, "n_pos", -1), 2),
    (lambda d: setattr(d, "p", None), 1),
    (lambda d: setattr(d, "q", (1 << 20) + 2), 2),
    (lambda d: (setattr(d, "n_seq", 2), setattr(d, "seq_mean", 1 << 20)), 2),   # no cu_pos
])
def test_fidelity_host_validation(mutate, status):
    d = _fid_ok()
    mutate(d)
    assert _call("focus_fidelity", d) == status


def test_window_attn_workspace_key_split_formula():
    """Key split of a bf16 C(t) launch: n = min(CUs // items, key tiles // 8, 16)
    splits when that is at least 2, each holding float32 (O, max, sum) per
    (listed window, padded row, head); otherwise no workspace.  (MI355X: 256
    CUs, also the fallback when no device answers.)"""
    d = _attn_ok()
    d.totals = F.focus_layout_plan([1_000_000], 1000, None, 100)
    d.n_heads = d.n_kv_heads = 32
    t = d.totals
    assert (t.max_window_tokens, t.max_window_cache) == (1010, 9990)
    ws = lambda: _abi.lib().focus_window_attn_workspace(C.byref(d))
    assert ws() == 0                                   # every window: 128 000 items
    d.win_ids, d.n_win = 1 << 20, 1                    # one window: 32 heads x 4 query tiles
    rows = 4 * 256
    assert ws() == 2 * 1 * rows * 32 * (128 + 2) * 4   # 256 // 128 = 2 splits
    d.n_heads = d.n_kv_heads = 4                       # 16 items: 16 splits (173 tiles // 8 = 21)
    assert ws() == 16 * 1 * rows * 4 * (128 + 2) * 4
    d.head_dim = 64
    assert ws() == 16 * 1 * rows * 4 * (64 + 2) * 4
    d.mask = 1
    assert ws() == 0                                   # k-mer-local: never split
    d.mask, d.dtype = 0, 1
    assert ws() == 0                                   # float32: never split
    d.dtype = 0
    d.totals = F.focus_layout_plan([100], 50, None, 10)
    assert ws() == 0                                   # two key tiles: nothing to split
