"""FOCUS hot path for AMD MI355X (gfx950): Python binding of libfocus.so.

A thin layer over the C ABI declared in include/focus.h: each function below
has the name of the C call it wraps and only marshals arguments (device
pointers of torch tensors, the current HIP stream, descriptor structs).  Every
step of the computation runs in the library's HIP kernels; torch provides
device memory and streams.  There is no CPU fallback: if libfocus.so is missing
the first call raises.

    totals = focus_layout_plan(seq_nt, window_nt, kmer)          # host
    lay    = focus_layout(totals, seq_nt, window_nt, kmer)       # device metadata
    focus_compact_kv(lay, k, v, cache_k, cache_v, cache_len)     # summary K/V -> cache
    o, lse = focus_window_attn(lay, q, k, v, cache_k, cache_v)   # [cache ; window] attention
    o, lse = focus_decode_step(q, k_new, v_new, kind, ...)       # one decode step
"""

from __future__ import annotations

import ctypes as C
from dataclasses import dataclass, field
from typing import Dict, Optional

import numpy as np
import torch

from ._abi import (AdapterDesc, AdapterLayerDesc, AttnDesc, CompactDesc, DecodeDesc, DecodeSched, FidelityDesc, FocusError, GemmDesc, LayoutDesc, LayoutTotals, QkvDesc,
                   FOCUS_BF16, FOCUS_F32, FOCUS_MASK_CT, FOCUS_MASK_KMER_LOCAL,
                   FOCUS_TOK_BASE, FOCUS_TOK_SUMMARY, FOCUS_STEP_SUMMARY, FOCUS_STEP_WINDOW_END,
                   FOCUS_ERR_CAPACITY, FOCUS_ERR_BOUNDS, FOCUS_ERR_PLAN,
                   FOCUS_FID_LOGITS, FOCUS_FID_PROBS, FOCUS_FID_N, check, lib)

__all__ = ["focus_layout_plan", "focus_layout", "focus_compact_kv", "focus_window_attn",
           "focus_window_attn_workspace", "focus_decode_step", "focus_decode_workspace",
           "focus_decode_step_noalloc", "DecodeSchedule",
           "focus_fidelity", "focus_gemm", "focus_adapter_attn", "focus_adapter_layer",
           "focus_adapter_layer_workspace", "focus_qkv_project", "focus_abi_version", "Layout", "LayoutTotals", "FocusError",
           "FOCUS_FID_LOGITS", "FOCUS_FID_PROBS", "FOCUS_FID_N",
           "FOCUS_BF16", "FOCUS_F32", "FOCUS_MASK_CT", "FOCUS_MASK_KMER_LOCAL",
           "FOCUS_TOK_BASE", "FOCUS_TOK_SUMMARY", "FOCUS_STEP_SUMMARY", "FOCUS_STEP_WINDOW_END",
           "FOCUS_ERR_CAPACITY", "FOCUS_ERR_BOUNDS", "FOCUS_ERR_PLAN"]

_DTYPES = {torch.bfloat16: FOCUS_BF16, torch.float32: FOCUS_F32}

WINDOW_FIELDS = ("win_seq", "win_nt", "win_nsum", "win_ntok", "win_cache_off",
                 "win_tok_off", "win_sum_off", "win_base_off")
TOKEN_FIELDS = ("tok_pos", "tok_kmer", "tok_win", "tok_kind", "tok_base")
_FIELD_DTYPE = {"cu_windows": torch.int64, "cu_tokens": torch.int64, "cu_summaries": torch.int64,
                "win_seq": torch.int32, "win_nt": torch.int32, "win_nsum": torch.int32,
                "win_ntok": torch.int32, "win_cache_off": torch.int32, "win_tok_off": torch.int64,
                "win_sum_off": torch.int64, "win_base_off": torch.int64, "tok_pos": torch.int32,
                "tok_kmer": torch.int32, "tok_win": torch.int32, "tok_kind": torch.uint8,
                "tok_base": torch.int64, "sum_tok": torch.int64, "token_ids": torch.int32,
                "tok_next_base": torch.int64}


def focus_abi_version() -> int:
    return lib().focus_abi_version()


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libfocus must be contiguous")
    return t.data_ptr()


def _ptr_rows(t) -> int:
    """Pointer of a 2-D tensor with unit column stride (any row stride)."""
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("expected a 2-D tensor with unit column stride")
    return t.data_ptr()


def _stream(stream, device) -> int:
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return stream.cuda_stream


def _scratch(nbytes: int, device, stream):
    """Scratch for the duration of one call: allocated on the stream the call's
    kernels run on, so the caching allocator hands the block to other work only
    behind them once it is freed (on the caller's current stream when stream is
    None)."""
    if stream is None:
        return torch.empty(nbytes, dtype=torch.uint8, device=device)
    with torch.cuda.stream(stream):
        return torch.empty(nbytes, dtype=torch.uint8, device=device)


def _dtype(t) -> int:
    if t.dtype not in _DTYPES:
        raise ValueError(f"unsupported dtype {t.dtype}")
    return _DTYPES[t.dtype]


def focus_layout_plan(seq_nt, window_nt: int, kmer=None, kmer_uniform: int = 0) -> LayoutTotals:
    """Host-side totals of the layout (sizes every device buffer)."""
    seq = np.ascontiguousarray(np.asarray(seq_nt, dtype=np.int64).reshape(-1))
    km = None if kmer is None else np.ascontiguousarray(np.asarray(kmer, dtype=np.int32).reshape(-1))
    out = LayoutTotals()
    st = lib().focus_layout_plan(len(seq), seq.ctypes.data if len(seq) else None, int(window_nt),
                                 None if km is None else km.ctypes.data, int(kmer_uniform),
                                 C.byref(out))
    check("focus_layout_plan", st)
    return out


@dataclass
class Layout:
    """Device-resident layout produced by focus_layout (arrays named as in focus.h)."""
    totals: LayoutTotals
    batch: int
    window_nt: int
    arrays: Dict[str, torch.Tensor] = field(default_factory=dict)
    kmer: Optional[torch.Tensor] = None   # per-window k given to focus_layout (device), or None
    kmer_uniform: int = 0                 # k of every window when kmer is None

    def __getitem__(self, name):
        return self.arrays[name]

    def to_numpy(self) -> Dict[str, np.ndarray]:
        return {k: v.cpu().numpy() for k, v in self.arrays.items()}


def focus_layout(totals: LayoutTotals, seq_nt, window_nt: int, kmer=None, kmer_uniform: int = 0,
                 bases=None, summary_token_id: int = 0, err=None, device="cuda", stream=None,
                 out: Optional[Layout] = None, next_base: bool = False) -> Layout:
    """Fill the layout arrays on the device.  seq_nt / kmer / bases may be host
    arrays (copied to the device) or device tensors.  `out`: a Layout of the
    same totals whose arrays are written again instead of allocating new ones.
    next_base: also fill tok_next_base (the target map pi(t))."""
    dev = torch.device(device)
    seq = torch.as_tensor(np.asarray(seq_nt, dtype=np.int64) if not torch.is_tensor(seq_nt) else seq_nt,
                          dtype=torch.int64).to(dev).contiguous()
    km = None
    if kmer is not None:
        km = torch.as_tensor(np.asarray(kmer, dtype=np.int32) if not torch.is_tensor(kmer) else kmer,
                             dtype=torch.int32).to(dev).contiguous()
    bs = None
    if bases is not None:
        bs = torch.as_tensor(np.asarray(bases, dtype=np.uint8) if not torch.is_tensor(bases) else bases,
                             dtype=torch.uint8).to(dev).contiguous()
    B = seq.numel()
    sizes = {"cu_windows": B + 1, "cu_tokens": B + 1, "cu_summaries": B + 1,
             "sum_tok": totals.n_summaries}
    sizes.update({f: totals.n_windows for f in WINDOW_FIELDS})
    sizes.update({f: totals.n_tokens for f in TOKEN_FIELDS})
    if bs is not None:
        sizes["token_ids"] = totals.n_tokens
    if next_base:
        sizes["tok_next_base"] = totals.n_tokens
    if out is not None:
        arrays = out.arrays
        if any(f not in arrays or arrays[f].numel() != max(int(n), 0) for f, n in sizes.items()):
            raise ValueError("`out` layout has different sizes")
    else:
        arrays = {f: torch.empty(max(int(n), 0), dtype=_FIELD_DTYPE[f], device=dev) for f, n in sizes.items()}
    d = LayoutDesc()
    d.totals = totals
    d.batch, d.window_nt, d.kmer_uniform, d.summary_token_id = B, int(window_nt), int(kmer_uniform), int(summary_token_id)
    d.seq_nt, d.kmer, d.bases, d.err = _ptr(seq), _ptr(km), _ptr(bs), _ptr(err)
    for f, t in arrays.items():
        setattr(d, f, _ptr(t))
    check("focus_layout", lib().focus_layout(C.byref(d), _stream(stream, dev)))
    return Layout(totals, B, int(window_nt), arrays, km, int(kmer_uniform))


def focus_compact_kv(lay: Layout, k, v, cache_k, cache_v, cache_len=None, win_ids=None,
                     kv_tok_base: int = 0, err=None, stream=None):
    """Append the summary K/V rows of the listed windows (all if win_ids is None)
    to cache_k / cache_v [batch, cap, H_kv, D]; raise cache_len."""
    d = CompactDesc()
    d.totals = lay.totals
    d.dtype = _dtype(k)
    d.n_kv_heads, d.head_dim = k.shape[1], k.shape[2]
    d.batch = lay.batch
    d.n_win = 0 if win_ids is None else win_ids.numel()
    d.win_ids = _ptr(win_ids)
    for f in ("win_seq", "win_nsum", "win_cache_off", "win_sum_off", "sum_tok"):
        setattr(d, f, _ptr(lay[f]))
    d.k, d.v, d.kv_tok_base, d.kv_rows = _ptr(k), _ptr(v), int(kv_tok_base), k.shape[0]
    if (cache_k.shape != cache_v.shape or cache_k.dtype != k.dtype or cache_k.shape[2:] != k.shape[1:]
            or cache_k.shape[0] < lay.batch or v.shape != k.shape):
        raise ValueError("cache shape/dtype does not match k, or holds fewer sequences than the layout")
    if cache_len is not None and cache_len.numel() < lay.batch:
        raise ValueError("cache_len needs one entry per sequence")
    d.cache_k, d.cache_v, d.cache_cap = _ptr(cache_k), _ptr(cache_v), cache_k.shape[1]
    d.cache_len, d.err = _ptr(cache_len), _ptr(err)
    check("focus_compact_kv", lib().focus_compact_kv(C.byref(d), _stream(stream, k.device)))


def _attn_desc(lay, q, k, v, cache_k, cache_v, o, lse, win_ids, qkv_tok_base, softmax_scale, mask,
               workspace, err):
    d = AttnDesc()
    d.totals = lay.totals
    d.dtype = _dtype(q)
    d.n_heads, d.head_dim = q.shape[1], q.shape[2]
    d.n_kv_heads = k.shape[1]
    d.softmax_scale = float(softmax_scale)
    d.mask = int(mask)
    d.batch = lay.batch
    d.kmer_uniform = int(lay.kmer_uniform)
    d.win_kmer = _ptr(lay.kmer)
    d.n_win = 0 if win_ids is None else win_ids.numel()
    d.win_ids = _ptr(win_ids)
    for f in ("win_seq", "win_ntok", "win_cache_off", "win_tok_off"):
        setattr(d, f, _ptr(lay[f]))
    if not (q.dtype == k.dtype == v.dtype) or k.shape != v.shape or q.shape[0] != k.shape[0]:
        raise ValueError("q/k/v shapes or dtypes disagree")
    d.q, d.k, d.v, d.qkv_tok_base, d.qkv_rows = _ptr(q), _ptr(k), _ptr(v), int(qkv_tok_base), q.shape[0]
    if cache_k is not None:
        if (cache_k.dtype != q.dtype or cache_k.shape[2:] != k.shape[1:] or cache_k.shape != cache_v.shape
                or cache_k.shape[0] < lay.batch):
            raise ValueError("cache shape/dtype does not match k, or holds fewer sequences than the layout")
        d.cache_k, d.cache_v, d.cache_cap = _ptr(cache_k), _ptr(cache_v), cache_k.shape[1]
    d.o, d.lse = _ptr(o), _ptr(lse)
    d.workspace = _ptr(workspace)
    d.workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    d.err = _ptr(err)
    return d


def focus_window_attn_workspace(lay: Layout, q, k, v, cache_k=None, cache_v=None, win_ids=None,
                                mask: int = FOCUS_MASK_CT) -> int:
    d = _attn_desc(lay, q, k, v, cache_k, cache_v, None, None, win_ids, 0, 0.0, mask, None, None)
    return lib().focus_window_attn_workspace(C.byref(d))


def focus_window_attn(lay: Layout, q, k, v, cache_k=None, cache_v=None, o=None, lse=None,
                      win_ids=None, qkv_tok_base: int = 0, softmax_scale: float = 0.0,
                      mask: int = FOCUS_MASK_CT, workspace=None, want_lse: bool = True,
                      err=None, stream=None):
    """Window attention over [cache ; window] for the listed windows (all if
    win_ids is None).  q [rows, H, D], k/v [rows, H_kv, D]; returns (o, lse).
    workspace None allocates what focus_window_attn_workspace asks for; an
    empty tensor runs without the key split."""
    if o is None:
        o = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty(q.shape[0], q.shape[1], dtype=torch.float32, device=q.device)
    if o.shape != q.shape or o.dtype != q.dtype or (lse is not None and tuple(lse.shape) != tuple(q.shape[:2])):
        raise ValueError("o must match q; lse must be [rows, heads]")
    if workspace is None:
        # key-split scratch for launches that would leave compute units idle
        n = focus_window_attn_workspace(lay, q, k, v, cache_k, cache_v, win_ids, mask)
        workspace = _scratch(n, q.device, stream) if n > 0 else None
    d = _attn_desc(lay, q, k, v, cache_k, cache_v, o, lse, win_ids, qkv_tok_base, softmax_scale,
                   mask, workspace, err)
    check("focus_window_attn", lib().focus_window_attn(C.byref(d), _stream(stream, q.device)))
    return o, lse


def _decode_desc(q, k_new, v_new, kind, cache_k, cache_v, cache_len, win_k, win_v, win_len,
                 o, lse, workspace, split_keys, softmax_scale, err):
    d = DecodeDesc()
    d.dtype = _dtype(q)
    d.batch, d.n_heads, d.head_dim = q.shape
    d.n_kv_heads = k_new.shape[1]
    d.softmax_scale = float(softmax_scale)
    d.split_keys = int(split_keys)
    d.q, d.k_new, d.v_new, d.kind = _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(kind)
    d.cache_k, d.cache_v, d.cache_cap, d.cache_len = _ptr(cache_k), _ptr(cache_v), cache_k.shape[1], _ptr(cache_len)
    d.win_k, d.win_v, d.win_cap, d.win_len = _ptr(win_k), _ptr(win_v), win_k.shape[1], _ptr(win_len)
    d.o, d.lse = _ptr(o), _ptr(lse)
    d.workspace = _ptr(workspace)
    d.workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    d.err = _ptr(err)
    return d


def focus_decode_workspace(q, k_new, cache_k, win_k, split_keys: int = 0) -> int:
    d = DecodeDesc()
    d.dtype = _dtype(q)
    d.batch, d.n_heads, d.head_dim = q.shape
    d.n_kv_heads = k_new.shape[1]
    d.split_keys = int(split_keys)
    d.cache_cap, d.win_cap = cache_k.shape[1], win_k.shape[1]
    return lib().focus_decode_workspace(C.byref(d))


def focus_decode_step(q, k_new, v_new, kind, cache_k, cache_v, cache_len, win_k, win_v, win_len,
                      o=None, lse=None, workspace=None, split_keys: int = 0,
                      softmax_scale: float = 0.0, want_lse: bool = True, err=None, stream=None):
    """One decode step for every sequence of the batch; returns (o, lse)."""
    if o is None:
        o = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty(q.shape[0], q.shape[1], dtype=torch.float32, device=q.device)
    B, H, D = q.shape
    Hkv = k_new.shape[1]
    if (k_new.shape != (B, Hkv, D) or v_new.shape != k_new.shape or kind.numel() < B
            or cache_k.shape[0] < B or cache_k.shape[2:] != (Hkv, D) or cache_v.shape != cache_k.shape
            or win_k.shape[0] < B or win_k.shape[2:] != (Hkv, D) or win_v.shape != win_k.shape
            or cache_len.numel() < B or win_len.numel() < B or o.shape != q.shape
            or (lse is not None and tuple(lse.shape) != (B, H))):
        raise ValueError("decode tensor shapes disagree")
    if workspace is None:
        n = focus_decode_workspace(q, k_new, cache_k, win_k, split_keys)
        workspace = _scratch(max(n, 16), q.device, stream)
    d = _decode_desc(q, k_new, v_new, kind, cache_k, cache_v, cache_len, win_k, win_v, win_len,
                     o, lse, workspace, split_keys, softmax_scale, err)
    check("focus_decode_step", lib().focus_decode_step(C.byref(d), _stream(stream, q.device)))
    return o, lse


class DecodeSchedule:
    """Device-side decode schedule of a batch (focus_decode_sched): each
    sequence's current window, bases in it and bases in its open k-mer.

    kmer: None (kmer_uniform for every window) or [batch, n] cadences of the
    windows j = 0, 1, ... of each sequence (the last one repeats); win_index:
    each sequence's current window (default 0)."""

    def __init__(self, batch: int, window_nt: int, kmer=None, kmer_uniform: int = 0, win_index=None,
                 device="cuda", err=None):
        dev = torch.device(device)
        self.batch, self.window_nt, self.kmer_uniform = int(batch), int(window_nt), int(kmer_uniform)
        self.kmer = None
        if kmer is not None:
            km = torch.as_tensor(np.asarray(kmer, np.int32) if not torch.is_tensor(kmer) else kmer,
                                 dtype=torch.int32).to(dev).contiguous()
            if km.dim() != 2 or km.shape[0] != batch or km.shape[1] < 1:
                raise ValueError("kmer must be [batch, windows]")
            self.kmer = km
        z = lambda dt: torch.zeros(batch, dtype=dt, device=dev)   # noqa: E731
        self.win_index = z(torch.int32) if win_index is None else \
            torch.as_tensor(win_index, dtype=torch.int32).to(dev).contiguous()
        self.bases_in_window, self.bases_in_kmer = z(torch.int32), z(torch.int32)
        self.kind = z(torch.uint8)
        self.summaries = z(torch.int32)
        self.err = err

    def _desc(self, tokens=None):
        d = DecodeSched()
        d.batch, d.window_nt, d.kmer_uniform = self.batch, self.window_nt, self.kmer_uniform
        d.kmer_stride = 0 if self.kmer is None else self.kmer.shape[1]
        d.kmer = _ptr(self.kmer)
        d.win_index, d.bases_in_window = _ptr(self.win_index), _ptr(self.bases_in_window)
        d.bases_in_kmer, d.kind = _ptr(self.bases_in_kmer), _ptr(self.kind)
        d.tokens, d.summaries, d.err = _ptr(tokens), _ptr(self.summaries), _ptr(self.err)
        return d

    def start(self, tokens, stream=None):
        """Walk tokens[b] tokens into each sequence's current window; returns
        the device tensor of how many of them are summaries."""
        t = torch.as_tensor(tokens, dtype=torch.int32).to(self.kind.device).contiguous()
        d = self._desc(t)
        check("focus_decode_sched_start", lib().focus_decode_sched_start(C.byref(d),
                                                                       _stream(stream, self.kind.device)))
        return self.summaries

    def next_kind(self, stream=None):
        """Derive the next token's kinds into self.kind (returned) and advance."""
        d = self._desc()
        check("focus_decode_next_kind", lib().focus_decode_next_kind(C.byref(d), _stream(stream, self.kind.device)))
        return self.kind


def focus_decode_step_noalloc(q, k_new, v_new, kind, cache_k, cache_v, cache_len, win_k, win_v, win_len,
                              o, lse=None, split_keys: int = 0, softmax_scale: float = 0.0, err=None,
                              stream=None):
    """focus_decode_step with the partials in the library's per-device scratch
    array: allocates nothing, so o (and lse, if wanted) must be given."""
    B, H, D = q.shape
    Hkv = k_new.shape[1]
    if (k_new.shape != (B, Hkv, D) or v_new.shape != k_new.shape or kind.numel() < B
            or cache_k.shape[0] < B or cache_k.shape[2:] != (Hkv, D) or cache_v.shape != cache_k.shape
            or win_k.shape[0] < B or win_k.shape[2:] != (Hkv, D) or win_v.shape != win_k.shape
            or cache_len.numel() < B or win_len.numel() < B or o.shape != q.shape
            or (lse is not None and tuple(lse.shape) != (B, H))):
        raise ValueError("decode tensor shapes disagree")
    d = _decode_desc(q, k_new, v_new, kind, cache_k, cache_v, cache_len, win_k, win_v, win_len,
                     o, lse, None, split_keys, softmax_scale, err)
    check("focus_decode_step_noalloc", lib().focus_decode_step_noalloc(C.byref(d), _stream(stream, q.device)))
    return o, lse


def focus_fidelity(p, q, input_kind: int = FOCUS_FID_LOGITS, cu_pos=None, out=None, seq_mean=None,
                   err=None, stream=None):
    """Per-position L1 / L2 / Hellinger / JS / KL between the rows of p and q
    ([n_pos, vocab], logits or probabilities); with cu_pos ([n_seq + 1] row
    offsets) also the per-sequence means.  Returns (out [n_pos, 5], seq_mean)."""
    if p.shape != q.shape or p.dtype != q.dtype or p.dim() != 2 or not p.is_contiguous() \
            or not q.is_contiguous():
        raise ValueError("p and q must be contiguous [n_pos, vocab] tensors of one dtype")
    n_pos, vocab = p.shape
    if out is None:
        out = torch.empty(n_pos, FOCUS_FID_N, dtype=torch.float32, device=p.device)
    if tuple(out.shape) != (n_pos, FOCUS_FID_N) or out.dtype != torch.float32:
        raise ValueError("out must be float32 [n_pos, 5]")
    n_seq = 0
    if cu_pos is not None:
        cu_pos = torch.as_tensor(cu_pos, dtype=torch.int64).to(p.device).contiguous()
        n_seq = cu_pos.numel() - 1
        if seq_mean is None:
            seq_mean = torch.empty(n_seq, FOCUS_FID_N, dtype=torch.float32, device=p.device)
    d = FidelityDesc()
    d.dtype = _dtype(p)
    d.input_kind = int(input_kind)
    d.n_pos, d.vocab, d.n_seq = n_pos, vocab, n_seq
    d.p, d.q, d.out = _ptr(p), _ptr(q), _ptr(out)
    d.cu_pos, d.seq_mean, d.err = _ptr(cu_pos), _ptr(seq_mean), _ptr(err)
    check("focus_fidelity", lib().focus_fidelity(C.byref(d), _stream(stream, p.device)))
    return out, seq_mean


def focus_gemm(a, b, out=None, a_rows=None, alpha: float = 1.0, out_dtype=torch.bfloat16, err=None,
               stream=None):
    """out[i] = alpha * a[a_rows[i] if a_rows is not None else i] @ b  (bf16 inputs,
    float32 accumulation).  a [rows, k], b [k, n] bf16 row-major (unit column
    stride); returns out [m, n] of out_dtype."""
    if a.dtype != torch.bfloat16 or b.dtype != torch.bfloat16 or a.dim() != 2 or b.dim() != 2:
        raise ValueError("a and b must be 2-D bfloat16 tensors")
    if a.stride(1) != 1 or b.stride(1) != 1 or a.shape[1] != b.shape[0]:
        raise ValueError("a [rows, k] and b [k, n] must be row-major with matching k")
    if a_rows is not None:
        a_rows = torch.as_tensor(a_rows, dtype=torch.int64).to(a.device).contiguous()
    m = a.shape[0] if a_rows is None else a_rows.numel()
    n = b.shape[1]
    if out is None:
        out = torch.empty(m, n, dtype=out_dtype, device=a.device)
    if tuple(out.shape) != (m, n) or out.stride(1) != 1:
        raise ValueError("out must be [m, n] row-major")
    d = GemmDesc()
    d.m, d.n, d.k = m, n, a.shape[1]
    d.a, d.lda, d.a_rows, d.a_nrows = _ptr_rows(a), a.stride(0), _ptr(a_rows), a.shape[0]
    d.b, d.ldb = _ptr_rows(b), b.stride(0)
    d.c, d.ldc, d.c_dtype = _ptr_rows(out), out.stride(0), _dtype(out)
    d.alpha = float(alpha)
    d.err = _ptr(err)
    check("focus_gemm", lib().focus_gemm(C.byref(d), _stream(stream, a.device)))
    return out


def focus_adapter_attn(lay: Layout, q_sum, k, v, cache_k=None, cache_v=None, o_sum=None, lse_sum=None,
                       win_ids=None, sum_base: int = 0, kv_tok_base: int = 0, mask: int = FOCUS_MASK_CT,
                       softmax_scale: float = 0.0, want_lse: bool = True, err=None, stream=None):
    """FOCUS adapter attention of the summary tokens: q_sum [rows, H, D] (row =
    global summary index - sum_base), k / v [rows, H_kv, D] (row = token -
    kv_tok_base), cache [batch, cap, H_kv, D].  Returns (o_sum, lse_sum)."""
    if o_sum is None:
        o_sum = torch.empty_like(q_sum)
    if lse_sum is None and want_lse:
        lse_sum = torch.empty(q_sum.shape[0], q_sum.shape[1], dtype=torch.float32, device=q_sum.device)
    if (o_sum.shape != q_sum.shape or q_sum.dtype != k.dtype or k.shape != v.shape
            or q_sum.shape[2] != k.shape[2]):
        raise ValueError("adapter attention shapes disagree")
    d = AdapterDesc()
    d.totals = lay.totals
    d.dtype = _dtype(q_sum)
    d.n_heads, d.head_dim = q_sum.shape[1], q_sum.shape[2]
    d.n_kv_heads = k.shape[1]
    d.softmax_scale, d.mask, d.batch = float(softmax_scale), int(mask), lay.batch
    d.kmer_uniform, d.win_kmer = int(lay.kmer_uniform), _ptr(lay.kmer)
    d.n_win = 0 if win_ids is None else win_ids.numel()
    d.win_ids = _ptr(win_ids)
    for f in ("win_seq", "win_ntok", "win_cache_off", "win_tok_off", "win_nsum", "win_sum_off", "sum_tok"):
        setattr(d, f, _ptr(lay[f]))
    d.q_sum, d.sum_base, d.sum_rows = _ptr(q_sum), int(sum_base), q_sum.shape[0]
    d.k, d.v, d.kv_tok_base, d.kv_rows = _ptr(k), _ptr(v), int(kv_tok_base), k.shape[0]
    if cache_k is not None:
        if cache_k.shape != cache_v.shape or cache_k.shape[2:] != k.shape[1:] or cache_k.dtype != k.dtype:
            raise ValueError("adapter cache shape/dtype does not match k")
        d.cache_k, d.cache_v, d.cache_cap = _ptr(cache_k), _ptr(cache_v), cache_k.shape[1]
    d.o_sum, d.lse_sum, d.err = _ptr(o_sum), _ptr(lse_sum), _ptr(err)
    check("focus_adapter_attn", lib().focus_adapter_attn(C.byref(d), _stream(stream, q_sum.device)))
    return o_sum, lse_sum


def _adapter_layer_desc(lay: Layout, hidden, w_q, w_k, w_v, w_o, n_heads, n_kv_heads, mask, softmax_scale,
                        out, workspace, err):
    d = AdapterLayerDesc()
    d.totals = lay.totals
    d.dtype = _dtype(hidden)
    d.n_heads, d.n_kv_heads = int(n_heads), int(n_kv_heads)
    d.d_model = hidden.shape[1]
    d.head_dim = w_q.shape[1] // int(n_heads)
    if (w_q.shape != (d.d_model, n_heads * d.head_dim) or w_k.shape != (d.d_model, n_kv_heads * d.head_dim)
            or w_v.shape != w_k.shape or w_o.shape != (n_heads * d.head_dim, d.d_model)
            or hidden.shape[0] != lay.totals.n_tokens):
        raise ValueError("adapter weight / hidden shapes disagree")
    d.softmax_scale, d.mask, d.batch = float(softmax_scale), int(mask), lay.batch
    d.kmer_uniform, d.win_kmer = int(lay.kmer_uniform), _ptr(lay.kmer)
    for f in ("win_seq", "win_ntok", "win_cache_off", "win_tok_off", "win_nsum", "win_sum_off", "sum_tok"):
        setattr(d, f, _ptr(lay[f]))
    d.hidden, d.w_q, d.w_k, d.w_v, d.w_o = _ptr(hidden), _ptr(w_q), _ptr(w_k), _ptr(w_v), _ptr(w_o)
    d.out = _ptr(out)
    d.workspace = _ptr(workspace)
    d.workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    d.err = _ptr(err)
    return d


def focus_adapter_layer_workspace(lay: Layout, hidden, w_q, w_k, w_v, w_o, n_heads: int, n_kv_heads: int,
                                  mask: int = FOCUS_MASK_CT) -> int:
    d = _adapter_layer_desc(lay, hidden, w_q, w_k, w_v, w_o, n_heads, n_kv_heads, mask, 0.0,
                            None, None, None)
    return lib().focus_adapter_layer_workspace(C.byref(d))


def focus_adapter_layer(lay: Layout, hidden, w_q, w_k, w_v, w_o, n_heads: int, n_kv_heads: int,
                        mask: int = FOCUS_MASK_CT, softmax_scale: float = 0.0, out=None, workspace=None,
                        err=None, stream=None):
    """FOCUS adapter update of the summary tokens (eq. focus-attn): returns
    out [n_summaries, d_model] in summary order."""
    if out is None:
        out = torch.empty(lay.totals.n_summaries, hidden.shape[1], dtype=hidden.dtype, device=hidden.device)
    if workspace is None:
        n = focus_adapter_layer_workspace(lay, hidden, w_q, w_k, w_v, w_o, n_heads, n_kv_heads, mask)
        workspace = _scratch(max(n, 256), hidden.device, stream)
    d = _adapter_layer_desc(lay, hidden, w_q, w_k, w_v, w_o, n_heads, n_kv_heads, mask, softmax_scale,
                            out, workspace, err)
    check("focus_adapter_layer", lib().focus_adapter_layer(C.byref(d), _stream(stream, hidden.device)))
    return out


def focus_qkv_project(lay: Layout, hidden, w_qkv, n_heads: int, n_kv_heads: int, rope_theta: float = 10000.0,
                      tok_base: int = 0, q=None, k=None, v=None, cache_k=None, cache_v=None, cache_len=None,
                      err=None, stream=None):
    """[Q | K | V] = hidden @ w_qkv with RoPE at the tokens' augmented-stream
    positions; summary K/V rows also written to the cache.  Returns (q, k, v)."""
    rows, d_model = hidden.shape
    D = w_qkv.shape[1] // (n_heads + 2 * n_kv_heads)
    if w_qkv.shape != (d_model, (n_heads + 2 * n_kv_heads) * D) or hidden.dtype != w_qkv.dtype:
        raise ValueError("w_qkv must be [d_model, (H + 2 H_kv) D] of hidden's dtype")
    mk = lambda h: torch.empty(rows, h, D, dtype=hidden.dtype, device=hidden.device)   # noqa: E731
    q = mk(n_heads) if q is None else q
    k = mk(n_kv_heads) if k is None else k
    v = mk(n_kv_heads) if v is None else v
    if q.shape != (rows, n_heads, D) or k.shape != (rows, n_kv_heads, D) or v.shape != k.shape:
        raise ValueError("q / k / v shapes")
    d = QkvDesc()
    d.totals = lay.totals
    d.dtype = _dtype(hidden)
    d.n_heads, d.n_kv_heads, d.head_dim, d.d_model, d.batch = int(n_heads), int(n_kv_heads), D, d_model, lay.batch
    d.rope_theta = float(rope_theta)
    for f in ("tok_pos", "tok_kind", "tok_kmer", "tok_win", "win_seq"):
        setattr(d, f, _ptr(lay[f]))
    d.tok_base, d.n_rows = int(tok_base), rows
    d.hidden, d.w_qkv, d.q, d.k, d.v = _ptr(hidden), _ptr(w_qkv), _ptr(q), _ptr(k), _ptr(v)
    if cache_k is not None:
        if cache_k.shape != cache_v.shape or cache_k.shape[2:] != (n_kv_heads, D):
            raise ValueError("cache shape")
        d.cache_k, d.cache_v, d.cache_cap = _ptr(cache_k), _ptr(cache_v), cache_k.shape[1]
    d.cache_len, d.err = _ptr(cache_len), _ptr(err)
    check("focus_qkv_project", lib().focus_qkv_project(C.byref(d), _stream(stream, hidden.device)))
    return q, k, v
