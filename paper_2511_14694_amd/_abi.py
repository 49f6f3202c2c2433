"""ctypes mirror of include/focus.h.  Loads libfocus.so; no fallback."""

from __future__ import annotations

import ctypes as C
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfocus.so")

FOCUS_OK = 0
STATUS_NAMES = {0: "FOCUS_OK", 1: "FOCUS_E_NULL", 2: "FOCUS_E_ARG", 3: "FOCUS_E_SHAPE",
                4: "FOCUS_E_DTYPE", 5: "FOCUS_E_UNSUPPORTED", 6: "FOCUS_E_WORKSPACE",
                7: "FOCUS_E_CAPACITY", 8: "FOCUS_E_HIP"}
FOCUS_BF16, FOCUS_F32 = 0, 1
FOCUS_MASK_CT, FOCUS_MASK_KMER_LOCAL = 0, 1
FOCUS_TOK_BASE, FOCUS_TOK_SUMMARY = 0, 1
FOCUS_STEP_SUMMARY, FOCUS_STEP_WINDOW_END = 1, 2
FOCUS_ERR_CAPACITY, FOCUS_ERR_BOUNDS, FOCUS_ERR_PLAN = 1, 2, 4
FOCUS_FID_LOGITS, FOCUS_FID_PROBS = 0, 1
FOCUS_FID_N = 5

p = C.c_void_p
i32, i64, f32, sz = C.c_int32, C.c_int64, C.c_float, C.c_size_t


class LayoutTotals(C.Structure):
    _fields_ = [("n_windows", i64), ("n_tokens", i64), ("n_summaries", i64),
                ("max_window_tokens", i64), ("max_window_summaries", i64),
                ("max_cache_per_seq", i64), ("max_window_cache", i64)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class LayoutDesc(C.Structure):
    _fields_ = [("totals", LayoutTotals), ("batch", i32), ("window_nt", i32),
                ("kmer_uniform", i32), ("summary_token_id", i32),
                ("seq_nt", p), ("kmer", p), ("bases", p),
                ("cu_windows", p), ("cu_tokens", p), ("cu_summaries", p),
                ("win_seq", p), ("win_nt", p), ("win_nsum", p), ("win_ntok", p),
                ("win_cache_off", p), ("win_tok_off", p), ("win_sum_off", p), ("win_base_off", p),
                ("tok_pos", p), ("tok_kmer", p), ("tok_win", p), ("tok_kind", p), ("tok_base", p),
                ("sum_tok", p), ("token_ids", p), ("tok_next_base", p), ("err", p)]


class CompactDesc(C.Structure):
    _fields_ = [("totals", LayoutTotals), ("dtype", i32), ("n_kv_heads", i32), ("head_dim", i32),
                ("batch", i32), ("n_win", i64), ("win_ids", p),
                ("win_seq", p), ("win_nsum", p), ("win_cache_off", p), ("win_sum_off", p),
                ("sum_tok", p), ("k", p), ("v", p), ("kv_tok_base", i64), ("kv_rows", i64),
                ("cache_k", p), ("cache_v", p), ("cache_cap", i64), ("cache_len", p), ("err", p)]


class AttnDesc(C.Structure):
    _fields_ = [("totals", LayoutTotals), ("dtype", i32), ("n_heads", i32), ("n_kv_heads", i32),
                ("head_dim", i32), ("softmax_scale", f32), ("mask", i32), ("batch", i32),
                ("kmer_uniform", i32), ("n_win", i64), ("win_ids", p),
                ("win_seq", p), ("win_ntok", p), ("win_cache_off", p), ("win_tok_off", p),
                ("win_kmer", p),
                ("q", p), ("k", p), ("v", p), ("qkv_tok_base", i64), ("qkv_rows", i64),
                ("cache_k", p), ("cache_v", p), ("cache_cap", i64), ("o", p), ("lse", p),
                ("workspace", p), ("workspace_bytes", sz), ("err", p)]


class DecodeDesc(C.Structure):
    _fields_ = [("dtype", i32), ("batch", i32), ("n_heads", i32), ("n_kv_heads", i32),
                ("head_dim", i32), ("softmax_scale", f32), ("split_keys", i32), ("reserved", i32),
                ("q", p), ("k_new", p), ("v_new", p), ("kind", p),
                ("cache_k", p), ("cache_v", p), ("cache_cap", i64), ("cache_len", p),
                ("win_k", p), ("win_v", p), ("win_cap", i64), ("win_len", p),
                ("o", p), ("lse", p), ("workspace", p), ("workspace_bytes", sz), ("err", p)]


class DecodeSched(C.Structure):
    _fields_ = [("batch", i32), ("window_nt", i32), ("kmer_uniform", i32), ("kmer_stride", i32),
                ("kmer", p), ("win_index", p), ("bases_in_window", p), ("bases_in_kmer", p),
                ("kind", p), ("tokens", p), ("summaries", p), ("err", p)]


class FidelityDesc(C.Structure):
    _fields_ = [("dtype", i32), ("input_kind", i32), ("n_pos", i64), ("vocab", i32), ("n_seq", i32),
                ("p", p), ("q", p), ("out", p), ("cu_pos", p), ("seq_mean", p), ("err", p)]


class GemmDesc(C.Structure):
    _fields_ = [("m", i64), ("n", i64), ("k", i64), ("a", p), ("lda", i64), ("a_rows", p),
                ("a_nrows", i64), ("b", p), ("ldb", i64), ("c", p), ("ldc", i64), ("c_dtype", i32),
                ("alpha", f32), ("err", p)]


class AdapterDesc(C.Structure):
    _fields_ = [("totals", LayoutTotals), ("dtype", i32), ("n_heads", i32), ("n_kv_heads", i32),
                ("head_dim", i32), ("softmax_scale", f32), ("mask", i32), ("batch", i32),
                ("kmer_uniform", i32), ("n_win", i64), ("win_ids", p),
                ("win_seq", p), ("win_ntok", p), ("win_cache_off", p), ("win_tok_off", p),
                ("win_kmer", p), ("win_nsum", p), ("win_sum_off", p), ("sum_tok", p),
                ("q_sum", p), ("sum_base", i64), ("sum_rows", i64),
                ("k", p), ("v", p), ("kv_tok_base", i64), ("kv_rows", i64),
                ("cache_k", p), ("cache_v", p), ("cache_cap", i64), ("o_sum", p), ("lse_sum", p),
                ("err", p)]


class AdapterLayerDesc(C.Structure):
    _fields_ = [("totals", LayoutTotals), ("dtype", i32), ("n_heads", i32), ("n_kv_heads", i32),
                ("head_dim", i32), ("d_model", i32), ("softmax_scale", f32), ("mask", i32), ("batch", i32),
                ("kmer_uniform", i32), ("reserved", i32),
                ("win_seq", p), ("win_ntok", p), ("win_cache_off", p), ("win_tok_off", p), ("win_kmer", p),
                ("win_nsum", p), ("win_sum_off", p), ("sum_tok", p),
                ("hidden", p), ("w_q", p), ("w_k", p), ("w_v", p), ("w_o", p), ("out", p),
                ("workspace", p), ("workspace_bytes", sz), ("err", p)]


class QkvDesc(C.Structure):
    _fields_ = [("totals", LayoutTotals), ("dtype", i32), ("n_heads", i32), ("n_kv_heads", i32),
                ("head_dim", i32), ("d_model", i32), ("batch", i32), ("rope_theta", f32), ("reserved", i32),
                ("tok_pos", p), ("tok_kind", p), ("tok_kmer", p), ("tok_win", p), ("win_seq", p),
                ("tok_base", i64), ("n_rows", i64), ("hidden", p), ("w_qkv", p),
                ("q", p), ("k", p), ("v", p), ("cache_k", p), ("cache_v", p), ("cache_cap", i64),
                ("cache_len", p), ("err", p)]


STRUCTS = [LayoutTotals, LayoutDesc, CompactDesc, AttnDesc, DecodeDesc, FidelityDesc, GemmDesc, AdapterDesc,
           AdapterLayerDesc, QkvDesc, DecodeSched]

# name -> (restype, argtypes): every symbol include/focus.h declares
SYMBOLS = {
    "focus_abi_version": (i32, []),
    "focus_status_str": (C.c_char_p, [i32]),
    "focus_struct_size": (i64, [i32]),
    "focus_layout_plan": (i32, [i32, p, i32, p, i32, C.POINTER(LayoutTotals)]),
    "focus_layout": (i32, [C.POINTER(LayoutDesc), p]),
    "focus_compact_kv": (i32, [C.POINTER(CompactDesc), p]),
    "focus_window_attn_workspace": (sz, [C.POINTER(AttnDesc)]),
    "focus_window_attn": (i32, [C.POINTER(AttnDesc), p]),
    "focus_decode_workspace": (sz, [C.POINTER(DecodeDesc)]),
    "focus_decode_step": (i32, [C.POINTER(DecodeDesc), p]),
    "focus_decode_step_noalloc": (i32, [C.POINTER(DecodeDesc), p]),
    "focus_decode_sched_start": (i32, [C.POINTER(DecodeSched), p]),
    "focus_decode_next_kind": (i32, [C.POINTER(DecodeSched), p]),
    "focus_fidelity": (i32, [C.POINTER(FidelityDesc), p]),
    "focus_gemm": (i32, [C.POINTER(GemmDesc), p]),
    "focus_adapter_attn": (i32, [C.POINTER(AdapterDesc), p]),
    "focus_adapter_layer_workspace": (sz, [C.POINTER(AdapterLayerDesc)]),
    "focus_adapter_layer": (i32, [C.POINTER(AdapterLayerDesc), p]),
    "focus_qkv_project": (i32, [C.POINTER(QkvDesc), p]),
}


class FocusError(RuntimeError):
    def __init__(self, call: str, status: int, text: str):
        super().__init__(f"{call} failed: {STATUS_NAMES.get(status, status)} ({text})")
        self.status = status


_lib = None


def lib():
    """The loaded libfocus.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2511_14694_amd.build` (or __graft_entry__.build())")
        handle = C.CDLL(LIB_PATH)
        for name, (res, args) in SYMBOLS.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        for i, st in enumerate(STRUCTS):
            if handle.focus_struct_size(i) != C.sizeof(st):
                raise ImportError(f"struct {st.__name__} mirror has size {C.sizeof(st)}, "
                                  f"library says {handle.focus_struct_size(i)}")
        _lib = handle
    return _lib


def check(call: str, status: int):
    if status != FOCUS_OK:
        raise FocusError(call, status, lib().focus_status_str(status).decode())
