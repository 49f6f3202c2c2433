"""Oracle: FOCUS summary-token layout by literal insertion -- TEST INFRASTRUCTURE.

What is computed (Appendix A, window and B_w definitions; Section 3.2 "Setup and
tokens"):

* A sequence of L bases is cut into base-domain windows
  I_w = [(w-1)W+1, wW] intersected with [1, L]; there are ceil(L/W) of them.
* Inside window w, one summary (FOCUS) token is inserted after every k_w real
  bases, at the right boundary of its k-mer; a trailing partial k-mer still gets
  its summary, so window w holds B_w = ceil(|I_w| / k_w) summaries.  k_w = 0
  means no summaries at all (plain causal attention; the dense reading).
* After window w only its summaries' KV are kept; they are appended to the
  sequence's summary cache, so the cache rows window w can see are the
  C_w = B_1 + ... + B_{w-1} summaries of the earlier windows.  The boundary
  summary shared by consecutive windows is stored once, as the last cache row
  written by the earlier window.

The walk below builds the augmented token stream one base at a time and records
everything as it goes.  It is deliberately the slow, literal construction: no
closed form, no scan.

Indexing conventions (shared with the C interface, 0-based):
  global window index  windows of all sequences, sequence-major
  global token index   augmented tokens of all sequences, sequence-major
  global base index    bases of all sequences concatenated
  tok_pos              index of the token inside its own sequence's stream
  tok_kmer             cache row (inside its sequence) of the summary that
                       closes the token's k-mer; -1 when the window has k_w = 0
  tok_next_base        global base index of pi(t), the first real base after
                       token t in its sequence (Appendix A.1, eq. loss), or -1
"""

from __future__ import annotations

import numpy as np

BASE = 0
SUMMARY = 1


def _ceil_div(a: int, b: int) -> int:
    return -(-a // b)


def build_layout(seq_nt, window_nt: int, kmer, bases=None, summary_token_id: int = -1):
    """Walk every sequence and return the layout as a dict of NumPy arrays.

    seq_nt: per-sequence base counts.  kmer: one int for all windows, or one
    int per global window.  bases: optional uint8 codes of all bases
    (concatenated); when given, token_ids holds the byte of each base token and
    summary_token_id for each summary token.
    """
    seq_nt = [int(x) for x in seq_nt]
    W = int(window_nt)
    if W <= 0:
        raise ValueError("window_nt must be positive")
    if any(x < 0 for x in seq_nt):
        raise ValueError("negative sequence length")

    n_windows_total = sum(_ceil_div(L, W) if L > 0 else 0 for L in seq_nt)
    if np.ndim(kmer) == 0:
        kmer_of = [int(kmer)] * n_windows_total
    else:
        kmer_of = [int(x) for x in kmer]
        if len(kmer_of) != n_windows_total:
            raise ValueError("kmer must have one entry per window")
    if any(k < 0 for k in kmer_of):
        raise ValueError("negative cadence")

    cu_windows, cu_tokens, cu_summaries = [0], [0], [0]
    win = {name: [] for name in ("seq", "nt", "nsum", "ntok", "tok_off", "cache_off", "sum_off",
                                 "base_off")}
    tok = {name: [] for name in ("pos", "kind", "base", "kmer", "win")}
    token_ids = []
    sum_tok = []

    g_window = 0      # global window index
    g_token = 0       # global token index
    g_summary = 0     # global summary index
    g_base0 = 0       # global index of the sequence's first base

    for b, L in enumerate(seq_nt):
        cache_rows = 0    # summaries retained so far by this sequence
        pos = 0           # position inside this sequence's augmented stream
        start = 0
        while start < L:
            stop = min(start + W, L)
            k = kmer_of[g_window]
            win["seq"].append(b)
            win["nt"].append(stop - start)
            win["tok_off"].append(g_token)
            win["cache_off"].append(cache_rows)
            win["sum_off"].append(g_summary)
            win["base_off"].append(g_base0 + start)

            since_summary = 0   # bases of the currently open k-mer
            j = 0               # summaries emitted so far in this window

            def emit(kind, base_index, kmer_row):
                nonlocal g_token, pos
                tok["pos"].append(pos)
                tok["kind"].append(kind)
                tok["base"].append(base_index)
                tok["kmer"].append(kmer_row)
                tok["win"].append(g_window)
                if bases is not None:
                    token_ids.append(int(bases[base_index]) if kind == BASE else summary_token_id)
                pos += 1
                g_token += 1

            for i in range(start, stop):
                emit(BASE, g_base0 + i, cache_rows + j if k > 0 else -1)
                since_summary += 1
                closes_kmer = since_summary == k
                closes_window = i == stop - 1 and since_summary > 0
                if k > 0 and (closes_kmer or closes_window):
                    sum_tok.append(g_token)
                    emit(SUMMARY, -1, cache_rows + j)
                    j += 1
                    since_summary = 0

            win["nsum"].append(j)
            win["ntok"].append((stop - start) + j)
            cache_rows += j
            g_summary += j
            g_window += 1
            start = stop
        g_base0 += L
        cu_windows.append(g_window)
        cu_tokens.append(g_token)
        cu_summaries.append(g_summary)

    # Target map of the training objective (Appendix A.1, eq. loss): for every
    # position t, pi(t) is the first real-base position after t; recorded as
    # that base's global index, -1 when t is past its sequence's last base.
    next_base = [-1] * g_token
    for b in range(len(seq_nt)):
        nxt = -1
        for t in range(cu_tokens[b + 1] - 1, cu_tokens[b] - 1, -1):
            next_base[t] = nxt
            if tok["kind"][t] == BASE:
                nxt = tok["base"][t]

    i32, i64 = np.int32, np.int64
    out = {
        "n_windows": g_window,
        "n_tokens": g_token,
        "n_summaries": g_summary,
        "cu_windows": np.asarray(cu_windows, i64),
        "cu_tokens": np.asarray(cu_tokens, i64),
        "cu_summaries": np.asarray(cu_summaries, i64),
        "win_seq": np.asarray(win["seq"], i32),
        "win_nt": np.asarray(win["nt"], i32),
        "win_nsum": np.asarray(win["nsum"], i32),
        "win_ntok": np.asarray(win["ntok"], i32),
        "win_tok_off": np.asarray(win["tok_off"], i64),
        "win_cache_off": np.asarray(win["cache_off"], i32),
        "win_sum_off": np.asarray(win["sum_off"], i64),
        "win_base_off": np.asarray(win["base_off"], i64),
        "tok_pos": np.asarray(tok["pos"], i32),
        "tok_kind": np.asarray(tok["kind"], np.uint8),
        "tok_base": np.asarray(tok["base"], i64),
        "tok_kmer": np.asarray(tok["kmer"], i32),
        "tok_win": np.asarray(tok["win"], i32),
        "tok_next_base": np.asarray(next_base, i64),
        "sum_tok": np.asarray(sum_tok, i64),
        "window_kmer": np.asarray(kmer_of, i32),
    }
    if bases is not None:
        out["token_ids"] = np.asarray(token_ids, i32)
    return out


def token_string(layout, b: int, summary_char: str = "S", sep: str = "|") -> str:
    """Human-readable augmented stream of sequence b: 'b' per base, summary_char
    per summary, sep between windows (used by the worked-example fixtures)."""
    parts = []
    lo, hi = layout["cu_windows"][b], layout["cu_windows"][b + 1]
    for w in range(lo, hi):
        t0 = layout["win_tok_off"][w]
        kinds = layout["tok_kind"][t0:t0 + layout["win_ntok"][w]]
        parts.append("".join(summary_char if x == SUMMARY else "b" for x in kinds))
    return sep.join(parts)
