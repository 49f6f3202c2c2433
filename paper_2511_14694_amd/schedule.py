"""Host side of streaming decode: which kind of token each step appends.

The kinds are read off one window of the device layout (tok_kind of a full
window, as focus_layout writes it): decoding walks the augmented stream of
consecutive identical windows, starting `start` tokens into the current one.
"""

from __future__ import annotations

import numpy as np

from ._abi import FOCUS_STEP_SUMMARY, FOCUS_STEP_WINDOW_END, FOCUS_TOK_SUMMARY


def initial_lengths(window_kinds: np.ndarray, start: int):
    """(summaries, bases) among the first `start` tokens of the window."""
    head = np.asarray(window_kinds[:start])
    n_sum = int((head == FOCUS_TOK_SUMMARY).sum())
    return n_sum, int(start - n_sum)


def step_kinds(window_kinds: np.ndarray, start: int, steps: int) -> np.ndarray:
    """focus_decode_step kind bits (uint8 [steps]) for tokens start, start+1, ..."""
    kinds = np.asarray(window_kinds)
    T = len(kinds)
    pos = (start + np.arange(steps)) % T
    out = np.where(kinds[pos] == FOCUS_TOK_SUMMARY, FOCUS_STEP_SUMMARY, 0)
    out = out | np.where(pos == T - 1, FOCUS_STEP_WINDOW_END, 0)
    return out.astype(np.uint8)
