"""The pins must catch plausible mistakes in the oracle.

Each case plants one mistake in a copy of an oracle module's source (an
off-by-one in the causal mask, a dropped cache row, a dropped scale, a summary on
the wrong side of its k-mer, a missing partial-k-mer summary, ...), loads the
copy in place of the real module, and checks that at least one pin test fails.
Everything runs on the CPU.
"""

import importlib.util
import os
import sys

import pytest

import oracle.adapter
import oracle.attention
import oracle.decode
import oracle.fidelity
import oracle.projection
import oracle.layout
import test_oracle_adapter as TAD
import test_oracle_attention as TA
import test_oracle_decode as TD
import test_oracle_fidelity as TF
import test_oracle_kmer_local as TK
import test_oracle_projection as TP
import test_oracle_layout as TL

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _mutant(module, old, new):
    path = module.__file__
    src = open(path).read()
    assert src.count(old) == 1, f"mutation anchor not unique in {path}: {old!r}"
    spec = importlib.util.spec_from_loader(module.__name__ + "_mutant", loader=None,
                                           origin=path)
    mod = importlib.util.module_from_spec(spec)
    mod.__package__ = "oracle"
    exec(compile(src.replace(old, new), path, "exec"), mod.__dict__)
    return mod


def _layout_pins():
    for case in TL._golden_cases():
        TL.test_worked_examples(*case)
    for seed in range(10):
        TL.test_appendix_a_closed_forms(seed)
        TL.test_kmer_membership_and_positions(seed)
        TL.test_literal_string_insertion(seed)
    for case in TL._next_base_cases():
        TL.test_next_base_worked_examples(*case)
    for seed in range(6):
        TL.test_next_base_brute_force(seed)


def _attention_pins():
    for seed in range(3):
        TA.test_zero_summaries_one_window_is_dense_causal(seed)
        TA.test_zero_keys_give_mean_of_visible_values_one_hot(seed)
        TA.test_sequential_equals_masked_parallel(seed)
    TA.test_window_attention_matches_brute_force_with_cache()
    TA.test_rows_sum_to_one_and_respect_mask()
    TA.test_constant_values_and_first_token()
    TA.test_discarded_ordinary_kv_is_invisible_but_summaries_are_not()
    TA.test_strict_causality()
    TA.test_grouped_kv_heads_equal_repeated_heads()
    TA.test_scale_enters_only_through_scores()
    TA.test_compaction_keeps_summary_rows_in_order(0)


def _kmer_local_pins():
    for seed in range(4):
        TK.test_stream_form_equals_window_form(seed)
        TK.test_zero_keys_one_hot_values_spell_out_the_visible_set(seed)
        TK.test_earlier_rows_and_other_kmer_bases_are_invisible(seed)
        TK.test_first_kmer_is_textbook_causal(seed)
        TK.test_one_kmer_per_window_is_causal_plus_boundary(seed)
    TK.test_zero_kmer_single_window_is_dense_causal()


def _fidelity_pins():
    for V in (2, 4, 17):
        TF.test_against_library_routines(V)
        TF.test_point_mass_against_uniform(V)
    TF.test_hellinger_forms_agree()
    TF.test_identical_inputs_are_zero()
    TF.test_point_masses_closed_forms()
    TF.test_bounds_and_symmetry()
    TF.test_softmax_and_clipping()
    TF.test_sequence_means()


def _adapter_pins():
    for seed in range(3):
        for mask in ("ct", "kmer_local"):
            TAD.test_summary_rows_of_the_main_attention(mask, seed)
        TAD.test_zero_keys_one_hot_values_count_the_visible_set(seed)
    TAD.test_identity_projections_give_the_attention()
    TAD.test_linear_in_output_and_value_weights()
    TAD.test_grouped_kv_heads_equal_repeated_heads()
    for mask in ("ct", "kmer_local"):
        TAD.test_causality_and_windows_without_summaries(mask)


def _projection_pins():
    TP.test_norm_and_identity()
    TP.test_two_dims_angle_is_the_position()
    for shift in (1, 100):
        TP.test_relative_positions(shift)
    TP.test_projection_without_rotation_and_positions()
    TP.test_store_bf16_matches_torch()
    TP.test_second_pair_frequency()
    TP.test_projection_rotates_at_the_stream_position()


def _decode_pins():
    TD.test_decode_from_empty_equals_prefill(37, 10, 3)
    TD.test_decode_from_empty_equals_prefill(25, 7, 7)
    TD.test_decode_mid_window_start_equals_prefill(11)
    TD.test_cache_growth_and_window_reset()
    for seed in range(4):
        TD.test_per_window_cadence_equals_prefill(seed)


ATTENTION_MUTATIONS = [
    ("strict causal mask", "((j - n_cache) <= i)", "((j - n_cache) < i)"),
    ("last cache row hidden", "return (j < n_cache) | ((j - n_cache) <= i)",
     "return (j < n_cache - 1) | ((j >= n_cache) & ((j - n_cache) <= i))"),
    ("window sees its future", "((j - n_cache) <= i)", "((j - n_cache) <= i + 1)"),
    ("scale dropped", "s = scale * (q @ keys.T)", "s = (q @ keys.T)"),
    ("no max shift in lse", "lse = (m + np.log(l))[:, 0]", "lse = np.log(l)[:, 0]"),
    ("values of the wrong rows", "o = p @ values", "o = p @ values[::-1]"),
    ("kv head of the wrong group",
     "vis = window_visibility(T, C)\n    o = np.empty((T, H, D), np.float64)\n    lse = np.empty((T, H), np.float64)\n"
     "    for h in range(H):\n        g = h // (H // Hkv)",
     "vis = window_visibility(T, C)\n    o = np.empty((T, H, D), np.float64)\n    lse = np.empty((T, H), np.float64)\n"
     "    for h in range(H):\n        g = h % Hkv"),
    ("ordinary rows kept", "keep = np.nonzero(layout[\"tok_kind\"][t0:t1] == SUMMARY)[0] + t0",
     "keep = np.arange(t0, t1)"),
    ("masked-parallel without summaries", "((win[None, :] == win[:, None]) | is_sum[None, :])",
     "((win[None, :] == win[:, None]))"),
    ("cache offset off by one", "first:first + int(layout[\"win_cache_off\"][w])]",
     "first:first + int(layout[\"win_cache_off\"][w]) + 1]"),
]

LAYOUT_MUTATIONS = [
    ("summary before its k-mer", "closes_kmer = since_summary == k", "closes_kmer = since_summary == 1"),
    ("partial k-mer without summary", "closes_window = i == stop - 1 and since_summary > 0",
     "closes_window = False"),
    ("cache rows not carried", "cache_rows += j\n", "cache_rows += 0\n"),
    ("window one base short", "stop = min(start + W, L)", "stop = min(start + W - 1, L)"),
    ("kmer row of next summary", "emit(BASE, g_base0 + i, cache_rows + j if k > 0 else -1)",
     "emit(BASE, g_base0 + i, cache_rows + j + 1 if k > 0 else -1)"),
    ("target is the token itself", "            next_base[t] = nxt\n            if tok[\"kind\"][t] == BASE:",
     "            if tok[\"kind\"][t] == BASE:\n                next_base[t] = tok[\"base\"][t]\n            if tok[\"kind\"][t] == BASE:"),
    ("target carried across sequences", "    for b in range(len(seq_nt)):\n        nxt = -1\n",
     "    nxt = -1\n    for b in range(len(seq_nt)):\n"),
]

DECODE_MUTATIONS = [
    ("no summary for partial window", "(self.bases_in_window == W and self.bases_in_kmer > 0)", "False"),
    ("window never reset", "self.win_k, self.win_v = [], []", "pass"),
    ("summary into window buffer", "self.cache_k.append(np.asarray(k_new))",
     "self.win_k.append(np.asarray(k_new))"),
    ("cadence never switches", "            self.win_index += 1\n", "            pass\n"),
]


KMER_LOCAL_MUTATIONS = [
    ("boundary row dropped", "        vis[:, C - 1] = True\n", "        vis[:, C - 1] = False\n"),
    ("every earlier summary visible", "            elif u == boundary:", "            elif is_sum[u]:"),
    ("boundary from the first window", "                boundary = u\n",
     "                boundary = u if boundary < 0 else boundary\n"),
    ("token does not see itself", "vis[:, C:] = (u <= i) & (", "vis[:, C:] = (u < i) & ("),
    ("bases of earlier k-mers visible", "((kmer[None, :] == kmer[:, None]) | is_sum[None, :])",
     "((kmer[None, :] <= kmer[:, None]) | is_sum[None, :])"),
    ("later summaries visible", "vis[:, C:] = (u <= i) & (", "vis[:, C:] = (u >= 0) & ("),
]


FIDELITY_MUTATIONS = [
    ("no renormalisation after the clip", "return p / p.sum(axis=-1, keepdims=True)", "return p"),
    ("L2 without the root", "l2 = np.sqrt((d * d).sum(axis=-1))", "l2 = (d * d).sum(axis=-1)"),
    ("Hellinger without 1/sqrt 2", " / np.sqrt(2.0)", ""),
    ("JS against one side only", "js = 0.5 * kl(p, m) + 0.5 * kl(q, m)", "js = kl(p, m)"),
    ("KL reversed", "kl(p, q)], axis=-1)", "kl(q, p)], axis=-1)"),
    ("log base 2", "np.log(a / b)", "np.log2(a / b)"),
    ("softmax over the wrong axis", "e / e.sum(axis=-1, keepdims=True)", "e / e.sum(axis=0, keepdims=True)"),
    ("clip above instead of below", "np.maximum(np.asarray(p, np.float64), CLIP)",
     "np.minimum(np.asarray(p, np.float64), 1 - CLIP)"),
]


ADAPTER_MUTATIONS = [
    ("summary rows shifted", 'rows = layout["sum_tok"][s0:s0 + B] - t0', 'rows = layout["sum_tok"][s0:s0 + B] - t0 - 1'),
    ("no output projection", "return st(o.reshape(n_sum, n_heads * D)) @ w_o",
     "return st(o.reshape(n_sum, n_heads * D))"),
    ("queries of the wrong tokens", 'for s in sums]] @ w_q)', 'for s in sums][::-1]] @ w_q)'),
    ("k-mer-local rule ignored", 'if mask == "kmer_local":\n        return A.kmer_local_window_visibility(layout, w)',
     'if mask == "kmer_local":\n        return A.window_visibility(int(layout["win_ntok"][w]), int(layout["win_cache_off"][w]))'),
]


PROJECTION_MUTATIONS = [
    ("rotation the wrong way", "out[..., 1::2] = e * s + o * c", "out[..., 1::2] = -e * s + o * c"),
    ("frequency exponent without the 2", "theta ** (-2.0 * i / D)", "theta ** (-1.0 * i / D)"),
    ("value heads from the key columns", "v = y[:, (n_heads + n_kv_heads) * D:]",
     "v = y[:, n_heads * D:(n_heads + 2 * n_kv_heads) * D][:, :n_kv_heads * D]"),
    ("positions off by one", 'pos = layout["tok_pos"][rows]', 'pos = layout["tok_pos"][rows] + 1'),
]


def _expect_caught(monkeypatch, pins, patches):
    for mod_obj, attr, value in patches:
        monkeypatch.setattr(mod_obj, attr, value)
    with pytest.raises((AssertionError, ValueError, IndexError)):
        pins()


@pytest.mark.parametrize("name,old,new", ATTENTION_MUTATIONS, ids=[m[0] for m in ATTENTION_MUTATIONS])
def test_attention_mutations_are_caught(monkeypatch, name, old, new):
    mut = _mutant(oracle.attention, old, new)
    _expect_caught(monkeypatch, _attention_pins, [(TA, "A", mut)])


@pytest.mark.parametrize("name,old,new", LAYOUT_MUTATIONS, ids=[m[0] for m in LAYOUT_MUTATIONS])
def test_layout_mutations_are_caught(monkeypatch, name, old, new):
    mut = _mutant(oracle.layout, old, new)
    _expect_caught(monkeypatch, _layout_pins, [(TL, "build_layout", mut.build_layout)])


@pytest.mark.parametrize("name,old,new", DECODE_MUTATIONS, ids=[m[0] for m in DECODE_MUTATIONS])
def test_decode_mutations_are_caught(monkeypatch, name, old, new):
    mut = _mutant(oracle.decode, old, new)
    _expect_caught(monkeypatch, _decode_pins, [(TD, "DecodeSequence", mut.DecodeSequence)])


@pytest.mark.parametrize("name,old,new", KMER_LOCAL_MUTATIONS, ids=[m[0] for m in KMER_LOCAL_MUTATIONS])
def test_kmer_local_mutations_are_caught(monkeypatch, name, old, new):
    mut = _mutant(oracle.attention, old, new)
    _expect_caught(monkeypatch, _kmer_local_pins, [(TK, "A", mut)])


@pytest.mark.parametrize("name,old,new", FIDELITY_MUTATIONS, ids=[m[0] for m in FIDELITY_MUTATIONS])
def test_fidelity_mutations_are_caught(monkeypatch, name, old, new):
    mut = _mutant(oracle.fidelity, old, new)
    _expect_caught(monkeypatch, _fidelity_pins, [(TF, "FD", mut)])


@pytest.mark.parametrize("name,old,new", ADAPTER_MUTATIONS, ids=[m[0] for m in ADAPTER_MUTATIONS])
def test_adapter_mutations_are_caught(monkeypatch, name, old, new):
    mut = _mutant(oracle.adapter, old, new)
    _expect_caught(monkeypatch, _adapter_pins, [(TAD, "AD", mut)])


@pytest.mark.parametrize("name,old,new", PROJECTION_MUTATIONS, ids=[m[0] for m in PROJECTION_MUTATIONS])
def test_projection_mutations_are_caught(monkeypatch, name, old, new):
    mut = _mutant(oracle.projection, old, new)
    _expect_caught(monkeypatch, _projection_pins, [(TP, "P", mut)])


def test_unmutated_pins_pass():
    _projection_pins()
    _adapter_pins()
    _fidelity_pins()
    _layout_pins()
    _attention_pins()
    _decode_pins()
    _kmer_local_pins()
