"""Planted mistakes in the oracle (on the CPU) must each fail at least one pin.

Every mutant is a textual edit of a temporary copy of ``oracle/dv_oracle.c``
(the oracle's own source is never changed), compiled with gcc and loaded in
place of the real oracle; the pins of ``test_oracle_pins`` then run against
it.  A mutant that no pin catches would mean a plausible mistake of that kind
could hide in the oracle.
"""
import os
import subprocess

import numpy as np
import pytest

import oracle
import workloads as W
from tests import test_oracle_pins as P

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle",
                   "dv_oracle.c")

MUTANTS = {
    "bit order msb-first": ("(uint32_t)1u << (t % 32)", "(uint32_t)0x80000000u >> (t % 32)"),
    "ties to highest index": ("v > best_v", "v >= best_v"),
    "nan not ranked as -inf": ("v = -INFINITY;", "v = v;"),
    "last state read as dead": ("x < num_states)", "x < num_states - 1)"),
    "bytes walked in reverse": ("str[i]], num_states", "str[len - 1 - i]], num_states"),
    "first byte skipped": ("for (int64_t i = 0; i < len; ++i)", "for (int64_t i = 1; i < len; ++i)"),
    "bf16 widened wrongly": ("<< 16;", "<< 15;"),
    "new state from wrong column": ("next_state[(int64_t)s * num_tokens + tok]",
                                    "next_state[(int64_t)s * num_tokens]"),
    "leading dimension ignored": ("(size_t)ld_logits", "(size_t)num_tokens"),
    "stale allow word kept": ("memset(al_row, 0,", "(void)(al_row + 0,"),
    "dead walk continues from state 0": ("return ORACLE_DEAD;\n        st =", "st = 0;\n        st ="),
    "eos allowed in every state": ("accepting != NULL && accepting[cs]", "accepting != NULL"),
    "eos moves to the start state": ("accepting[cs]) ? cs : ORACLE_DEAD", "accepting[cs]) ? 0 : ORACLE_DEAD"),
    "spec compares with the next proposal": ("tok != prop[j])", "tok != prop[j + (j + 1 < num_proposed)])"),
    "spec keeps the state after an illegal proposal": ("else\n                    st = ORACLE_DEAD;",
                                                       "else\n                    st = st;"),
    "spec matches a -1 choice with a -1 proposal": ("tok == -1 || tok != prop[j]", "tok != prop[j]"),
    "spec walk ignores the allow bit": ("return (int)((allow[", "return 1 | (int)((allow["),
    "spec walk does not advance": ("fin = next_state[(int64_t)st * num_tokens + prop[a]];", "fin = st;"),
    "spec new state from the row's start state": (
        "ns = tok == -1 ? ORACLE_DEAD : next_state[(int64_t)st * num_tokens + tok];",
        "ns = tok == -1 ? ORACLE_DEAD : next_state[(int64_t)oracle_canon(states[b], num_states) * num_tokens + tok];"),
    "spec position stride ignored": ("j * ld_pos", "j * (int64_t)num_tokens"),
    "spec stops one position late": ("a = j;\n", "a = j + (j < num_proposed);\n"),
    "opportunistic skips the check": ("tok = ok ? free_tok :", "tok = 1 ? free_tok :"),
    "opportunistic free ties to highest": ("if (i == 0 || v > best_v)", "if (i == 0 || v >= best_v)"),
    "opportunistic free keeps nan": ("v = -INFINITY;\n                if (i == 0", "v = v;\n                if (i == 0"),
    "sample noise sign flipped": ("fmaf(x, inv_temperature, oracle_gumbel(", "fmaf(x, inv_temperature, -oracle_gumbel("),
    "sample temperature ignored": ("float key = fmaf(x, inv_temperature,", "float key = fmaf(x, 1.0f,"),
    "sample takes the next philox word": ("uint32_t w = out[token % 4u];", "uint32_t w = out[(token + 1u) % 4u];"),
    "sample counter fields swapped": ("{token / 4u, row, (uint32_t)offset,", "{row, token / 4u, (uint32_t)offset,"),
    "ln without the exponent": ("return fmaf((float)e, 0x1.62e430p-1f, lnm);", "return lnm;"),
    "philox key not bumped": ("k1 += 0xBB67AE85u;", "k1 += 0u;"),
    "sample ignores the mask": ("            for (int32_t i = 0; i < num_tokens; ++i) {\n                if (((arow[i / 32] >> (i % 32)) & 1u) == 0)\n                    continue;\n                float x",
                                "            for (int32_t i = 0; i < num_tokens; ++i) {\n                float x"),
    "zero-length token dies": ("int32_t st = oracle_canon(s, num_states);\n    for",
                               "int32_t st = len ? oracle_canon(s, num_states) : ORACLE_DEAD;\n    for"),
}


def _checks(lib):
    """The pins, run against ``lib``; returns the names of those that failed."""
    trans, _ = W.dfa(1)
    offsets, data = W.vocab(1)
    try:
        ns, al = oracle.align(trans, offsets, data, lib=lib)
    except Exception:
        return ["align raised"]
    table = (trans, offsets, data, ns, al)
    checks = [
        ("monoid", lambda: [P.test_align_matches_transition_monoid(s, lib) for s in range(6)]),
        ("rows", lambda: P.test_align_rows_equals_full_table(lib)),
        ("fig_nfa", lambda: P.test_fig_nfa_int_rows(lib)),
        ("fig_overview", lambda: P.test_fig_overview_subterminal_landing(lib)),
        ("single_byte", lambda: P.test_single_byte_rows_equal_transition_row(table)),
        ("allow_iff", lambda: P.test_allow_bit_iff_alive_and_padding_zero(table)),
        ("concat", lambda: P.test_concatenation_homomorphism(table, lib)),
        ("dead_row", lambda: P.test_dead_row_is_empty(table, lib)),
        ("emitted", lambda: P.test_emitted_token_is_allowed_and_state_follows_walk(table, lib)),
        ("numpy_f32", lambda: P.test_masked_step_equals_numpy_argmax("f32", table, lib)),
        ("numpy_bf16", lambda: P.test_masked_step_equals_numpy_argmax("bf16", table, lib)),
        ("one_state", lambda: P.test_single_accepting_state_is_unconstrained_argmax(lib)),
        ("ld", lambda: P.test_leading_dimension_and_row_independence(table, lib)),
        ("ties_f32", lambda: [P.test_planted_ties_and_specials_f32(v, a, e, lib)
                              for v, a, e in [([100, 9, 9, 5], [1, 2], 1),
                                              ([5, float("nan"), 3, 3, -np.inf], [1, 4], 1),
                                              ([float("nan"), 2.0, 1.0], [0, 1, 2], 1)]]),
        ("eos_fig_nfa", lambda: P.test_fig_nfa_eos_column(lib)),
        ("eos_invariants", lambda: P.test_eos_column_invariants(table, lib)),
        ("spec_fig_nfa", lambda: P.test_fig_nfa_spec_walk_and_verify(lib)),
        ("spec_sequential", lambda: [P.test_spec_verify_equals_sequential_greedy(d, l, table, lib)
                                     for d, l in [("f32", "rows"), ("bf16", "rows"), ("f32", "steps")]]),
        ("spec_later", lambda: P.test_spec_verify_later_positions_follow_the_proposals(table, lib)),
        ("spec_bytes", lambda: P.test_spec_walk_matches_byte_walk(table, lib)),
        ("spec_legal", lambda: P.test_spec_verify_accepts_only_legal_prefixes(table, lib)),
        ("spec_zero", lambda: P.test_spec_zero_proposals_is_one_masked_step(table, lib)),
        ("spec_perfect", lambda: P.test_spec_perfect_draft_is_fully_accepted(table, lib)),
        ("opportunistic", lambda: [P.test_opportunistic_equals_masked_step(a, d, table, lib)
                                   for a in (0.0, 0.7, 1.0) for d in ("f32", "bf16")]),
        ("opportunistic_tie", lambda: P.test_opportunistic_planted_tie_goes_to_lowest_allowed(lib)),
        ("philox_kat", lambda: [P.test_philox_known_answers(c, k, o, lib) for c, k, o in P.PHILOX_KAT]),
        ("gumbel_words", lambda: [P.test_gumbel_noise_from_published_philox_words(k, lib) for k in (0, 2)]),
        ("ln_f32", lambda: P.test_ln_f32_accuracy(lib)),
        ("gumbel_ks", lambda: P.test_gumbel_noise_is_gumbel_distributed(lib)),
        ("sample_softmax", lambda: [P.test_sample_frequencies_follow_masked_softmax(t, d, lib)
                                    for t in (1.0, 2.0) for d in ("f32", "bf16")]),
        ("sample_greedy", lambda: P.test_sample_at_low_temperature_is_the_masked_argmax(table, lib)),
        ("sample_inv", lambda: P.test_sample_invariants(table, lib)),
        ("ties_bf16", lambda: [P.test_planted_ties_and_specials_bf16(b, a, e, lib)
                               for b, a, e in [([0x8000, 0x0000, 0x0001], [0, 1, 2], 2),
                                               ([0x3F80, 0x3F80, 0x3F80], [1, 2], 1),
                                               ([0x7FC1, 0xC000, 0x7F80], [0, 1], 1)]]),
    ]
    failed = []
    for name, fn in checks:
        try:
            fn()
        except (AssertionError, IndexError, ValueError):
            failed.append(name)
    return failed


def test_unmutated_copy_passes_every_pin(tmp_path):
    out = str(tmp_path / "liboracle_plain.so")
    subprocess.run(["gcc", "-O2", "-std=c11", "-shared", "-fPIC", "-o", out, SRC, "-lm"], check=True)
    assert _checks(oracle.load(out)) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation anchor not found: {old!r}"
    mutated = src.replace(old, new)
    path = tmp_path / "mutant.c"
    path.write_text(mutated)
    out = str(tmp_path / "libmutant.so")
    subprocess.run(["gcc", "-O2", "-std=c11", "-shared", "-fPIC", "-o", out, str(path), "-lm"],
                   check=True)
    failed = _checks(oracle.load(out))
    assert failed, f"no pin caught the planted mistake '{name}'"
