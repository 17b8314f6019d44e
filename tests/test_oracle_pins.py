"""Pins for the CPU oracle: checks against what the paper and mathematics fix,
not against the oracle itself.

* brute force through an independent formulation (the DFA's transition
  monoid as 0/1 matrices; a token's matrix is the product of its bytes');
* the paper's worked examples (fig:nfa, fig:overview (b)-(d)) from
  ``tests/golden``;
* invariants: single-byte rows, the dead row, concatenation, prefix closure,
  emitted-token-is-allowed, allow bit iff not dead, padding bits zero;
* reductions to library routines (numpy argmax, numpy packbits, torch's
  bf16 -> fp32 conversion);
* the minimal-invasiveness property (Sec. 2 definition);
* planted ties and special values with expected indices known by construction.
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _tiny_dfa(rng, S, symbols, junk=True):
    """Random DFA over ``symbols`` with DEAD moves and (optionally) junk
    out-of-range targets that must read as DEAD."""
    trans = np.full((S, 256), -1, np.int32)
    for s in range(S):
        for b in symbols:
            r = rng.random()
            if r < 0.6:
                trans[s, b] = rng.integers(0, S)
            elif junk and r < 0.75:
                trans[s, b] = S + int(rng.integers(0, 5))  # out of range -> DEAD
            elif junk and r < 0.85:
                trans[s, b] = -int(rng.integers(2, 9))     # negative -> DEAD
    return trans


def _matrix_table(trans, tokens):
    """Independent formulation: M_b is the (S+1)x(S+1) 0/1 matrix of byte b
    with index S standing for DEAD (absorbing); a token maps s to the column of
    the single 1 in row s of the product of its bytes' matrices."""
    S = trans.shape[0]
    D = S
    mats = {}
    for b in range(256):
        M = np.zeros((S + 1, S + 1), np.int64)
        for s in range(S):
            tgt = int(trans[s, b])
            M[s, tgt if 0 <= tgt < S else D] = 1
        M[D, D] = 1
        mats[b] = M
    ns = np.empty((S, len(tokens)), np.int32)
    for t, tok in enumerate(tokens):
        P = np.eye(S + 1, dtype=np.int64)
        for b in tok:
            P = P @ mats[b]
        assert (P.sum(axis=1) == 1).all()
        cols = P.argmax(axis=1)[:S]
        ns[:, t] = np.where(cols == D, -1, cols)
    return ns


def _pack_allow(alive):
    """Library packing: numpy packbits (little bit order) into uint32 words."""
    S, V = alive.shape
    Wd = (V + 31) // 32
    padded = np.zeros((S, Wd * 32), bool)
    padded[:, :V] = alive
    return np.packbits(padded, axis=1, bitorder="little").view("<u4").reshape(S, Wd)


# ------------------------------------------------------------------ P1 brute force

@pytest.mark.parametrize("seed", range(6))
def test_align_matches_transition_monoid(seed, oracle_lib):
    rng = np.random.default_rng(1000 + seed)
    S = int(rng.integers(1, 6))
    alphabet = [ord("a"), ord("b"), ord("c"), ord("x"), 0xFF]
    trans = _tiny_dfa(rng, S, alphabet[:3])
    tokens = [bytes(p) for n in range(0, 5) for p in itertools.product(alphabet, repeat=n)]
    assert len(tokens) == 781
    offsets, data = W.vocab_from_tokens(tokens)
    ns, al = oracle.align(trans, offsets, data, lib=oracle_lib)
    expect = _matrix_table(trans, tokens)
    np.testing.assert_array_equal(ns, expect)
    np.testing.assert_array_equal(al, _pack_allow(expect != -1))


def test_align_rows_equals_full_table(oracle_lib):
    rng = np.random.default_rng(7)
    trans = _tiny_dfa(rng, 9, [ord(c) for c in "abcd"])
    tokens = [bytes(p) for n in range(1, 4) for p in itertools.product(b"abcdz", repeat=n)]
    offsets, data = W.vocab_from_tokens(tokens)
    ns, al = oracle.align(trans, offsets, data, lib=oracle_lib)
    rows = np.array([8, 0, 3, -1, 9, 100, 3], np.int32)
    ns_r, al_r = oracle.align_rows(trans, offsets, data, rows, lib=oracle_lib)
    for i, s in enumerate(rows):
        if 0 <= s < 9:
            np.testing.assert_array_equal(ns_r[i], ns[s])
            np.testing.assert_array_equal(al_r[i], al[s])
        else:  # the dead row: every token dead, no bit set
            assert (ns_r[i] == -1).all() and (al_r[i] == 0).all()


# ----------------------------------------------------------- P2 paper worked examples

def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_fig_nfa_int_rows(oracle_lib):
    g = _golden("fig_nfa_int.json")
    trans = W.dfa_from_spec(len(g["states"]), g["moves"])
    offsets, data = W.vocab_from_tokens([t.encode() for t in g["vocab"]])
    ns, al = oracle.align(trans, offsets, data, lib=oracle_lib)
    np.testing.assert_array_equal(ns, np.array(g["expected_next_state"], np.int32))
    np.testing.assert_array_equal(al[:, 0], np.array([int(x, 16) for x in g["expected_allow"]],
                                                     np.uint32))


def test_fig_overview_subterminal_landing(oracle_lib):
    g = _golden("fig_overview_scanner.json")
    trans = W.dfa_from_spec(len(g["states"]), g["moves"])
    toks = g["vocab"]
    offsets, data = W.vocab_from_tokens([t.encode() for t in toks])
    ns, al = oracle.align(trans, offsets, data, lib=oracle_lib)
    q = g["from_state"]
    for i, t in enumerate(toks):
        assert ns[q, i] == g["expected_landing"][t], t
        assert ns[0, i] == g["expected_from_start"][t], t
    # every byte token of (c) is a valid scanner continuation from the int state
    assert al[q, 0] == (1 << len(toks)) - 1
    # a token with no continuation (Sec. 3.3 adds 'a' as the example)
    assert oracle.walk(trans, q, b"a", lib=oracle_lib) == -1


# --------------------------------------------------------------------- P3 invariants

@pytest.fixture(scope="module")
def tiny_table(oracle_lib):
    trans, _ = W.dfa(1)
    offsets, data = W.vocab(1)
    ns, al = oracle.align(trans, offsets, data, lib=oracle_lib)
    return trans, offsets, data, ns, al


def test_single_byte_rows_equal_transition_row(tiny_table):
    trans, offsets, data, ns, _ = tiny_table
    lens = np.diff(offsets)
    S = trans.shape[0]
    for t in np.nonzero(lens == 1)[0]:
        b = data[offsets[t]]
        col = trans[:, b]
        np.testing.assert_array_equal(ns[:, t], np.where((col >= 0) & (col < S), col, -1))


def test_allow_bit_iff_alive_and_padding_zero(tiny_table):
    _, _, _, ns, al = tiny_table
    np.testing.assert_array_equal(al, _pack_allow(ns != -1))
    V = ns.shape[1]
    if V % 32:
        assert (al[:, -1] >> np.uint32(V % 32) == 0).all()


def test_concatenation_homomorphism(tiny_table, oracle_lib):
    trans, offsets, data, ns, _ = tiny_table
    toks = W.tokens_of(offsets, data)
    rng = np.random.default_rng(3)
    S, V = ns.shape
    for _ in range(3000):
        s = int(rng.integers(0, S))
        t1, t2 = (int(x) for x in rng.integers(0, V, 2))
        mid = ns[s, t1]
        via_table = -1 if mid == -1 else ns[mid, t2]
        assert oracle.walk(trans, s, toks[t1] + toks[t2], lib=oracle_lib) == via_table


def test_prefix_closure(tiny_table, oracle_lib):
    trans, offsets, data, ns, _ = tiny_table
    toks = W.tokens_of(offsets, data)
    S = ns.shape[0]
    for t, tok in enumerate(toks):
        for s in range(S):
            if ns[s, t] != -1:
                for k in range(len(tok)):
                    assert oracle.walk(trans, s, tok[:k], lib=oracle_lib) != -1


def test_dead_row_is_empty(tiny_table, oracle_lib):
    trans, offsets, data, ns, al = tiny_table
    V = ns.shape[1]
    x = np.random.default_rng(0).standard_normal((3, V)).astype(np.float32)
    tok, nst = oracle.masked_step(ns, al, np.array([-1, 16, 1 << 30], np.int32), x, lib=oracle_lib)
    assert (tok == -1).all() and (nst == -1).all()


def test_emitted_token_is_allowed_and_state_follows_walk(tiny_table, oracle_lib):
    trans, offsets, data, ns, al = tiny_table
    toks = W.tokens_of(offsets, data)
    S, V = ns.shape
    rng = np.random.default_rng(11)
    states = rng.integers(0, S, 64).astype(np.int32)
    x = (rng.standard_normal((64, V)) * 2).astype(np.float32)
    tok, nst = oracle.masked_step(ns, al, states, x, lib=oracle_lib)
    for b in range(64):
        if tok[b] == -1:
            assert (al[states[b]] == 0).all() and nst[b] == -1
            continue
        assert (al[states[b], tok[b] // 32] >> np.uint32(tok[b] % 32)) & 1
        assert nst[b] == oracle.walk(trans, int(states[b]), toks[tok[b]], lib=oracle_lib) != -1


def test_walk_lookup_count_small_case(oracle_lib):
    g = _golden("fig_nfa_int.json")
    trans = W.dfa_from_spec(len(g["states"]), g["moves"])
    offsets, data = W.vocab_from_tokens([t.encode() for t in g["vocab"]])
    # from state 0: 0,1,2 one move each; 12 two; ) ( + one (dies);
    # +1 one (dies at '+'); '1 (' two ('1' then dies at ' ') -> 11
    assert oracle.walk_lookups(trans, offsets, data, np.array([0], np.int32), lib=oracle_lib) == 11


def test_walk_length_histogram_small_case(oracle_lib):
    g = _golden("fig_nfa_int.json")
    trans = W.dfa_from_spec(len(g["states"]), g["moves"])
    offsets, data = W.vocab_from_tokens([t.encode() for t in g["vocab"]])
    hist = oracle.walk_length_hist(trans, offsets, data, np.array([0], np.int32), lib=oracle_lib)
    # from state 0: 0 1 2 ) ( + one move each, +1 one (dies at '+'): seven
    # walks of length 1; 12 and '1 (' two each
    assert hist.tolist() == [0, 7, 2, 0]  # up to the longest token (3 bytes)
    assert int((np.arange(len(hist)) * hist).sum()) == 11  # the lookup count above


def test_walk_length_histogram_brute_force(oracle_lib):
    rng = np.random.default_rng(21)
    S = 9
    trans = np.where(rng.random((S, 256)) < 0.5, rng.integers(0, S, (S, 256)), -1).astype(np.int32)
    trans[:, :3] = rng.integers(-2, S + 2, (S, 3))  # out-of-range entries read as DEAD
    toks = [bytes(rng.integers(0, 4, int(rng.integers(0, 7))).astype(np.uint8)) for _ in range(60)]
    offsets, data = W.vocab_from_tokens(toks)
    rows = np.array([0, 3, 8, 3], np.int32)
    expect = np.zeros(7, np.int64)
    for r in rows:
        for tok in toks:
            st, n = int(r), 0
            for byte in tok:
                if st == -1:
                    break
                nxt = int(trans[st, byte])
                st = nxt if 0 <= nxt < S else -1
                n += 1
            expect[n] += 1
    hist = oracle.walk_length_hist(trans, offsets, data, rows, lib=oracle_lib)
    assert hist.tolist() == expect[:len(hist)].tolist() and expect[len(hist):].sum() == 0
    assert int((np.arange(len(hist)) * hist).sum()) == oracle.walk_lookups(trans, offsets, data, rows,
                                                                            lib=oracle_lib)


# ------------------------------------------------------- P4 reductions to library calls

def _reference_choice(x_f32, allowed):
    return int(np.argmax(np.where(allowed, x_f32, -np.inf)))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_masked_step_equals_numpy_argmax(dtype, tiny_table, oracle_lib):
    _, _, _, ns, al = tiny_table
    S, V = ns.shape
    rng = np.random.default_rng(5)
    B, ld = 40, V + 13
    states = rng.integers(0, S, B).astype(np.int32)
    xt = torch.from_numpy(rng.standard_normal((B, ld)).astype(np.float32) * 3)
    if dtype == "bf16":
        xt = xt.to(torch.bfloat16)
        arr = xt.view(torch.int16).numpy().view(np.uint16)
        ref = xt.float().numpy()          # torch's own bf16 -> fp32 conversion
    else:
        arr = xt.numpy()
        ref = arr
    tok, _ = oracle.masked_step(ns, al, states, arr, lib=oracle_lib)
    alive = ns != -1
    checked = 0
    for b in range(B):
        allowed = alive[states[b]]
        if allowed.any():
            assert tok[b] == _reference_choice(ref[b, :V], allowed)
            checked += 1
        else:
            assert tok[b] == -1
    assert checked > B // 2


def test_single_accepting_state_is_unconstrained_argmax(oracle_lib):
    trans = np.zeros((1, 256), np.int32)  # every byte loops on state 0
    offsets, data = W.vocab(1)
    ns, al = oracle.align(trans, offsets, data, lib=oracle_lib)
    assert (ns == 0).all()
    x = np.random.default_rng(9).standard_normal((8, ns.shape[1])).astype(np.float32)
    tok, nst = oracle.masked_step(ns, al, np.zeros(8, np.int32), x, lib=oracle_lib)
    np.testing.assert_array_equal(tok, np.argmax(x, axis=1))
    assert (nst == 0).all()


# ------------------------------------------------ P5 minimal invasiveness (Sec. 2)

def test_minimally_invasive_when_unconstrained_choice_is_valid(tiny_table, oracle_lib):
    _, _, _, ns, al = tiny_table
    S, V = ns.shape
    rng = np.random.default_rng(21)
    hits = 0
    for trial in range(200):
        s = int(rng.integers(0, S))
        x = rng.standard_normal(V).astype(np.float32)
        allowed_idx = np.nonzero(ns[s] != -1)[0]
        if trial % 2 and allowed_idx.size:
            x[allowed_idx[rng.integers(0, allowed_idx.size)]] = 50.0  # model prefers a valid token
        free = int(np.argmax(x))
        tok, _ = oracle.masked_step(ns, al, np.array([s], np.int32), x[None], lib=oracle_lib)
        if ns[s, free] != -1:
            assert tok[0] == free
            hits += 1
        else:
            assert tok[0] != free
    assert hits >= 90


# ------------------------------------------------------------- P6 planted specials

def _one_row(values, allowed_idx, dtype="f32"):
    V = len(values)
    ns = np.full((1, V), -1, np.int32)
    ns[0, list(allowed_idx)] = 0
    al = _pack_allow(ns != -1)
    if dtype == "f32":
        x = np.array(values, np.float32)[None]
    else:
        x = np.array(values, np.uint16)[None]
    return ns, al, x


@pytest.mark.parametrize("values,allowed,expect", [
    ([100, 9, 9, 5, 1, 9, 0, 9, 0, 0.5], [1, 2, 5, 7, 9], 1),       # equal maxima: lowest index
    ([0, 1, -0.0, 7, 7, 0.0, 9], [2, 5], 2),                          # -0 ties +0
    ([0, 1, 0.0, 7, 7, -0.0, 9], [2, 5], 2),
    ([5, float("nan"), 3, 3, -np.inf], [1, 4], 1),                    # NaN ranks as -inf: tie
    ([5, -np.inf, 3, 3, float("nan")], [1, 4], 1),
    ([float("nan")] * 6, [3, 5], 3),                                  # all NaN: lowest allowed
    ([float("nan"), 2.0, 1.0], [0, 1, 2], 1),                         # NaN first, a number wins
    ([float("nan"), -3e38, 1.0], [0, 1], 1),
    ([np.inf, 1e30, np.inf, 2, 3], [1, 3], 1),                        # disallowed +inf ignored
    ([1, np.inf, 1e38, np.inf], [1, 2, 3], 1),
    ([-np.inf, -np.inf, -3e38], [0, 1], 0),
    ([-1e-45, 0.0, 1e-45, -0.0], [0, 1, 3], 1),                       # subnormals
    ([-1e-45, 0.0, 1e-45, -0.0], [0, 2, 3], 2),
    ([1, 2, 3], [], -1),                                              # empty row
])
def test_planted_ties_and_specials_f32(values, allowed, expect, oracle_lib):
    ns, al, x = _one_row(values, allowed)
    tok, nst = oracle.masked_step(ns, al, np.array([0], np.int32), x, lib=oracle_lib)
    assert tok[0] == expect
    assert nst[0] == (0 if expect >= 0 else -1)


@pytest.mark.parametrize("bits,allowed,expect", [
    ([0x3F80, 0x3F80, 0x3F80], [1, 2], 1),                 # 1.0 ties
    ([0x8000, 0x0000, 0x0001], [0, 1], 0),                 # -0 vs +0 tie
    ([0x8000, 0x0000, 0x0001], [0, 1, 2], 2),              # smallest positive subnormal wins
    ([0x7FC1, 0xFF80, 0xFFC1], [0, 1, 2], 0),              # +NaN, -inf, -NaN all rank -inf
    ([0x7FC1, 0xC000, 0x7F80], [0, 1], 1),                 # NaN first, -2 wins
    ([0xFFC1, 0xFF7F], [0, 1], 1),                         # -NaN first, lowest finite wins
    ([0x7F80, 0x7F7F, 0xFF80], [1, 2], 1),                 # largest finite vs -inf
    ([0xBF80, 0xC000, 0xBF80], [0, 1, 2], 0),              # -1 beats -2, tie to lowest
])
def test_planted_ties_and_specials_bf16(bits, allowed, expect, oracle_lib):
    ns, al, x = _one_row(bits, allowed, "bf16")
    tok, _ = oracle.masked_step(ns, al, np.array([0], np.int32), x, lib=oracle_lib)
    assert tok[0] == expect


def test_leading_dimension_and_row_independence(tiny_table, oracle_lib):
    _, _, _, ns, al = tiny_table
    S, V = ns.shape
    rng = np.random.default_rng(2)
    x = rng.standard_normal((6, V + 7)).astype(np.float32)
    states = rng.integers(0, S, 6).astype(np.int32)
    tok, nst = oracle.masked_step(ns, al, states, x, lib=oracle_lib)
    for b in range(6):
        t1, n1 = oracle.masked_step(ns, al, states[b:b + 1], np.ascontiguousarray(x[b:b + 1, :V]),
                                    lib=oracle_lib)
        assert (t1[0], n1[0]) == (tok[b], nst[b])


def test_oracle_is_deterministic(tiny_table, oracle_lib):
    trans, offsets, data, ns, al = tiny_table
    ns2, al2 = oracle.align(trans, offsets, data, lib=oracle_lib)
    np.testing.assert_array_equal(ns, ns2)
    np.testing.assert_array_equal(al, al2)


def test_masked_chain_matches_batch_steps(tiny_table, oracle_lib):
    trans, offsets, data, ns, al = tiny_table
    S, V = ns.shape
    rng = np.random.default_rng(4)
    steps = 12
    x = rng.standard_normal((steps, 3, V)).astype(np.float32)
    states = np.array([0, 5, 11], np.int32)
    cache = oracle.RowCache(trans, offsets, data, lib=oracle_lib)
    chains = [oracle.masked_chain(cache, states[b], x[:, b]) for b in range(3)]
    cur = states
    for k in range(steps):
        tok, nxt = oracle.masked_step(ns, al, cur, x[k], lib=oracle_lib)
        for b in range(3):
            assert chains[b][0][k] == tok[b] and chains[b][1][k + 1] == nxt[b]
        cur = nxt


# ------------------------------------------------- end-of-sequence token (EOS)

def test_fig_nfa_eos_column(oracle_lib):
    g = _golden("fig_nfa_int.json")
    e = g["eos"]
    trans = W.dfa_from_spec(len(g["states"]), g["moves"])
    toks = [t.encode() for t in g["vocab"]] + [b"</s>"]
    offsets, data = W.vocab_from_tokens(toks)
    ns, al = oracle.align_eos(trans, offsets, data, np.array(e["accepting"], np.uint8),
                              e["eos_token"], lib=oracle_lib)
    np.testing.assert_array_equal(ns[:, e["eos_token"]], e["expected_eos_column"])
    np.testing.assert_array_equal(ns[:, :9], np.array(g["expected_next_state"]))
    np.testing.assert_array_equal(al[:, 0], np.array([int(x, 16) for x in e["expected_allow"]],
                                                     np.uint32))


def test_eos_column_invariants(tiny_table, oracle_lib):
    trans, offsets, data, ns, al = tiny_table
    _, acc = W.dfa(1)
    S, V = ns.shape
    for eos in (0, 17, V - 1):
        ns_e, al_e = oracle.align_eos(trans, offsets, data, acc, eos, lib=oracle_lib)
        expect = np.where(acc.astype(bool), np.arange(S), -1)
        np.testing.assert_array_equal(ns_e[:, eos], expect)
        others = np.ones(V, bool)
        others[eos] = False
        np.testing.assert_array_equal(ns_e[:, others], ns[:, others])  # every other column unchanged
        np.testing.assert_array_equal(al_e, _pack_allow(ns_e != -1))
    # no accepting flags: EOS never allowed; dead / out-of-range rows stay empty
    ns_n, al_n = oracle.align_eos(trans, offsets, data, None, 5, rows=np.array([0, -1, S]), lib=oracle_lib)
    assert (ns_n[:, 5] == -1).all() and (al_n[1:] == 0).all()


def test_eos_is_chosen_when_it_is_the_best_allowed(tiny_table, oracle_lib):
    trans, offsets, data, ns, al = tiny_table
    _, acc = W.dfa(1)
    S, V = ns.shape
    eos = V - 1
    ns_e, al_e = oracle.align_eos(trans, offsets, data, acc, eos, lib=oracle_lib)
    x = np.random.default_rng(8).standard_normal((S, V)).astype(np.float32)
    x[:, eos] = 100.0  # the model wants to stop everywhere
    tok, nxt = oracle.masked_step(ns_e, al_e, np.arange(S, dtype=np.int32), x, lib=oracle_lib)
    for s in range(S):
        if acc[s]:
            assert tok[s] == eos and nxt[s] == s  # stops, state unchanged
        else:
            assert tok[s] != eos


# ------------------------------------------- speculative chain check (Sec. 3.6)

def _fig_nfa_spec_case():
    g = _golden("fig_nfa_int.json")
    e, sp = g["eos"], g["spec"]
    trans = W.dfa_from_spec(len(g["states"]), g["moves"])
    offsets, data = W.vocab_from_tokens([t.encode() for t in g["vocab"]] + [b"</s>"])
    lg = np.array([[[float(v) for v in r] for r in rows] for rows in sp["logits"]], np.float32)
    return trans, offsets, data, np.array(e["accepting"], np.uint8), e["eos_token"], sp, lg


def test_fig_nfa_spec_walk_and_verify(oracle_lib):
    trans, offsets, data, acc, eos, sp, lg = _fig_nfa_spec_case()
    ns, al = oracle.align_eos(trans, offsets, data, acc, eos, lib=oracle_lib)
    states, props = np.array(sp["states"], np.int32), np.array(sp["proposals"], np.int32)
    a, fin = oracle.spec_walk(ns, al, states, props, lib=oracle_lib)
    np.testing.assert_array_equal(a, sp["expected_walk_accepted"])
    np.testing.assert_array_equal(fin, sp["expected_walk_final_state"])
    tok, a, nst = oracle.spec_verify(ns, al, states, props, lg, lib=oracle_lib)
    np.testing.assert_array_equal(tok, sp["expected_token"])
    np.testing.assert_array_equal(a, sp["expected_accepted"])
    np.testing.assert_array_equal(nst, sp["expected_new_state"])


def _bf16_bits(x):
    return (np.ascontiguousarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint16)


def _spec_inputs(ns, al, rng, B, s, keep, lib, dtype="f32"):
    """States (some dead or out of range), position logits [B][s+1][V] and
    proposals that follow the greedy chain with probability ``keep`` per
    position (otherwise: a random id, possibly out of range)."""
    S, V = ns.shape
    states = rng.integers(0, S, B).astype(np.int32)
    states[rng.random(B) < 0.1] = -1
    states[rng.random(B) < 0.05] = S
    x = rng.standard_normal((B, s + 1, V)).astype(np.float32)
    lg = _bf16_bits(x) if dtype == "bf16" else x
    props = np.empty((B, s), np.int32)
    cur = states
    for j in range(s):
        t, nxt = oracle.masked_step(ns, al, cur, lg[:, j], lib=lib)
        other = rng.integers(-2, V + 2, B).astype(np.int32)
        props[:, j] = np.where(rng.random(B) < keep, t, other)
        cur = nxt
    return states, props, lg


def _sequential_greedy(ns, al, state, props, pos_logits, lib):
    """Algorithm 1 one step at a time over the positions, stopping at the first
    choice that differs from the proposal: (tokens, accepted, new_state)."""
    s = props.shape[0]
    toks, cur, j = [], int(state), 0
    while True:
        t, n = oracle.masked_step(ns, al, np.array([cur], np.int32), pos_logits[j][None], lib=lib)
        toks.append(int(t[0]))
        if j == s or t[0] == -1 or t[0] != props[j]:
            return toks, j, int(n[0])
        cur, j = int(n[0]), j + 1


@pytest.mark.parametrize("dtype,layout", [("f32", "rows"), ("bf16", "rows"), ("f32", "steps")])
def test_spec_verify_equals_sequential_greedy(dtype, layout, tiny_table, oracle_lib):
    """Speculation only saves model passes: the emitted tokens and the state are
    those of plain greedy decoding, and the accepted count is where the two
    first disagree (Sec. 3.6)."""
    _, _, _, ns, al = tiny_table
    rng = np.random.default_rng(31)
    B, s = 24, 5
    states, props, lg = _spec_inputs(ns, al, rng, B, s, 0.8, oracle_lib, dtype)
    if layout == "steps":  # the model's output as [positions][B][V], seen through strides
        lg = np.ascontiguousarray(lg.transpose(1, 0, 2)).transpose(1, 0, 2)
    tok, acc, nst = oracle.spec_verify(ns, al, states, props, lg, lib=oracle_lib)
    seen = set()
    for b in range(B):
        toks, a, n = _sequential_greedy(ns, al, states[b], props[b], lg[b], oracle_lib)
        assert acc[b] == a and nst[b] == n
        np.testing.assert_array_equal(tok[b, :a + 1], toks)
        seen.add(a)
    assert len(seen) >= 3  # early, middle and full acceptance all occur


def test_spec_verify_later_positions_follow_the_proposals(tiny_table, oracle_lib):
    """token[b][j] is the masked greedy choice in the state the first j proposals
    lead to; DEAD (token -1) once a proposal was not allowed."""
    _, _, _, ns, al = tiny_table
    rng = np.random.default_rng(32)
    B, s = 16, 4
    states, props, lg = _spec_inputs(ns, al, rng, B, s, 0.6, oracle_lib)
    tok, _, _ = oracle.spec_verify(ns, al, states, props, lg, lib=oracle_lib)
    for j in range(s + 1):
        a, fin = oracle.spec_walk(ns, al, states, props[:, :j], lib=oracle_lib)
        st_j = np.where(a == j, fin, -1).astype(np.int32)
        t, _ = oracle.masked_step(ns, al, st_j, lg[:, j], lib=oracle_lib)
        np.testing.assert_array_equal(tok[:, j], t)


def test_spec_walk_matches_byte_walk(tiny_table, oracle_lib):
    """The accepted proposals, read as one byte string from the row's state,
    land on the final state; the first rejected one is out of range or makes
    that byte walk die (concatenation of walks, Sec. 3.3)."""
    trans, offsets, data, ns, al = tiny_table
    S, V = ns.shape
    rng = np.random.default_rng(33)
    B, s = 40, 6
    states, props, _ = _spec_inputs(ns, al, rng, B, s, 0.85, oracle_lib)
    acc, fin = oracle.spec_walk(ns, al, states, props, lib=oracle_lib)
    tok_bytes = [bytes(data[offsets[t]:offsets[t + 1]]) for t in range(V)]
    for b in range(B):
        a = int(acc[b])
        text = b"".join(tok_bytes[t] for t in props[b, :a])
        assert oracle.walk(trans, states[b], text, lib=oracle_lib) == fin[b]
        if a < s:
            t = int(props[b, a])
            assert not (0 <= t < V) or oracle.walk(trans, states[b], text + tok_bytes[t],
                                                   lib=oracle_lib) == -1
    assert 0 < (acc == s).sum() < B


def test_spec_verify_accepts_only_legal_prefixes(tiny_table, oracle_lib):
    _, _, _, ns, al = tiny_table
    rng = np.random.default_rng(34)
    states, props, lg = _spec_inputs(ns, al, rng, 32, 6, 0.7, oracle_lib)
    walk_acc, _ = oracle.spec_walk(ns, al, states, props, lib=oracle_lib)
    _, acc, _ = oracle.spec_verify(ns, al, states, props, lg, lib=oracle_lib)
    assert (acc <= walk_acc).all()


def test_spec_zero_proposals_is_one_masked_step(tiny_table, oracle_lib):
    _, _, _, ns, al = tiny_table
    S, V = ns.shape
    rng = np.random.default_rng(35)
    states = np.array([0, 3, -1, S, 7], np.int32)
    x = rng.standard_normal((5, 1, V)).astype(np.float32)
    tok, acc, nst = oracle.spec_verify(ns, al, states, np.zeros((5, 0), np.int32), x, lib=oracle_lib)
    t, n = oracle.masked_step(ns, al, states, x[:, 0], lib=oracle_lib)
    np.testing.assert_array_equal(tok[:, 0], t)
    np.testing.assert_array_equal(nst, n)
    assert (acc == 0).all()
    a, fin = oracle.spec_walk(ns, al, states, np.zeros((5, 0), np.int32), lib=oracle_lib)
    assert (a == 0).all()
    np.testing.assert_array_equal(fin, [0, 3, -1, -1, 7])


def test_spec_perfect_draft_is_fully_accepted(tiny_table, oracle_lib):
    _, _, _, ns, al = tiny_table
    rng = np.random.default_rng(36)
    B, s = 12, 7
    states = rng.integers(0, ns.shape[0], B).astype(np.int32)
    lg = rng.standard_normal((B, s + 1, ns.shape[1])).astype(np.float32)
    props = np.empty((B, s), np.int32)
    cur = states
    for j in range(s):  # proposals = the greedy chain from these states
        t, cur = oracle.masked_step(ns, al, cur, lg[:, j], lib=oracle_lib)
        props[:, j] = t
    bonus, after = oracle.masked_step(ns, al, cur, lg[:, s], lib=oracle_lib)
    tok, acc, nst = oracle.spec_verify(ns, al, states, props, lg, lib=oracle_lib)
    live = (props != -1).all(axis=1)
    assert live.sum() >= B // 2
    assert (acc[live] == s).all()
    np.testing.assert_array_equal(tok[live, s], bonus[live])
    np.testing.assert_array_equal(nst[live], after[live])


def test_spec_verify_rows_matches_table_version(tiny_table, oracle_lib):
    """The row-cache form used for full-size workloads agrees with the
    whole-table form on a workload small enough for both."""
    trans, offsets, data, ns, al = tiny_table
    rng = np.random.default_rng(37)
    states, props, lg = _spec_inputs(ns, al, rng, 20, 5, 0.7, oracle_lib, "bf16")
    tok, acc, nst = oracle.spec_verify(ns, al, states, props, lg, lib=oracle_lib)
    cache = oracle.RowCache(trans, offsets, data, lib=oracle_lib)
    for b in range(20):
        t, a, n = oracle.spec_verify_rows(cache, states[b], props[b], lg[b], lib=oracle_lib)
        np.testing.assert_array_equal(t, tok[b])
        assert a == acc[b] and n == nst[b]


# ------------------------------------- opportunistic masking (Sec. 3.5, optimizations)

@pytest.mark.parametrize("adherent", [0.0, 0.7, 1.0])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_opportunistic_equals_masked_step(adherent, dtype, tiny_table, oracle_lib):
    """Checking the model's own choice first never changes the result, and the
    check succeeds exactly when numpy's argmax (NaN as -inf) is allowed."""
    _, _, _, ns, al = tiny_table
    S, V = ns.shape
    rng = np.random.default_rng(41)
    B = 64
    states = rng.integers(0, S, B).astype(np.int32)
    states[:3] = [-1, S, 0]
    x = rng.standard_normal((B, V)).astype(np.float32)
    x[5, rng.integers(0, V, 40)] = np.nan
    x[6] = np.nan
    t, _ = oracle.masked_step(ns, al, states, x, lib=oracle_lib)
    adh = rng.random(B) < adherent
    x[adh & (t >= 0), t[adh & (t >= 0)]] = 40.0   # the model wants the masked choice itself
    lg = _bf16_bits(x) if dtype == "bf16" else x
    tok, nst, ok = oracle.masked_step_opportunistic(ns, al, states, lg, lib=oracle_lib)
    t2, n2 = oracle.masked_step(ns, al, states, lg, lib=oracle_lib)
    np.testing.assert_array_equal(tok, t2)
    np.testing.assert_array_equal(nst, n2)
    xf = lg.astype(np.uint32) << 16 if dtype == "bf16" else lg
    xf = xf.view(np.float32) if dtype == "bf16" else xf
    free = np.argmax(np.where(np.isnan(xf), -np.inf, xf), axis=1)
    live = (states >= 0) & (states < S)
    allowed_free = np.array([ns[s, f] != -1 if l else False for s, f, l in zip(states, free, live)])
    np.testing.assert_array_equal(ok, allowed_free)
    if adherent == 1.0:
        assert ok[live & (t >= 0)].all()


def test_opportunistic_planted_tie_goes_to_lowest_allowed(oracle_lib):
    V = 40
    ns = np.full((1, V), -1, np.int32)
    ns[0, [3, 7, 11]] = 0
    al = _pack_allow(ns != -1)
    x = np.zeros((1, V), np.float32)
    x[0, [3, 7, 20]] = 5.0        # tie at 3 and 7 (allowed) and 20 (not allowed)
    tok, _, ok = oracle.masked_step_opportunistic(ns, al, np.zeros(1, np.int32), x, lib=oracle_lib)
    assert tok[0] == 3 and ok[0]
    x[0, 1] = 5.0                 # now the lowest maximum (1) is not allowed
    tok, _, ok = oracle.masked_step_opportunistic(ns, al, np.zeros(1, np.int32), x, lib=oracle_lib)
    assert tok[0] == 3 and not ok[0]


# ---------------------------------------- masked sampling (Sec. 4 samples at T = 1)

# Known-answer vectors of Philox4x32-10 published with the generator
# (Salmon et al., SC 2011; the Random123 distribution's test vectors).
PHILOX_KAT = [
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF,) * 4, (0xFFFFFFFF,) * 2, (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]


@pytest.mark.parametrize("ctr,key,out", PHILOX_KAT)
def test_philox_known_answers(ctr, key, out, oracle_lib):
    assert tuple(int(x) for x in oracle.philox4x32_10(ctr, key, lib=oracle_lib)) == out


def _gumbel_from_words(w):
    u = (2.0 * (np.uint64(w) >> np.uint64(9)) + 1.0) * 2.0 ** -24
    return -np.log(-np.log(u))


@pytest.mark.parametrize("k", [0, 2])
def test_gumbel_noise_from_published_philox_words(k, oracle_lib):
    """The noise of the tokens whose counters are the published inputs equals
    -ln(-ln u) of the published outputs (float64 reference): pins the counter
    layout (token / 4, row, offset) and the word each token takes."""
    ctr, key, out = PHILOX_KAT[k]
    seed = key[0] | (key[1] << 32)
    offset = ctr[2] | (ctr[3] << 32)
    for j in range(4):
        g = oracle.gumbel(seed, offset, ctr[1], 4 * ctr[0] + j, lib=oracle_lib)
        ref = _gumbel_from_words(out[j])
        assert abs(g - ref) <= 4e-6 * max(1.0, abs(ref)), (j, g, ref)


def test_ln_f32_accuracy(oracle_lib):
    rng = np.random.default_rng(51)
    xs = np.concatenate([rng.uniform(2.0 ** -24, 1.0, 4000), rng.uniform(5.9e-8, 20.0, 4000),
                         2.0 ** rng.uniform(-24, 5, 2000), [1.0, 2.0, 0.5, np.sqrt(2.0), 0.70710678]])
    worst = 0.0
    for x in xs.astype(np.float32):
        ref = np.log(np.float64(x))
        got = oracle.ln_f32(x, lib=oracle_lib)
        ulp = np.spacing(np.float32(max(abs(ref), 2.0 ** -24)))
        worst = max(worst, abs(got - ref) / ulp)
    assert worst <= 2.5
    assert oracle.ln_f32(1.0, lib=oracle_lib) == 0.0


def test_gumbel_noise_is_gumbel_distributed(oracle_lib):
    """Kolmogorov-Smirnov distance to the Gumbel CDF exp(-exp(-g))."""
    n = 40000
    g = np.array([oracle.gumbel(7, 3, r, t, lib=oracle_lib) for r in range(4) for t in range(n // 4)])
    g.sort()
    cdf = np.exp(-np.exp(-g))
    emp = np.arange(1, n + 1) / n
    ks = max(np.abs(cdf - emp).max(), np.abs(cdf - (emp - 1.0 / n)).max())
    assert ks < 1.63 / np.sqrt(n) * 1.5   # well inside the 1 % critical value's range
    assert abs(g.mean() - 0.5772) < 0.02  # Euler-Mascheroni constant


def _one_state_table(V, allowed):
    ns = np.full((1, V), -1, np.int32)
    ns[0, allowed] = 0
    return ns, _pack_allow(ns != -1)


@pytest.mark.parametrize("inv_t", [1.0, 2.0])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sample_frequencies_follow_masked_softmax(inv_t, dtype, oracle_lib):
    """Many draws (different offsets) of one row: chi-square of the counts
    against softmax(x / T) over the allowed tokens; disallowed never drawn."""
    V = 40
    allowed = [1, 5, 6, 17, 30, 39]
    ns, al = _one_state_table(V, allowed)
    x = np.linspace(-1.5, 1.2, V).astype(np.float32)
    x[[5, 30]] = 0.3                            # a tie in value
    lg = _bf16_bits(x[None]) if dtype == "bf16" else x[None]
    xv = (lg.astype(np.uint32) << 16).view(np.float32)[0] if dtype == "bf16" else x
    n = 6000
    B = 8                                         # rows of one call draw independently
    counts = np.zeros(V)
    for off in range(n // B):
        tok, _ = oracle.masked_sample(ns, al, np.zeros(B, np.int32), np.repeat(lg, B, 0), inv_t, 11, off,
                                      lib=oracle_lib)
        np.add.at(counts, tok, 1)
    p = np.exp(xv[allowed].astype(np.float64) * inv_t)
    p /= p.sum()
    exp = p * n
    chi2 = ((counts[allowed] - exp) ** 2 / exp).sum()
    assert counts.sum() == n and counts[np.setdiff1d(np.arange(V), allowed)].sum() == 0
    assert chi2 < 25.7                            # 5 degrees of freedom, p = 1e-4


def test_sample_at_low_temperature_is_the_masked_argmax(tiny_table, oracle_lib):
    """With 1/T = 10^4 and logits at least 0.01 apart the noise (range < 20)
    cannot reorder them: the draw is the masked greedy choice."""
    _, _, _, ns, al = tiny_table
    S, V = ns.shape
    rng = np.random.default_rng(52)
    B = 32
    x = np.stack([rng.permutation(V).astype(np.float32) * 0.01 for _ in range(B)])
    x[3, :5] = np.nan
    states = rng.integers(0, S, B).astype(np.int32)
    states[:2] = [-1, S]
    t_s, n_s = oracle.masked_sample(ns, al, states, x, 1e4, 5, 9, lib=oracle_lib)
    t_g, n_g = oracle.masked_step(ns, al, states, x, lib=oracle_lib)
    np.testing.assert_array_equal(t_s, t_g)
    np.testing.assert_array_equal(n_s, n_g)


def test_sample_invariants(tiny_table, oracle_lib):
    trans, _, _, ns, al = tiny_table
    S, V = ns.shape
    rng = np.random.default_rng(53)
    B = 48
    x = rng.standard_normal((B, V)).astype(np.float32) * 3
    states = rng.integers(0, S, B).astype(np.int32)
    states[:3] = [-1, S, 2 ** 30]
    t1, n1 = oracle.masked_sample(ns, al, states, x, 1.0, 99, 0, lib=oracle_lib)
    t2, n2 = oracle.masked_sample(ns, al, states, x, 1.0, 99, 0, lib=oracle_lib)
    t3, _ = oracle.masked_sample(ns, al, states, x, 1.0, 99, 1, lib=oracle_lib)
    np.testing.assert_array_equal(t1, t2)        # reproducible
    assert (t1 != t3).sum() > B // 4              # another offset draws anew
    assert (t1[:3] == -1).all() and (n1[:3] == -1).all()
    live = t1 >= 0
    assert (ns[states[live], t1[live]] != -1).all()  # always an allowed token
    np.testing.assert_array_equal(n1[live], ns[states[live], t1[live]])
