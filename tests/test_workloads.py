"""The seeded input generators: determinism, shapes and the stated structure."""
import numpy as np
import pytest

import workloads as W


def test_seeded_generators_are_deterministic():
    t1, a1 = W.dfa(1)
    W.dfa.cache_clear()
    t2, a2 = W.dfa(1)
    assert W.sha256(t1) == W.sha256(t2) and W.sha256(a1) == W.sha256(a2)
    o1, d1 = W.vocab(1)
    W._vocab_of.cache_clear()
    o2, d2 = W.vocab(1)
    assert W.sha256(o1) == W.sha256(o2) and W.sha256(d1) == W.sha256(d2)


@pytest.mark.parametrize("wid", [1, 2])
def test_random_dfa_shape(wid):
    w = W.WORKLOADS[wid]
    trans, acc = W.dfa(wid)
    assert trans.shape == (w.S, 256) and trans.dtype == np.int32
    assert int(acc.sum()) == round(0.25 * w.S)
    live = trans != -1
    per_state = live.sum(axis=1)
    lo, hi = w.subset
    assert per_state.min() >= lo and per_state.max() <= min(hi, 95)
    assert (trans[live] < w.S).all()
    # only printable ASCII moves
    assert not live[:, :0x20].any() and not live[:, 0x7F:].any()


@pytest.mark.parametrize("wid", [1, 2])
def test_vocab_unique_and_lengths(wid):
    w = W.WORKLOADS[wid]
    offsets, data = W.vocab(wid)
    assert offsets.shape == (w.V + 1,) and offsets[0] == 0 and offsets[-1] == data.shape[0]
    toks = W.tokens_of(offsets, data)
    assert len(set(toks)) == w.V
    lens = np.diff(offsets)
    hi = w.lengths[2]
    assert lens.min() >= 1 and lens.max() <= hi
    frac_printable = np.mean((data >= 0x20) & (data < 0x7F))
    assert abs(frac_printable - (w.p_printable + (1 - w.p_printable) * 95 / 256)) < 0.02


def test_union_dfa_structure():
    rng = W.rng_for(99, 0)
    trans, acc = W.union_dfa(rng, n_terminals=5, total_states=41, subset=(3, 6))
    assert trans.shape == (41, 256)
    sizes = [8] * 5
    starts = [1 + 8 * i for i in range(5)]
    # moves stay inside a terminal unless taken from the start state's row
    for i, st in enumerate(starts):
        block = range(st, st + sizes[i])
        for s in block:
            for b in range(256):
                tgt = trans[s, b]
                if tgt == -1:
                    continue
                if not (st <= tgt < st + sizes[i]):
                    assert acc[s] and tgt == trans[0, b]
    # start row: first terminal with a move wins
    for b in range(256):
        owners = [st for st in starts if trans[st, b] != -1 and not acc[st]]
        if trans[0, b] == -1:
            assert not owners
    # bytes outside the lexer alphabet are dead everywhere
    alpha = set(W.LEXER_ALPHABET.tolist())
    outside = [b for b in range(256) if b not in alpha]
    assert (trans[:, outside] == -1).all()


def test_union_workload_sizes():
    w = W.WORKLOADS[4]
    assert 31 * 205 + 9 * 204 + 1 == w.S
    assert w.vocab_from == 3


def test_init_states():
    assert (W.init_states(1) == 0).all()
    s3 = W.init_states(3)
    assert s3.shape == (64,) and s3.min() >= 0 and s3.max() < 1024
    assert len(np.unique(s3)) > 32


def test_logits_seeded_cpu():
    import torch
    a = W.logits(1, 3)
    b = W.logits(1, 3)
    c = W.logits(1, 4)
    assert a.dtype == torch.float32 and a.shape == (1, 1000)
    assert torch.equal(a, b) and not torch.equal(a, c)
    assert abs(float(a.std()) - 1.0) < 0.15


def test_dfa_from_spec():
    t = W.dfa_from_spec(2, [(0, "ab", 1), (1, "\t", 0)])
    assert t[0, ord("a")] == 1 and t[0, ord("b")] == 1 and t[1, 9] == 0
    assert (t != -1).sum() == 3
