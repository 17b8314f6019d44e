"""The scanner workloads' automata against Python's own regular-expression
engine (an independent implementation), on the CPU.

``workloads.regex_dfa`` compiles byte regexes to minimal trimmed DFAs; these
tests check, for every terminal of the JSON and C scanners, the JSON-schema
expression and the scanners themselves (``(?:t1|...|tn)*``, Sec. 3.2), that
the automaton accepts exactly the strings ``re.fullmatch`` accepts -- on
corpus text, its substrings, mutated copies and random strings -- and that
every state is reachable from the start and can still reach acceptance.
"""
import re

import numpy as np
import pytest

import workloads as W
from workloads import grammars as G
from workloads.regex_dfa import compile_regex, scanner


def accepts(trans, accepting, text: bytes) -> bool:
    s = 0
    for b in text:
        s = int(trans[s, b])
        if s < 0:
            return False
    return bool(accepting[s])


def _samples(rng, docs, alphabet, n, max_len):
    out = []
    for _ in range(n):
        r = rng.random()
        d = docs[int(rng.integers(len(docs)))].encode()
        if r < 0.3:                                # a substring of real text
            i = int(rng.integers(0, max(1, len(d) - 1)))
            out.append(d[i:i + int(rng.integers(0, max_len))])
        elif r < 0.6:                              # ... with one byte changed, inserted or dropped
            i = int(rng.integers(0, max(1, len(d) - 1)))
            t = bytearray(d[i:i + int(rng.integers(1, max_len))])
            j = int(rng.integers(0, len(t) + 1))
            op = rng.integers(3)
            c = int(alphabet[rng.integers(len(alphabet))])
            if op == 0 and j < len(t):
                t[j] = c
            elif op == 1:
                t.insert(j, c)
            elif j < len(t):
                del t[j]
            out.append(bytes(t))
        else:                                      # random over the grammar's bytes
            out.append(bytes(alphabet[rng.integers(len(alphabet), size=int(rng.integers(0, max_len)))]
                             .astype(np.uint8)))
    return out


@pytest.fixture(scope="module")
def docs():
    return G.corpus(np.random.default_rng(5), 300_000)


JSON_BYTES = np.frombuffer(b' \t\n{}[]:,"\\/bfnrtu0123456789abcdefABCDEF.eE+-xyz\x01\xc3', np.uint8)
C_BYTES = np.frombuffer(b' \t\n/*#_azAZ09xXuUlL.eE+-\'"\\{}[]();,?:~!<>=&|^%@$\x80', np.uint8)


@pytest.mark.parametrize("i", range(len(G.JSON_TERMINALS)))
def test_json_terminal_matches_re(i, docs):
    pat = G.JSON_TERMINALS[i]
    trans, acc = compile_regex(pat)
    rx = re.compile(pat.encode())
    for s in _samples(np.random.default_rng(i), docs, JSON_BYTES, 3000, 24):
        assert accepts(trans, acc, s) == bool(rx.fullmatch(s)), (pat, s)


@pytest.mark.parametrize("i", range(len(G.C_TERMINALS)))
def test_c_terminal_matches_re(i, docs):
    pat = G.C_TERMINALS[i]
    trans, acc = compile_regex(pat)
    rx = re.compile(pat.encode())
    for s in _samples(np.random.default_rng(100 + i), docs, C_BYTES, 3000, 24):
        assert accepts(trans, acc, s) == bool(rx.fullmatch(s)), (pat, s)


@pytest.mark.parametrize("name", ["json-scanner", "json-schema", "c-lexer"])
def test_workload_automaton_matches_re(name, docs):
    if name == "json-scanner":
        (trans, acc), pat, alpha = G.json_scanner(), "(?:" + "|".join(f"(?:{t})" for t in G.JSON_TERMINALS) + ")*", JSON_BYTES
    elif name == "json-schema":
        (trans, acc), pat, alpha = G.json_schema(), G.json_schema_regex(), JSON_BYTES
    else:
        (trans, acc), pat, alpha = G.c_scanner(), "(?:" + "|".join(f"(?:{t})" for t in G.C_TERMINALS) + ")*", C_BYTES
    rx = re.compile(pat.encode())
    rng = np.random.default_rng(7)
    samples = _samples(rng, docs, alpha, 2500, 20)
    hits = 0
    for s in samples:
        got = accepts(trans, acc, s)
        assert got == bool(rx.fullmatch(s)), (name, s)
        hits += got
    if name != "json-schema":
        assert 0 < hits < len(samples)
        return
    # the schema matches whole documents only: whole documents of its shape
    # (compact and pretty-printed) and one-byte mutations of them
    whole = [d.strip() for d in docs if d.startswith('{') and '"enabled"' in d and '"id"' in d][:300]
    assert len(whole) > 100
    mutated = _samples(rng, whole, alpha, 3000, 400)
    hits = 0
    for s in [d.encode() for d in whole] + [m for m in mutated if len(m) > 40]:
        got = accepts(trans, acc, s)
        assert got == bool(rx.fullmatch(s)), (name, s)
        hits += got
    assert hits >= len(whole)
    assert not accepts(trans, acc, b'{"name": "x", "id": 1, "price": 2, "tags": [], "enabled": true}')


@pytest.mark.parametrize("wid", [6, 7, 8])
def test_workload_automata_are_trimmed(wid):
    """Every state is reachable from state 0 and can reach an accepting state
    (so DEAD means "cannot be completed"); no move leaves [0, S)."""
    trans, acc = W.dfa(wid)
    S = trans.shape[0]
    assert S == W.WORKLOADS[wid].S
    assert ((trans >= -1) & (trans < S)).all()
    seen = {0}
    stack = [0]
    while stack:
        s = stack.pop()
        for t in set(trans[s].tolist()) - {-1}:
            if t not in seen:
                seen.add(t)
                stack.append(t)
    assert len(seen) == S
    good = set(np.nonzero(acc)[0].tolist())
    grew = True
    while grew:
        grew = False
        for s in range(S):
            if s not in good and any(t in good for t in trans[s].tolist() if t >= 0):
                good.add(s)
                grew = True
    assert len(good) == S


def test_prefixes_of_real_text_stay_alive(docs):
    """Prefixes of documents the automata accept never walk into DEAD."""
    trans, acc = G.json_scanner()
    for d in [x.encode() for x in docs if x.startswith("{")][:100]:
        s = 0
        for b in d:
            s = int(trans[s, b])
            assert s >= 0
        assert acc[s]


def test_small_automata_by_hand():
    t, a = compile_regex("ab|ac")
    assert t.shape[0] == 3 and a.tolist() == [0, 0, 1]  # the two branches share their end
    t, a = compile_regex("a{2,3}")
    assert accepts(t, a, b"aa") and accepts(t, a, b"aaa") and not accepts(t, a, b"a") and not accepts(t, a, b"aaaa")
    t, a = compile_regex("[^\\x00-\\xfe]")
    assert accepts(t, a, b"\xff") and not accepts(t, a, b"a")
    t, a = scanner(["a", "bc"])
    assert accepts(t, a, b"") and accepts(t, a, b"abca") and not accepts(t, a, b"ab")
    t, a = compile_regex("a(?:b[^\\x00-\\xff])")  # b can never be completed: trimmed away
    assert t.shape[0] == 1 and (t == -1).all() and a[0] == 0


def test_bpe_vocabulary_shape():
    offsets, data = W.vocab(6)
    toks = W.tokens_of(offsets, data)
    assert len(toks) == 32000 and len(set(toks)) == 32000
    assert toks[:256] == [bytes([b]) for b in range(256)]
    assert all(len(t) >= 2 and max(t) < 0x80 for t in toks[256:])
    bridges = {b'":', b'",', b'"}', b'},', b'],'}
    assert bridges <= set(toks)  # tokens that cross JSON terminal boundaries
