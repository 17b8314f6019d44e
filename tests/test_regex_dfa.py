"""The Appendix C grammar automata against Python's own regular-expression
engine (an independent implementation), on the CPU.

``workloads.regex_dfa`` compiles byte regexes to minimal trimmed DFAs; these
tests check, for every terminal of the basic-JSON, simple-C and XML scanners,
for the scanners themselves (R = r+ over the terminals, the lemma of Sec.
3.2) and for the GSM8K and fixed-template grammars (one expression each),
that the automaton accepts exactly the strings ``re.fullmatch`` accepts -- on
corpus text, its substrings, mutated copies and random strings -- that whole
documents of each grammar's shape are accepted and that every prefix of one
stays alive, and that every state is reachable from the start and can still
reach acceptance.
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


def alive(trans, text: bytes) -> bool:
    s = 0
    for b in text:
        s = int(trans[s, b])
        if s < 0:
            return False
    return True


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


def _mutants(rng, docs, alphabet, n):
    """Whole documents with one byte changed, inserted or dropped."""
    out = []
    for _ in range(n):
        t = bytearray(docs[int(rng.integers(len(docs)))].encode())
        j = int(rng.integers(0, len(t) + 1))
        c = int(alphabet[rng.integers(len(alphabet))])
        op = rng.integers(3)
        if op == 0 and j < len(t):
            t[j] = c
        elif op == 1:
            t.insert(j, c)
        elif j < len(t):
            del t[j]
        out.append(bytes(t))
    return out


@pytest.fixture(scope="module")
def docs():
    return G.corpus(np.random.default_rng(5), 400_000)


def _of(docs, kind):
    """The corpus documents of one kind (each generator's shape is distinct)."""
    if kind == "gsm8k":
        return [d for d in docs if '"thoughts"' in d]
    if kind == "template":
        return [d for d in docs if '"A nimble fighter"' in d]
    if kind == "xml":
        return [d for d in docs if d.startswith("<person>")]
    if kind == "json":
        return [d for d in docs if d.startswith("{") and '"name"' in d and '"thoughts"' not in d
                and "nimble" not in d]
    if kind == "c":
        return [d for d in docs if d.split(" ", 1)[0] in ("int", "float", "char")]
    raise KeyError(kind)


JSON_BYTES = np.frombuffer(b' \t\n{}[]:,"\\/bfnrtu0123456789abcdefABCDEF.eE+-xyz\x01\xc3', np.uint8)
C_BYTES = np.frombuffer(b' \t\n/*_azAZ09xX.eE+-"\\{}[]();,<>=!#\'%&|\x80', np.uint8)
XML_BYTES = np.frombuffer(b' \t\n</>personamgjobfridtlsy0123456789ABZ"&\xc3', np.uint8)
TEMPLATE_BYTES = np.frombuffer(b' \t\n\r{}[]:,"idescrptonamgwhlfANb0123456789xyz', np.uint8)
ALPHA = {"json-scanner": JSON_BYTES, "gsm8k-json": JSON_BYTES, "c-scanner": C_BYTES,
         "xml-scanner": XML_BYTES, "template": TEMPLATE_BYTES}
DOC_KIND = {"json-scanner": "json", "gsm8k-json": "gsm8k", "c-scanner": "c", "xml-scanner": "xml",
            "template": "template"}
TERMINALS = {"json": G.JSON_TERMINALS, "c": G.C_TERMINALS, "xml": G.XML_TERMINALS}
TERM_BYTES = {"json": JSON_BYTES, "c": C_BYTES, "xml": XML_BYTES}


@pytest.mark.parametrize("grammar,i", [(g, i) for g in TERMINALS for i in range(len(TERMINALS[g]))])
def test_terminal_matches_re(grammar, i, docs):
    pat = TERMINALS[grammar][i]
    trans, acc = compile_regex(pat)
    rx = re.compile(pat.encode())
    for s in _samples(np.random.default_rng(i), docs, TERM_BYTES[grammar], 2000, 24):
        assert accepts(trans, acc, s) == bool(rx.fullmatch(s)), (pat, s)


@pytest.mark.parametrize("name", list(G.AUTOMATA))
def test_workload_automaton_matches_re(name, docs):
    """Fragments of every kind of document, mutated copies and random strings;
    whole documents of the grammar's shape; and, for the two grammars that
    are one expression each, whole-document mutants.  (A scanner's
    ``(?:t1|...|tn)+`` splits a long text in exponentially many ways, which
    a backtracking engine explores when the text fails to match: the
    scanners are compared on fragments only.)"""
    build, regex = G.AUTOMATA[name]
    trans, acc = build()
    rx = re.compile(regex().encode())
    alpha = ALPHA[name]
    rng = np.random.default_rng(7)
    for s in _samples(rng, docs, alpha, 2500, 20):
        assert accepts(trans, acc, s) == bool(rx.fullmatch(s)), (name, s)
    whole = _of(docs, DOC_KIND[name])[:150]
    assert len(whole) >= 50
    for d in whole:                                  # every document of the shape is accepted
        assert accepts(trans, acc, d.encode()), (name, d)
    if name not in ("gsm8k-json", "template"):
        return
    hits = 0
    for m in _mutants(rng, whole, alpha, 1500):
        got = accepts(trans, acc, m)
        assert got == bool(rx.fullmatch(m)), (name, m)
        hits += got
    assert hits < 1500 // 2                          # the fixed shapes reject most mutants


def test_prefixes_of_real_text_stay_alive(docs):
    """No prefix of a document of a grammar's shape walks into DEAD (the
    mask of Sec. 2 allows exactly continuations that can still complete)."""
    for name, (build, _) in G.AUTOMATA.items():
        trans, acc = build()
        for d in _of(docs, DOC_KIND[name])[:40]:
            s = 0
            for b in d.encode():
                s = int(trans[s, b])
                assert s >= 0, (name, d)
            assert acc[s], name


def test_fixed_shapes_reject_out_of_order_or_missing_fields():
    g, ga = G.gsm8k_json()
    ok = b'{"thoughts": [{"step": "a", "calculation": "1 + 1 = 2", "result": 2}], "answer": 2}'
    assert accepts(g, ga, ok)
    assert not accepts(g, ga, ok.replace(b'"thoughts":', b'"thoughts" :'))    # no ws before the colon
    assert not accepts(g, ga, b'{"thoughts": [], "answer": 2}')                 # at least one thought
    assert not accepts(g, ga, ok.replace(b'"result": 2', b'"result": 02'))     # no leading zero
    t, ta = G.template()
    doc = ('{"id": 1, "description": "A nimble fighter", "name": "Ann", "age": 30, "armor": "plate", '
           '"weapon": "bow", "class": "rogue", "mantra": "Go", "strength": 9, "items": ["a", "b", "c"]}')
    assert accepts(t, ta, doc.encode())
    assert not accepts(t, ta, doc.replace('"plate"', '"cloth"').encode())       # armor is one of three
    assert not accepts(t, ta, doc.replace('"b", ', '').encode())                # exactly three items
    assert not accepts(t, ta, doc.replace('"name": "Ann"', '"name": ""').encode())   # STRING is non-empty
    assert not accepts(t, ta, doc.replace("A nimble", "A strong").encode())     # the fixed description


@pytest.mark.parametrize("wid", [6, 7, 8, 9, 10])
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


def test_scanner_is_r_plus():
    """R = r+ (Sec. 3.2): non-empty terminal sequences only."""
    t, a = scanner(["a", "bc"])
    assert not accepts(t, a, b"") and accepts(t, a, b"a") and accepts(t, a, b"abca")
    assert not accepts(t, a, b"ab") and alive(t, b"ab")
    j, ja = G.json_scanner()
    assert not ja[0]                               # an empty output is not a JSON terminal sequence
    assert accepts(j, ja, b'{"a": [1, 2.5e3, true]}') and accepts(j, ja, b"}}{")   # terminals in any order
    assert not alive(j, b"tru3") and not alive(j, b"01x")


def test_small_automata_by_hand():
    t, a = compile_regex("ab|ac")
    assert t.shape[0] == 3 and a.tolist() == [0, 0, 1]  # the two branches share their end
    t, a = compile_regex("a{2,3}")
    assert accepts(t, a, b"aa") and accepts(t, a, b"aaa") and not accepts(t, a, b"a") and not accepts(t, a, b"aaaa")
    t, a = compile_regex("[^\\x00-\\xfe]")
    assert accepts(t, a, b"\xff") and not accepts(t, a, b"a")
    t, a = compile_regex("a(?:b[^\\x00-\\xff])")  # b can never be completed: trimmed away
    assert t.shape[0] == 1 and (t == -1).all() and a[0] == 0
    assert G.lit("a{b}[c].*") == "a\\{b\\}\\[c\\]\\.\\*"


def test_bpe_vocabulary_shape():
    offsets, data = W.vocab(6)
    toks = W.tokens_of(offsets, data)
    assert len(toks) == 32000 and len(set(toks)) == 32000
    assert toks[:256] == [bytes([b]) for b in range(256)]
    assert all(len(t) >= 2 and max(t) < 0x80 for t in toks[256:])
    # tokens that cross terminal boundaries of the grammars
    bridges = {b'":', b'",', b'"}', b'},', b'],', b'</', b');'}
    assert bridges <= set(toks), bridges - set(toks)
