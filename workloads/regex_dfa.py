"""Regular expressions over bytes -> minimal, trimmed byte DFAs.

Input construction for the scanner workloads (Sec. 3.1-3.2): a terminal's
regular expression becomes a nondeterministic automaton with epsilon moves
(Thompson's construction), the subset construction determinises it, Moore's
partition refinement minimises it, and states from which no accepting state
can be reached are removed, so that a move to DEAD means exactly "this text
can no longer be completed".  A scanner over several terminals, each of
which may follow any other (the chaining of Sec. 3.2), is the automaton of
``(?:t1|t2|...)+`` (the lemma's R = r+).

Like the rest of ``workloads``, this builds inputs only: it walks no
vocabulary and computes no mask.

Supported syntax (bytes; ASCII in the pattern):
  literals, ``.`` (any byte but newline), ``[...]`` / ``[^...]`` with ranges,
  escapes ``\\n \\t \\r \\f \\v \\xHH \\d \\D \\s \\S \\w \\W`` and escaped
  metacharacters, groups ``(...)`` / ``(?:...)``, ``|``, and the greedy
  quantifiers ``* + ? {m} {m,} {m,n}``.
"""
from __future__ import annotations

import numpy as np

DEAD = -1
ALL = frozenset(range(256))
_DIGIT = frozenset(range(0x30, 0x3A))
_SPACE = frozenset(b" \t\n\r\f\v")
_WORD = frozenset(range(0x30, 0x3A)) | frozenset(range(0x41, 0x5B)) | frozenset(range(0x61, 0x7B)) | {0x5F}
_SIMPLE_ESC = {"n": 0x0A, "t": 0x09, "r": 0x0D, "f": 0x0C, "v": 0x0B, "0": 0x00}
_CLASS_ESC = {"d": _DIGIT, "D": ALL - _DIGIT, "s": _SPACE, "S": ALL - _SPACE, "w": _WORD, "W": ALL - _WORD}


# ------------------------------------------------------------------------ parser

class _Parser:
    """Recursive descent: alt := cat ('|' cat)* ; cat := rep* ; rep := atom quant*."""

    def __init__(self, pattern: str):
        self.p = pattern
        self.i = 0

    def parse(self):
        node = self._alt()
        if self.i != len(self.p):
            raise ValueError(f"unexpected {self.p[self.i]!r} at {self.i} in {self.p!r}")
        return node

    def _peek(self):
        return self.p[self.i] if self.i < len(self.p) else None

    def _take(self):
        c = self.p[self.i]
        self.i += 1
        return c

    def _alt(self):
        items = [self._cat()]
        while self._peek() == "|":
            self._take()
            items.append(self._cat())
        return items[0] if len(items) == 1 else ("alt", items)

    def _cat(self):
        items = []
        while self._peek() is not None and self._peek() not in "|)":
            items.append(self._rep())
        if not items:
            return ("eps",)
        return items[0] if len(items) == 1 else ("cat", items)

    def _rep(self):
        node = self._atom()
        while self._peek() is not None and self._peek() in "*+?{":
            c = self._take()
            if c == "*":
                node = ("rep", node, 0, None)
            elif c == "+":
                node = ("rep", node, 1, None)
            elif c == "?":
                node = ("rep", node, 0, 1)
            else:
                j = self.p.index("}", self.i)
                body = self.p[self.i:j]
                self.i = j + 1
                if "," in body:
                    lo, hi = body.split(",", 1)
                    node = ("rep", node, int(lo), int(hi) if hi else None)
                else:
                    node = ("rep", node, int(body), int(body))
        return node

    def _escape(self):
        c = self._take()
        if c in _SIMPLE_ESC:
            return frozenset([_SIMPLE_ESC[c]])
        if c in _CLASS_ESC:
            return _CLASS_ESC[c]
        if c == "x":
            h = self.p[self.i:self.i + 2]
            self.i += 2
            return frozenset([int(h, 16)])
        return frozenset([ord(c)])

    def _atom(self):
        c = self._take()
        if c == "(":
            if self.p.startswith("?:", self.i):
                self.i += 2
            node = self._alt()
            if self._take() != ")":
                raise ValueError(f"missing ) in {self.p!r}")
            return node
        if c == "[":
            return ("set", self._class())
        if c == ".":
            return ("set", ALL - {0x0A})
        if c == "\\":
            return ("set", self._escape())
        if c in "*+?{":
            raise ValueError(f"nothing to repeat at {self.i - 1} in {self.p!r}")
        return ("set", frozenset([ord(c)]))

    def _class(self):
        negate = self._peek() == "^"
        if negate:
            self._take()
        out = set()
        first = True
        while True:
            c = self._take()
            if c == "]" and not first:
                break
            first = False
            if c == "\\":
                lo_set = self._escape()
            else:
                lo_set = frozenset([ord(c)])
            if self._peek() == "-" and self.p[self.i + 1] != "]" and len(lo_set) == 1:
                self._take()
                d = self._take()
                hi = next(iter(self._escape())) if d == "\\" else ord(d)
                lo = next(iter(lo_set))
                out.update(range(lo, hi + 1))
            else:
                out.update(lo_set)
        return frozenset(ALL - out) if negate else frozenset(out)


# ---------------------------------------------------------------- Thompson's NFA

class _NFA:
    def __init__(self):
        self.eps: list[list[int]] = []
        self.moves: list[list[tuple[frozenset, int]]] = []

    def state(self) -> int:
        self.eps.append([])
        self.moves.append([])
        return len(self.eps) - 1

    def build(self, node) -> tuple[int, int]:
        kind = node[0]
        if kind == "eps":
            s = self.state()
            return s, s
        if kind == "set":
            a, b = self.state(), self.state()
            self.moves[a].append((node[1], b))
            return a, b
        if kind == "cat":
            start, end = self.build(node[1][0])
            for part in node[1][1:]:
                s, e = self.build(part)
                self.eps[end].append(s)
                end = e
            return start, end
        if kind == "alt":
            a, b = self.state(), self.state()
            for part in node[1]:
                s, e = self.build(part)
                self.eps[a].append(s)
                self.eps[e].append(b)
            return a, b
        if kind == "rep":
            _, sub, lo, hi = node
            a = self.state()
            end = a
            for _ in range(lo):                       # the mandatory copies
                s, e = self.build(sub)
                self.eps[end].append(s)
                end = e
            if hi is None:                             # then a loop
                s, e = self.build(sub)
                self.eps[end].append(s)
                self.eps[e].append(s)
                out = self.state()
                self.eps[end].append(out)
                self.eps[e].append(out)
                return a, out
            out = self.state()
            self.eps[end].append(out)
            for _ in range(hi - lo):                   # then optional copies
                s, e = self.build(sub)
                self.eps[end].append(s)
                self.eps[e].append(out)
                end = e
            return a, out
        raise ValueError(kind)


def _closure(nfa: _NFA, states) -> frozenset:
    seen = set(states)
    stack = list(states)
    while stack:
        s = stack.pop()
        for t in nfa.eps[s]:
            if t not in seen:
                seen.add(t)
                stack.append(t)
    return frozenset(seen)


def _byte_classes(nfa: _NFA) -> list[list[int]]:
    """Bytes no move of the NFA tells apart, grouped (alphabet compression)."""
    sig = {b: [] for b in range(256)}
    for moves in nfa.moves:
        for bs, _ in moves:
            for b in bs:
                sig[b].append(id(bs))
    groups: dict = {}
    for b in range(256):
        groups.setdefault(tuple(sorted(sig[b])), []).append(b)
    return list(groups.values())


# ------------------------------------------------------- subset construction etc.

def compile_regex(pattern: str):
    """(trans[S][256] int32, accepting[S] uint8) of the minimal automaton of
    ``pattern`` (whole-string match), trimmed: every state is reachable from
    the start state 0 and can reach an accepting state; other moves are DEAD.
    An empty language gives a single non-accepting state with no moves."""
    nfa = _NFA()
    start, end = nfa.build(_Parser(pattern).parse())
    classes = _byte_classes(nfa)
    reps = [c[0] for c in classes]
    d0 = _closure(nfa, [start])
    index = {d0: 0}
    order = [d0]
    rows = []
    k = 0
    while k < len(order):
        cur = order[k]
        row = []
        for b in reps:
            nxt = set()
            for s in cur:
                for bs, t in nfa.moves[s]:
                    if b in bs:
                        nxt.add(t)
            if not nxt:
                row.append(DEAD)
                continue
            tgt = _closure(nfa, nxt)
            if tgt not in index:
                index[tgt] = len(order)
                order.append(tgt)
            row.append(index[tgt])
        rows.append(row)
        k += 1
    accepting = [end in st for st in order]
    return _finish(np.array(rows, dtype=np.int64).reshape(len(order), len(reps)), np.array(accepting),
                   classes)


def _finish(ctab: np.ndarray, accepting: np.ndarray, classes):
    """Trim, minimise (Moore) and renumber a class-compressed DFA whose start
    is state 0; expand to 256 byte columns."""
    n, C = ctab.shape
    # co-reachable: can reach an accepting state
    good = accepting.copy()
    changed = True
    while changed:
        tgt_good = np.zeros_like(ctab, dtype=bool)
        live = ctab >= 0
        tgt_good[live] = good[ctab[live]]
        new = good | tgt_good.any(axis=1)
        changed = bool((new != good).any())
        good = new
    ctab = np.where((ctab >= 0) & good[np.maximum(ctab, 0)], ctab, DEAD)
    # Moore refinement over the good states (DEAD is its own block, -1)
    block = np.where(good, accepting.astype(np.int64), -1)
    while True:
        tb = np.where(ctab >= 0, block[np.maximum(ctab, 0)], -1)
        sigs = {}
        new = np.full(n, -1, dtype=np.int64)
        for s in range(n):
            if not good[s]:
                continue
            key = (int(block[s]),) + tuple(int(x) for x in tb[s])
            new[s] = sigs.setdefault(key, len(sigs))
        if len(sigs) == len(set(block[good].tolist())):
            block = new
            break
        block = new
    if not good[0]:
        trans = np.full((1, 256), DEAD, dtype=np.int32)
        return trans, np.zeros(1, dtype=np.uint8)
    # renumber blocks in breadth-first order from the start
    nb = int(block.max()) + 1
    rep = np.zeros(nb, dtype=np.int64)
    for s in range(n - 1, -1, -1):
        if block[s] >= 0:
            rep[block[s]] = s
    number = {int(block[0]): 0}
    queue = [int(block[0])]
    q = 0
    while q < len(queue):
        bl = queue[q]
        q += 1
        for t in ctab[rep[bl]]:
            if t >= 0 and int(block[t]) not in number:
                number[int(block[t])] = len(number)
                queue.append(int(block[t]))
    S = len(number)
    trans = np.full((S, 256), DEAD, dtype=np.int32)
    acc = np.zeros(S, dtype=np.uint8)
    for bl, i in number.items():
        s = rep[bl]
        acc[i] = 1 if accepting[s] else 0
        for c, bytes_ in enumerate(classes):
            t = ctab[s, c]
            if t >= 0:
                trans[i, bytes_] = number[int(block[t])]
    return trans, acc


def scanner_regex(terminals) -> str:
    """R = r+ with r the union of the terminal regexes (the lemma of Sec.
    3.2): every non-empty sequence of terminals, each one allowed to follow
    any other."""
    body = "|".join(f"(?:{t})" for t in terminals)
    return f"(?:{body})+"


def scanner(terminals) -> tuple:
    """The scanner automaton of Sec. 3.2 for a list of terminal regexes (the
    automaton of ``scanner_regex``).  Its start state accepts only if some
    terminal matches the empty string: an empty output is not a terminal
    sequence."""
    return compile_regex(scanner_regex(terminals))

