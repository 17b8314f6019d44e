"""Scanner automata of real grammars and a byte-level BPE vocabulary.

Stand-ins for the paper's grammar workloads (Sec. 4: JSON, C; Appendix C)
and its models' 32,000-token vocabularies, none of which are available here:

* ``JSON_TERMINALS`` -- the lexical terminals of JSON (whitespace,
  punctuation, string, number, true / false / null), written from the JSON
  grammar of RFC 8259; ``json_scanner()`` is the Sec. 3.2 scanner over them
  (any terminal may follow any other).
* ``json_schema()`` -- one fixed JSON object shape (keys, value types, a list
  of strings) as a single regular expression: the kind of constraint that
  schema-driven generation produces, with every separator and key forced.
* ``C_TERMINALS`` / ``c_scanner()`` -- the lexical terminals of C
  (identifiers and keywords, integer and floating constants, character and
  string literals, comments, preprocessor lines, punctuators), written from
  the C language's lexical grammar.
* ``bpe_vocab(V)`` -- a byte-level BPE vocabulary trained with the
  ``tokenizers`` library on a seeded synthetic corpus (pseudo-word prose,
  JSON documents, C-like code), pre-split into words with an optional
  leading space, digit groups of up to three, runs of other symbols with an
  optional leading space, and whitespace.  Its first 256 tokens are the 256
  single bytes (every byte string stays encodable), then the learned tokens
  in merge order.  Multi-symbol tokens such as ``":``, ``",`` or ``});``
  cross terminal boundaries: the bridge tokens the alignment exists for.

Only inputs are built here (no walk, no mask, no argmax).
"""
from __future__ import annotations

import functools

import numpy as np

from .regex_dfa import compile_regex, scanner

WS = r"[ \t\n\r]"

JSON_TERMINALS = [
    WS + "+",
    r"[{}\[\]:,]",
    r'"(?:[^"\\\x00-\x1f]|\\(?:["\\/bfnrt]|u[0-9a-fA-F]{4}))*"',
    r"-?(?:0|[1-9][0-9]*)(?:\.[0-9]+)?(?:[eE][+-]?[0-9]+)?",
    r"true|false|null",
]

_JSTR = JSON_TERMINALS[2]
_JNUM = JSON_TERMINALS[3]
_JINT = r"-?(?:0|[1-9][0-9]*)"

C_TERMINALS = [
    r"[ \t\n\r\f\v]+",
    r"//[^\n]*",
    r"/\*(?:[^*]|\*+[^*/])*\*+/",
    r"#[^\n]*",
    r"[A-Za-z_][A-Za-z0-9_]*",
    r"(?:0[xX][0-9a-fA-F]+|0[0-7]*|[1-9][0-9]*)(?:[uU](?:l|L|ll|LL)?|(?:l|L|ll|LL)[uU]?)?",
    r"(?:[0-9]+\.[0-9]*|\.[0-9]+)(?:[eE][+-]?[0-9]+)?[fFlL]?|[0-9]+[eE][+-]?[0-9]+[fFlL]?",
    r"'(?:[^'\\\n]|\\.)+'",
    r'"(?:[^"\\\n]|\\.)*"',
    r"->|\+\+|--|<<=?|>>=?|[<>=!]=|&&|\|\||[-+*/%&|^]=|\.\.\.|[{}\[\]();,.?:~!<>=+\-*/%&|^]",
]


def _kv(key: str, value: str) -> str:
    w = WS + "*"
    return f'"{key}"{w}:{w}{value}'


def json_schema_regex() -> str:
    """{"id": int, "name": string, "price": number, "tags": [string, ...],
    "enabled": true|false|null}, keys in this order, any JSON whitespace."""
    w = WS + "*"
    tags = rf"\[{w}(?:{_JSTR}(?:{w},{w}{_JSTR})*)?{w}\]"
    fields = [_kv("id", _JINT), _kv("name", _JSTR), _kv("price", _JNUM), _kv("tags", tags),
              _kv("enabled", "(?:true|false|null)")]
    return r"\{" + w + f"{w},{w}".join(fields) + w + r"\}"


@functools.lru_cache(maxsize=None)
def json_scanner():
    return scanner(JSON_TERMINALS)


@functools.lru_cache(maxsize=None)
def json_schema():
    return compile_regex(json_schema_regex())


@functools.lru_cache(maxsize=None)
def c_scanner():
    return scanner(C_TERMINALS)


# ------------------------------------------------------------------- the corpus

_CONS = "bcdfghjklmnprstvwz"
_VOW = "aeiou"
_C_TYPES = ["int", "char", "float", "double", "void", "long", "unsigned", "short", "size_t", "struct node"]
_C_OPS = ["+", "-", "*", "/", "%", "<<", ">>", "&", "|", "^", "==", "!=", "<", ">", "<=", ">=", "&&", "||"]


def _words(rng: np.random.Generator, n: int) -> list:
    out = []
    seen = set()
    while len(out) < n:
        k = int(rng.integers(1, 5))
        w = "".join(_CONS[rng.integers(len(_CONS))] + _VOW[rng.integers(len(_VOW))] for _ in range(k))
        if rng.random() < 0.3:
            w += _CONS[rng.integers(len(_CONS))]
        if w not in seen:
            seen.add(w)
            out.append(w)
    return out


class _Corpus:
    def __init__(self, rng: np.random.Generator):
        self.rng = rng
        self.words = _words(rng, 20000)
        ranks = np.arange(1, len(self.words) + 1)
        p = 1.0 / ranks
        self.p = p / p.sum()          # Zipf frequencies
        self.buf = []

    def word(self) -> str:
        if not self.buf:              # word ranks drawn in batches
            self.buf = self.rng.choice(len(self.words), size=100_000, p=self.p).tolist()[::-1]
        return self.words[self.buf.pop()]

    def number(self) -> str:
        r = self.rng.random()
        if r < 0.5:
            return str(int(self.rng.integers(0, 10 ** int(self.rng.integers(1, 7)))))
        if r < 0.9:
            return f"{self.rng.uniform(-1000, 1000):.{int(self.rng.integers(0, 4))}f}"
        return f"{self.rng.uniform(0, 10):.2e}"

    def sentence(self) -> str:
        n = int(self.rng.integers(4, 18))
        ws = [self.word() for _ in range(n)]
        if self.rng.random() < 0.2:
            ws[int(self.rng.integers(n))] = self.number()
        ws[0] = ws[0].capitalize()
        parts = []
        for i, w in enumerate(ws):
            parts.append(w)
            if i < n - 1 and self.rng.random() < 0.1:
                parts[-1] += ","
        return " ".join(parts) + str(self.rng.choice([".", ".", ".", "?", "!", ":"]))

    def prose(self) -> str:
        return " ".join(self.sentence() for _ in range(int(self.rng.integers(2, 7)))) + "\n"

    def json_value(self, depth: int) -> str:
        r = self.rng.random()
        if depth < 3 and r < 0.15:
            return self.json_object(depth + 1)
        if depth < 3 and r < 0.3:
            return "[" + ", ".join(self.json_value(depth + 1) for _ in range(int(self.rng.integers(0, 5)))) + "]"
        if r < 0.6:
            return '"' + " ".join(self.word() for _ in range(int(self.rng.integers(1, 4)))) + '"'
        if r < 0.85:
            return self.number()
        return str(self.rng.choice(["true", "false", "null"]))

    def json_object(self, depth: int = 0) -> str:
        n = int(self.rng.integers(1, 6))
        items = [f'"{self.word()}": {self.json_value(depth)}' for _ in range(n)]
        return "{" + ", ".join(items) + "}"

    def json_doc(self) -> str:
        if self.rng.random() < 0.5:  # the schema's shape
            tags = ", ".join(f'"{self.word()}"' for _ in range(int(self.rng.integers(0, 5))))
            name = " ".join(self.word() for _ in range(int(self.rng.integers(1, 4))))
            doc = (f'{{"id": {int(self.rng.integers(0, 10**6))}, "name": "{name}", "price": {self.number()}, '
                   f'"tags": [{tags}], "enabled": {self.rng.choice(["true", "false", "null"])}}}')
        else:
            doc = self.json_object()
        if self.rng.random() < 0.4:  # pretty-printed
            doc = doc.replace("{", "{\n  ").replace(", ", ",\n  ").replace("}", "\n}")
        return doc + "\n"

    def c_expr(self, depth: int = 0) -> str:
        r = self.rng.random()
        if depth < 2 and r < 0.35:
            return f"{self.c_expr(depth + 1)} {self.rng.choice(_C_OPS)} {self.c_expr(depth + 1)}"
        if depth < 2 and r < 0.45:
            return f"{self.word()}({', '.join(self.c_expr(depth + 1) for _ in range(int(self.rng.integers(0, 3))))})"
        if r < 0.7:
            return self.word()
        if r < 0.8:
            return f"0x{int(self.rng.integers(0, 65536)):x}"
        if r < 0.9:
            return self.number().lstrip("-")
        return f"'{self.rng.choice(list('abcxyz0'))}'"

    def c_stmt(self, indent: str) -> str:
        r = self.rng.random()
        if r < 0.4:
            return f"{indent}{self.word()} = {self.c_expr()};\n"
        if r < 0.55:
            return f"{indent}if ({self.c_expr()}) {{\n{indent}    {self.word()}++;\n{indent}}}\n"
        if r < 0.65:
            v = self.word()
            return f"{indent}for (int {v} = 0; {v} < {self.c_expr()}; {v}++) {{\n{indent}    {self.c_stmt('').strip()}\n{indent}}}\n"
        if r < 0.75:
            return f'{indent}printf("{self.sentence()}\\n", {self.word()});\n'
        if r < 0.85:
            return f"{indent}// {self.sentence()}\n"
        return f"{indent}return {self.c_expr()};\n"

    def c_func(self) -> str:
        head = ""
        if self.rng.random() < 0.3:
            head = f"#include <{self.word()}.h>\n#define {self.word().upper()} {self.number().lstrip('-')}\n"
        if self.rng.random() < 0.3:
            head += f"/* {self.sentence()} */\n"
        args = ", ".join(f"{self.rng.choice(_C_TYPES)} {self.word()}" for _ in range(int(self.rng.integers(0, 4))))
        body = "".join(self.c_stmt("    ") for _ in range(int(self.rng.integers(2, 8))))
        return f"{head}{self.rng.choice(_C_TYPES)} {self.word()}({args}) {{\n{body}}}\n"


def corpus(rng: np.random.Generator, n_bytes: int) -> list:
    """Seeded training text, about n_bytes long: prose, JSON and C-like code
    in a 4 : 3 : 3 byte mix, as separate documents."""
    c = _Corpus(rng)
    docs = []
    sizes = [0, 0, 0]
    share = np.array([0.4, 0.3, 0.3])
    while sum(sizes) < n_bytes:
        k = int(np.argmin(np.array(sizes) / share))
        d = (c.prose, c.json_doc, c.c_func)[k]()
        sizes[k] += len(d)
        docs.append(d)
    return docs


# The pre-split of the training text: a word with an optional leading space,
# a group of up to three digits, a run of other symbols with an optional
# leading space, or whitespace.
PRESPLIT = r" ?[A-Za-z]+| ?[0-9]{1,3}| ?[^\sA-Za-z0-9]+|\s+"


def bpe_vocab(rng: np.random.Generator, V: int, n_bytes: int = 8_000_000) -> list:
    """V byte strings: the 256 single bytes, then BPE tokens in merge order."""
    from tokenizers import Regex, Tokenizer, models, pre_tokenizers, trainers

    docs = corpus(rng, n_bytes)
    tok = Tokenizer(models.BPE())
    tok.pre_tokenizer = pre_tokenizers.Split(Regex(PRESPLIT), behavior="isolated")
    alphabet = [chr(c) for c in range(0x20, 0x7F)] + ["\n", "\t"]
    trainer = trainers.BpeTrainer(vocab_size=V + 64, initial_alphabet=alphabet, min_frequency=2,
                                  show_progress=False)
    tok.train_from_iterator(docs, trainer)
    learned = sorted(tok.get_vocab().items(), key=lambda kv: kv[1])
    out = [bytes([b]) for b in range(256)]
    seen = set(out)
    for s, _ in learned:
        t = s.encode("ascii")
        if t not in seen:
            seen.add(t)
            out.append(t)
        if len(out) == V:
            break
    if len(out) < V:
        raise RuntimeError(f"BPE training produced {len(out)} tokens, {V} wanted")
    return out
