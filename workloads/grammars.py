"""Automata of the paper's Appendix C grammars and a byte-level BPE vocabulary.

The paper measures constrained decoding on five grammars, listed in its
Appendix C (Sec. 4, efficiency).  Their automata are built here from the
productions as the appendix gives them, restated as byte regular
expressions:

* ``json_scanner()`` -- the basic JSON grammar is context-free (objects and
  arrays nest), so its automaton is the Sec. 3.2 scanner: R = r+ over the
  grammar's terminals ``JSON_TERMINALS`` (the six punctuation literals, the
  three keyword literals, ``string``, ``number`` and whitespace).
* ``gsm8k_json()`` -- the guided-math-reasoning (GSM8K) grammar never
  recurses from ``root`` (``object`` holds a list of ``thought`` objects and
  an answer; ``value`` and ``array`` are unreachable), so the whole grammar
  is one regular expression, ``gsm8k_regex()``, and one automaton.
* ``c_scanner()`` -- the simple C program grammar nests statements, so its
  automaton is the scanner over ``C_TERMINALS`` (keywords, punctuation and
  operators, identifiers, numbers, strings, both comment forms, whitespace).
* ``xml_scanner()`` -- the XML-with-schema grammar nests persons inside
  ``friends``: the scanner over ``XML_TERMINALS`` (the fourteen tags,
  ``NAME`` / ``NUMBER`` = ``[^<]+``, whitespace).
* ``template()`` -- the fixed RPG-character template is one regular
  expression, ``template_regex()``.  The listing declares ``WS`` without
  saying where it may occur; it is read as whitespace that may appear
  between any two tokens and around the document (how such a declared
  whitespace terminal is used in that grammar notation).

* ``bpe_vocab(V)`` -- a byte-level BPE vocabulary trained with the
  ``tokenizers`` library on a seeded synthetic corpus whose documents have
  the shapes these grammars constrain (person objects in JSON and XML,
  step-by-step JSON reasoning records, RPG character profiles, small C
  programs) plus pseudo-word prose.  All text is generated from seeded
  pseudo-words and numbers.  The text is pre-split into words with an
  optional leading space, digit groups of up to three, runs of other symbols
  with an optional leading space, and whitespace.  Its first 256 tokens are
  the 256 single bytes (every byte string stays encodable), then the learned
  tokens in merge order.  Multi-symbol tokens such as ``":``, ``",`` or
  ``</`` cross terminal boundaries: the bridge tokens the alignment exists
  for.

Only inputs are built here (no walk, no mask, no argmax).
"""
from __future__ import annotations

import functools

import numpy as np

from .regex_dfa import compile_regex, scanner, scanner_regex

_META = set("\\()[]{}.|*+?")


def lit(s: str) -> str:
    """A regular expression matching exactly the string ``s``."""
    return "".join("\\" + c if c in _META else c for c in s)


WS = r"[ \t\n]"              # the grammars' whitespace characters

# ----------------------------------------------------- basic JSON (Appendix C)
# string ::= '"' ( [^"\\] | '\' ( ["\/bfnrt] | 'u' hex hex hex hex ) )* '"'
JSON_STRING = r'"(?:[^"\\]|\\(?:["\\/bfnrt]|u[0-9a-fA-F]{4}))*"'
# number ::= '-'? ( [0-9] | [1-9] [0-9]* ) ( '.' [0-9]+ )? ( [eE] [-+]? [0-9]+ )?
JSON_NUMBER = r"-?(?:[0-9]|[1-9][0-9]*)(?:\.[0-9]+)?(?:[eE][-+]?[0-9]+)?"
JSON_TERMINALS = ([lit(c) for c in "{}[],:"] + ["true", "false", "null", JSON_STRING, JSON_NUMBER, WS + "+"])


# ------------------------------------------------- GSM8K reasoning (Appendix C)
def gsm8k_regex() -> str:
    """The guided-math-reasoning grammar as one regular expression:
    object ::= ws '{' ws '"thoughts"' ':' ws '[' ws thought (ws ',' ws thought)* ']' ws ',' ws
               '"answer"' ':' ws number ws '}' ws
    thought ::= '{' ws '"step"' ':' ws string ',' ws '"calculation"' ':' ws string ',' ws
                '"result"' ':' ws number '}' ws
    where string and number carry their trailing ws (as in the grammar) and
    ws ::= ([ \\t\\n] ws)? is any run of whitespace (possibly empty)."""
    w = WS + "*"
    string = JSON_STRING + w
    number = JSON_NUMBER + w
    thought = (r"\{" + w + lit('"step"') + ":" + w + string + "," + w + lit('"calculation"') + ":" + w + string
               + "," + w + lit('"result"') + ":" + w + number + r"\}" + w)
    return (w + r"\{" + w + lit('"thoughts"') + ":" + w + r"\[" + w + thought + f"(?:{w},{w}{thought})*" + r"\]"
            + w + "," + w + lit('"answer"') + ":" + w + number + w + r"\}" + w)


# ----------------------------------------------------- simple C (Appendix C)
C_KEYWORDS = ["int", "float", "char", "return", "while", "for", "if", "else"]
C_PUNCT = ["(", ")", "{", "}", "=", ";", "[", "]", "<=", "<", "==", "!=", ">=", ">", "+", "-", "*", "/", ","]
C_IDENTIFIER = r"[a-zA-Z_][a-zA-Z_0-9]*"
C_NUMBER = r"[0-9]+"
C_LINE_COMMENT = r"//[^\n]*\n"                      # singleLineComment ::= '//' [^\n]* '\n'
C_BLOCK_COMMENT = r"/\*(?:[^*]|\*[^/])*\*/"         # multiLineComment ::= '/*' ( [^*] | '*' [^/] )* '*/'
C_TERMINALS = ([lit(k) for k in C_KEYWORDS] + [lit(p) for p in C_PUNCT]
               + [C_IDENTIFIER, C_NUMBER, JSON_STRING, C_LINE_COMMENT, C_BLOCK_COMMENT, WS + "+"])

# ------------------------------------------------ XML with schema (Appendix C)
XML_TAGS = ["person", "name", "age", "job", "friends", "title", "salary"]
XML_TEXT = r"[^<]+"                                  # NAME ::= ( [^<] )+ ; NUMBER ::= ( [^<] )+
XML_TERMINALS = ([lit(f"<{t}>") for t in XML_TAGS] + [lit(f"</{t}>") for t in XML_TAGS]
                 + [XML_TEXT, WS + "+"])


# -------------------------------------------------- fixed template (Appendix C)
TEMPLATE_STRING = r'"[^\n\r"]+"'                     # STRING: /"[^\n\r"]+"/
TEMPLATE_NUMBER = r"[0-9]+"                          # NUMBER: /[0-9]+/


def template_regex() -> str:
    """dict: '{' content '}' with the ten pairs of the listing in order
    (id NUMBER, description the fixed string, name STRING, age NUMBER, armor
    one of three strings, weapon one of three, class / mantra STRING,
    strength NUMBER, items a list of exactly three STRINGs), each key a
    quoted literal followed by ':'; whitespace may separate any two tokens."""
    w = WS + "*"

    def pair(key, value):
        return lit(f'"{key}"') + w + ":" + w + value

    def one_of(*xs):
        return "(?:" + "|".join(lit(f'"{x}"') for x in xs) + ")"

    s, n = TEMPLATE_STRING, TEMPLATE_NUMBER
    items = r"\[" + w + s + w + "," + w + s + w + "," + w + s + w + r"\]"
    pairs = [pair("id", n), pair("description", lit('"A nimble fighter"')), pair("name", s), pair("age", n),
             pair("armor", one_of("leather", "chainmail", "plate")), pair("weapon", one_of("sword", "axe", "bow")),
             pair("class", s), pair("mantra", s), pair("strength", n), pair("items", items)]
    return w + r"\{" + w + (w + "," + w).join(pairs) + w + r"\}" + w


@functools.lru_cache(maxsize=None)
def json_scanner():
    return scanner(JSON_TERMINALS)


@functools.lru_cache(maxsize=None)
def gsm8k_json():
    return compile_regex(gsm8k_regex())


@functools.lru_cache(maxsize=None)
def c_scanner():
    return scanner(C_TERMINALS)


@functools.lru_cache(maxsize=None)
def xml_scanner():
    return scanner(XML_TERMINALS)


@functools.lru_cache(maxsize=None)
def template():
    return compile_regex(template_regex())


# Each workload automaton with the regular expression it accepts (for tests).
AUTOMATA = {
    "json-scanner": (json_scanner, lambda: scanner_regex(JSON_TERMINALS)),
    "gsm8k-json": (gsm8k_json, gsm8k_regex),
    "c-scanner": (c_scanner, lambda: scanner_regex(C_TERMINALS)),
    "xml-scanner": (xml_scanner, lambda: scanner_regex(XML_TERMINALS)),
    "template": (template, template_regex),
}

# ------------------------------------------------------------------- the corpus

_CONS = "bcdfghjklmnprstvwz"
_VOW = "aeiou"


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
    """Seeded documents of the shapes the Appendix C grammars constrain.  The
    ``*_doc`` generators of the JSON-reasoning, template, XML and C kinds
    always conform to their grammar; prose and some JSON do not need to."""

    def __init__(self, rng: np.random.Generator):
        self.rng = rng
        self.words = _words(rng, 20000)
        ranks = np.arange(1, len(self.words) + 1)
        p = 1.0 / ranks
        self.p = p / p.sum()          # Zipf frequencies
        self.buf = []

    def r(self, n) -> int:
        return int(self.rng.integers(n))

    def word(self) -> str:
        if not self.buf:              # word ranks drawn in batches
            self.buf = self.rng.choice(len(self.words), size=100_000, p=self.p).tolist()[::-1]
        return self.words[self.buf.pop()]

    def name(self) -> str:
        return " ".join(self.word().capitalize() for _ in range(1 + self.r(2)))

    def integer(self, digits=4) -> str:
        return str(int(self.rng.integers(0, 10 ** int(self.rng.integers(1, digits + 1)))))

    def number(self) -> str:
        x = self.rng.random()
        if x < 0.5:
            return self.integer(6)
        if x < 0.9:
            return f"{self.rng.uniform(-1000, 1000):.{int(self.rng.integers(1, 4))}f}"
        return f"{self.rng.uniform(1, 10):.2e}"

    def phrase(self, lo=2, hi=8) -> str:
        return " ".join(self.word() for _ in range(int(self.rng.integers(lo, hi))))

    def sentence(self) -> str:
        n = int(self.rng.integers(4, 18))
        ws = [self.word() for _ in range(n)]
        if self.rng.random() < 0.2:
            ws[self.r(n)] = self.number()
        ws[0] = ws[0].capitalize()
        parts = []
        for i, w in enumerate(ws):
            parts.append(w)
            if i < n - 1 and self.rng.random() < 0.1:
                parts[-1] += ","
        return " ".join(parts) + str(self.rng.choice([".", ".", ".", "?", "!", ":"]))

    def prose(self) -> str:
        return " ".join(self.sentence() for _ in range(int(self.rng.integers(2, 7)))) + "\n"

    # -- layout: compact or pretty-printed JSON-like text
    def _layout(self, items, open_, close, depth, pretty):
        if not items:
            return open_ + close
        if not pretty:
            return open_ + ", ".join(items) + close
        pad, inner = "  " * depth, "  " * (depth + 1)
        return open_ + "\n" + ",\n".join(inner + it for it in items) + "\n" + pad + close

    # -- basic JSON: a person, with friends
    def json_person(self, depth=0, pretty=False) -> str:
        items = [f'"name": "{self.name()}"', f'"age": {self.integer(2)}']
        if self.rng.random() < 0.6:
            items.append(f'"email": "{self.word()}@{self.word()}.com"')
        if self.rng.random() < 0.5:
            items.append(f'"married": {self.rng.choice(["true", "false", "null"])}')
        if self.rng.random() < 0.4:
            items.append(f'"address": ' + self._layout([f'"street": "{self.integer(3)} {self.name()}"',
                                                        f'"city": "{self.name()}"'], "{", "}", depth + 1, pretty))
        if depth < 2 and self.rng.random() < 0.5:
            friends = [self.json_person(depth + 2, pretty) for _ in range(self.r(3) + 1)]
            items.append('"friends": ' + self._layout(friends, "[", "]", depth + 1, pretty))
        if self.rng.random() < 0.3:
            items.append(f'"score": {self.number()}')
        return self._layout(items, "{", "}", depth, pretty)

    def json_doc(self) -> str:
        return self.json_person(pretty=self.rng.random() < 0.5) + "\n"

    # -- step-by-step JSON reasoning records (the GSM8K grammar's shape)
    def gsm8k_doc(self) -> str:
        pretty = self.rng.random() < 0.6
        thoughts = []
        for _ in range(1 + self.r(4)):
            a, b = int(self.rng.integers(1, 200)), int(self.rng.integers(1, 50))
            op = str(self.rng.choice(["+", "-", "*", "/"]))
            res = {"+": a + b, "-": a - b, "*": a * b, "/": a // b}[op]
            calc = f"{a} {op} {b} = {res}"
            thoughts.append(self._layout([f'"step": "{self.phrase(3, 10).capitalize()}"',
                                          f'"calculation": "{calc}"', f'"result": {res}'], "{", "}", 2, pretty))
        body = [f'"thoughts": ' + self._layout(thoughts, "[", "]", 1, pretty), f'"answer": {self.integer(4)}']
        return self._layout(body, "{", "}", 0, pretty) + "\n"

    # -- RPG character profiles (the fixed template's shape)
    def template_doc(self) -> str:
        pretty = self.rng.random() < 0.6
        items = [f'"id": {self.integer(4)}', '"description": "A nimble fighter"', f'"name": "{self.name()}"',
                 f'"age": {self.integer(2)}', f'"armor": "{self.rng.choice(["leather", "chainmail", "plate"])}"',
                 f'"weapon": "{self.rng.choice(["sword", "axe", "bow"])}"', f'"class": "{self.word()}"',
                 f'"mantra": "{self.phrase(2, 7).capitalize()}"', f'"strength": {self.integer(2)}',
                 '"items": [' + ", ".join(f'"{self.phrase(1, 3)}"' for _ in range(3)) + "]"]
        return self._layout(items, "{", "}", 0, pretty) + "\n"

    # -- XML persons (the XML-with-schema grammar's shape)
    def xml_person(self, depth=0) -> str:
        pad, inner = "  " * depth, "  " * (depth + 1)
        job = (f"{inner}<job>\n{inner}  <title>{self.phrase(1, 4).title()}</title>\n"
               f"{inner}  <salary>{self.integer(6)}</salary>\n{inner}</job>\n")
        out = (f"{pad}<person>\n{inner}<name>{self.name()}</name>\n{inner}<age>{self.integer(2)}</age>\n" + job)
        if depth < 2 and self.rng.random() < 0.4:
            out += f"{inner}<friends>\n" + "".join(self.xml_person(depth + 2) for _ in range(1 + self.r(2)))
            out += f"{inner}</friends>\n"
        return out + f"{pad}</person>\n"

    def xml_doc(self) -> str:
        return self.xml_person()

    # -- small C programs (the simple C grammar's statements and expressions)
    def c_expr(self, depth=0) -> str:
        x = self.rng.random()
        if depth < 2 and x < 0.35:
            return f"{self.c_expr(depth + 1)} {self.rng.choice(['+', '-', '*', '/'])} {self.c_expr(depth + 1)}"
        if depth < 2 and x < 0.45:
            return f"{self.word()}({', '.join(self.c_expr(depth + 1) for _ in range(self.r(3)))})"
        if depth < 2 and x < 0.5:
            return f"({self.c_expr(depth + 1)})"
        if x < 0.75:
            return self.word()
        if x < 0.9:
            return self.integer(3)
        return f'"{self.sentence()}\\n"'

    def c_cond(self) -> str:
        return f"{self.c_expr(1)} {self.rng.choice(['<', '<=', '==', '!=', '>=', '>'])} {self.c_expr(1)}"

    def c_stmt(self, ind, depth=0) -> str:
        x = self.rng.random()
        t = self.rng.choice(["int", "float", "char"])
        v = self.word()
        if x < 0.25:
            return f"{ind}{t} {v} = {self.c_expr()};\n"
        if x < 0.35:
            return f"{ind}{t} {v}[{self.integer(2)}];\n"
        if x < 0.5:
            return f"{ind}{v} = {self.c_expr()};\n"
        if x < 0.62:
            return f'{ind}printf("{self.sentence()}\\n", {self.word()});\n'
        if depth < 2 and x < 0.72:
            body = "".join(self.c_stmt(ind + "    ", depth + 1) for _ in range(1 + self.r(3)))
            return f"{ind}for(int {v} = 0; {v} < {self.c_expr(1)}; {v} = {v} + 1){{\n{body}{ind}}}\n"
        if depth < 2 and x < 0.8:
            body = "".join(self.c_stmt(ind + "    ", depth + 1) for _ in range(1 + self.r(3)))
            return f"{ind}while({self.c_cond()}) {{\n{body}{ind}}}\n"
        if depth < 2 and x < 0.88:
            body = "".join(self.c_stmt(ind + "    ", depth + 1) for _ in range(1 + self.r(2)))
            return f"{ind}if({self.c_cond()}){{\n{body}{ind}}}\n"
        if x < 0.94:
            return f"{ind}// {self.sentence()}\n"
        return f"{ind}/* {self.sentence()} */\n"

    def c_doc(self) -> str:
        out = ""
        for _ in range(1 + self.r(2)):
            t = self.rng.choice(["int", "float", "char"])
            par = f"{self.rng.choice(['int', 'float', 'char'])} {self.word()}" if self.rng.random() < 0.6 else ""
            body = "".join(self.c_stmt("    ") for _ in range(2 + self.r(6)))
            out += f"{t} {self.word()}({par}) {{\n{body}    return {self.c_expr()};\n}}\n"
        return out


KINDS = ("prose", "json", "gsm8k", "template", "xml", "c")
_SHARE = np.array([0.25, 0.15, 0.15, 0.15, 0.15, 0.15])


def corpus(rng: np.random.Generator, n_bytes: int, kinds=KINDS) -> list:
    """Seeded training text, about n_bytes long, as separate documents of the
    given kinds (prose, JSON persons, JSON reasoning records, RPG profiles,
    XML persons, C programs) in fixed byte shares."""
    c = _Corpus(rng)
    make = {"prose": c.prose, "json": c.json_doc, "gsm8k": c.gsm8k_doc, "template": c.template_doc,
            "xml": c.xml_doc, "c": c.c_doc}
    share = np.array([_SHARE[KINDS.index(k)] for k in kinds])
    docs = []
    sizes = np.zeros(len(kinds))
    while sizes.sum() < n_bytes:
        k = int(np.argmin(sizes / share))
        d = make[kinds[k]]()
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
