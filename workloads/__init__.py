"""Seeded synthetic inputs for vocabulary alignment and masked decoding.

This module only builds inputs: DFAs, vocabularies, initial states and logits.
It holds none of the method's arithmetic (no walk, no mask, no argmax), so the
HIP path and the CPU oracle can both consume what it produces without sharing
any code with each other.

The paper's workloads (the JSON / C / XML / template grammars of its
Appendix C, the Mistral-7B and Llama-2-13B tokenizers) are not available here;
these generators stand in for them with the shapes below.  Ten workloads:

====  ==========================  =======  ========  ======  =====  =====  ===========
 id    name                        S        V         B       steps  dtype  logits
====  ==========================  =======  ========  ======  =====  =====  ===========
 1     tiny                        16       1,000     1       64     f32    N(0, 1)
 2     regex-scale                 256      32,000    8       256    f32    N(0, 2)
 3     llm-tokenizer-scale         1,024    128,256   64      512    bf16   N(0, 3)
 4     grammar-lexer-union         8,192    128,256   256     256    bf16   N(0, 3)
 5     large-vocab-high-batch      4,096    256,000   1,024   128    bf16   N(0, 3)
 6     json-scanner-bpe32k         23       32,000    64      256    bf16   N(0, 3)
 7     gsm8k-json-bpe32k           92       32,000    64      256    bf16   N(0, 3)
 8     c-scanner-bpe32k            62       32,000    64      256    bf16   N(0, 3)
 9     xml-scanner-bpe32k          30       32,000    64      256    bf16   N(0, 3)
 10    template-bpe32k             175      32,000    64      256    bf16   N(0, 3)
====  ==========================  =======  ========  ======  =====  =====  ===========

Workloads 6-10 are the automata of the paper's five Appendix C grammars
(``workloads.grammars``): the Sec. 3.2 scanners (R = r+ over the
terminals) of the basic JSON, simple C and XML-with-schema grammars, whose
productions nest, and the GSM8K reasoning grammar and the fixed RPG
template, which are regular and compile to one automaton each; all compiled
from regular expressions by ``workloads.regex_dfa`` (minimal, trimmed:
every state can still reach acceptance).  They share one byte-level BPE
vocabulary of 32,000 tokens trained on a seeded synthetic corpus of those
grammars' document shapes (the size of the paper's two models'
vocabularies); the accepting states are the automata's own.

Readings of points the workload description leaves open:

* Byte mix is drawn per byte: printable ASCII 0x20-0x7E with probability p
  (0.95 for workloads 1-2, 0.90 for 3-5), else uniform over 0x00-0xFF.
* Geometric lengths have support {1, 2, ...} (numpy's ``geometric``) and are
  clipped at the upper bound only.
* Tokens are unique: a candidate equal to an earlier token is discarded and
  the next fresh (length, bytes) draw is used; ids are assigned in acceptance
  order.  Only 256 one-byte strings exist, so the realised length histogram
  differs from the drawn one (``length_histogram`` reports it).
* The allowed-byte subset size U[lo, hi] is clipped to the alphabet size.
* Workloads 3 and 5 use workload 2's subset size U[8, 96]; the terminals of
  workload 4 use workload 1's U[8, 64] over the 97-byte alphabet
  0x20-0x7E + \\n + \\t.
* Exactly round(0.25 * S) states are accepting (per terminal in workload 4);
  the hot path does not read them.
* N(0, sigma): sigma is the standard deviation; bf16 logits are fp32 draws
  rounded to nearest even.  Workload 4's logits are N(0, 3) in bf16.
* Initial states: workloads 1, 2 and 4 start every row in state 0; workloads
  3 and 5 draw each row's state uniformly from [0, S) (every state of these
  DFAs has at least 8 outgoing bytes, so none is the dead sentinel).
* Workload 4 is the union construction of Sec. 3.2 made deterministic: state
  0 is the shared start, followed by 40 terminal DFAs (31 of 205 states and 9
  of 204, 8,191 in all) whose transitions stay inside the terminal.  The start
  state's move on byte b is the first terminal's (lowest index) start move on
  b.  Every accepting state of a terminal also takes the start state's move
  on each byte it has no move of its own on, so one terminal can be followed
  by the next (the r+ chaining of the terminal union).
* Logits are fresh for every step and independent of the chosen tokens.
* Seeds: root seed 0 for every workload;
  ``numpy.random.SeedSequence(0, spawn_key=(workload, component, ...))`` with
  components dfa=0, vocab=1, init=2, logits=3.  Workload 4 reuses workload
  3's vocabulary stream.  Device logits use torch's generator seeded from the
  same sequence, so they are reproducible for a given torch build and device.
"""
from __future__ import annotations

import dataclasses
import functools
import hashlib

import numpy as np

DEAD = -1
PRINTABLE = np.arange(0x20, 0x7F, dtype=np.int64)          # 95 bytes
LEXER_ALPHABET = np.concatenate([PRINTABLE, np.array([0x0A, 0x09])])  # 97 bytes

COMPONENT_DFA, COMPONENT_VOCAB, COMPONENT_INIT, COMPONENT_LOGITS = 0, 1, 2, 3


@dataclasses.dataclass(frozen=True)
class Workload:
    id: int
    name: str
    S: int
    V: int
    B: int
    steps: int
    dtype: str            # "f32" or "bf16"
    sigma: float
    subset: tuple          # allowed-byte subset size U[lo, hi]
    lengths: tuple         # ("uniform", lo, hi) or ("geometric", p, hi)
    p_printable: float
    init: str              # "zero" or "uniform"
    kind: str = "random"   # "random", "union" or an Appendix C grammar (workloads.grammars.AUTOMATA)
    vocab_from: int = 0    # reuse another workload's vocabulary stream

    @property
    def words(self) -> int:
        return (self.V + 31) // 32

    @property
    def elt(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def describe(self) -> str:
        return (f"{self.name}: S={self.S} V={self.V} B={self.B} steps={self.steps} "
                f"{self.dtype} logits N(0,{self.sigma:g})")


WORKLOADS = {
    1: Workload(1, "tiny", 16, 1000, 1, 64, "f32", 1.0, (8, 64), ("uniform", 1, 8), 0.95, "zero"),
    2: Workload(2, "regex-scale", 256, 32000, 8, 256, "f32", 2.0, (8, 96), ("geometric", 0.25, 16),
                0.95, "zero"),
    3: Workload(3, "llm-tokenizer-scale", 1024, 128256, 64, 512, "bf16", 3.0, (8, 96),
                ("geometric", 0.2, 32), 0.90, "uniform"),
    4: Workload(4, "grammar-lexer-union", 8192, 128256, 256, 256, "bf16", 3.0, (8, 64),
                ("geometric", 0.2, 32), 0.90, "zero", kind="union", vocab_from=3),
    5: Workload(5, "large-vocab-high-batch", 4096, 256000, 1024, 128, "bf16", 3.0, (8, 96),
                ("geometric", 0.2, 48), 0.90, "uniform"),
    6: Workload(6, "json-scanner-bpe32k", 23, 32000, 64, 256, "bf16", 3.0, (0, 0), ("bpe",), 1.0, "zero",
                kind="json-scanner"),
    7: Workload(7, "gsm8k-json-bpe32k", 92, 32000, 64, 256, "bf16", 3.0, (0, 0), ("bpe",), 1.0, "zero",
                kind="gsm8k-json", vocab_from=6),
    8: Workload(8, "c-scanner-bpe32k", 62, 32000, 64, 256, "bf16", 3.0, (0, 0), ("bpe",), 1.0, "zero",
                kind="c-scanner", vocab_from=6),
    9: Workload(9, "xml-scanner-bpe32k", 30, 32000, 64, 256, "bf16", 3.0, (0, 0), ("bpe",), 1.0, "zero",
                kind="xml-scanner", vocab_from=6),
    10: Workload(10, "template-bpe32k", 175, 32000, 64, 256, "bf16", 3.0, (0, 0), ("bpe",), 1.0, "zero",
                 kind="template", vocab_from=6),
}


def rng_for(workload: int, component: int, *extra: int) -> np.random.Generator:
    ss = np.random.SeedSequence(0, spawn_key=(workload, component) + tuple(extra))
    return np.random.Generator(np.random.PCG64(ss))


def seed_int(workload: int, component: int, *extra: int) -> int:
    ss = np.random.SeedSequence(0, spawn_key=(workload, component) + tuple(extra))
    return int(ss.generate_state(1, dtype=np.uint64)[0] & 0x7FFF_FFFF_FFFF_FFFF)


# --------------------------------------------------------------------------- DFAs

def random_dfa(rng: np.random.Generator, S: int, subset: tuple, alphabet=PRINTABLE):
    """Random byte DFA: each state moves on a random subset of ``alphabet``
    (size U[lo, hi], clipped to the alphabet) to uniform random states; every
    other byte goes to DEAD.  Returns (trans[S][256] int32, accepting[S] uint8)."""
    trans = np.full((S, 256), DEAD, dtype=np.int32)
    lo, hi = subset
    hi = min(hi, alphabet.shape[0])
    lo = min(lo, hi)
    for s in range(S):
        k = int(rng.integers(lo, hi + 1))
        chosen = rng.choice(alphabet, size=k, replace=False)
        trans[s, chosen] = rng.integers(0, S, size=k)
    accepting = np.zeros(S, dtype=np.uint8)
    accepting[rng.choice(S, size=int(round(0.25 * S)), replace=False)] = 1
    return trans, accepting


def union_dfa(rng: np.random.Generator, n_terminals: int = 40, total_states: int = 8192,
              subset: tuple = (8, 64), alphabet=LEXER_ALPHABET):
    """Shared start state 0 plus ``n_terminals`` terminal DFAs with chaining
    from accepting states back through the start state's moves."""
    inner = total_states - 1
    base, extra = divmod(inner, n_terminals)
    # 8,191 = 31 * 205 + 9 * 204: the first ``extra`` terminals get one more state
    sizes = [base + 1 if i < extra else base for i in range(n_terminals)]
    trans = np.full((total_states, 256), DEAD, dtype=np.int32)
    accepting = np.zeros(total_states, dtype=np.uint8)
    starts = []
    first = 1
    for n in sizes:
        t, acc = random_dfa(rng, n, subset, alphabet)
        block = np.where(t >= 0, t + first, DEAD)
        trans[first:first + n] = block
        accepting[first:first + n] = acc
        starts.append(first)
        first += n
    # start state: first terminal (lowest index) with a move on the byte wins
    for b in range(256):
        for st in starts:
            if trans[st, b] != DEAD:
                trans[0, b] = trans[st, b]
                break
    # chaining: accepting states take the start state's moves where they have none
    acc_idx = np.nonzero(accepting)[0]
    sub = trans[acc_idx]
    trans[acc_idx] = np.where(sub == DEAD, trans[0][None, :], sub)
    return trans, accepting


# ----------------------------------------------------------------------- vocabulary

def _draw_lengths(rng: np.random.Generator, spec: tuple, n: int) -> np.ndarray:
    if spec[0] == "uniform":
        return rng.integers(spec[1], spec[2] + 1, size=n)
    if spec[0] == "geometric":
        return np.minimum(rng.geometric(spec[1], size=n), spec[2])
    raise ValueError(spec)


def random_vocab(rng: np.random.Generator, V: int, lengths: tuple, p_printable: float):
    """V unique byte-string tokens in CSR form: (offsets[V+1] int32, bytes uint8)."""
    seen: set = set()
    toks: list = []
    while len(toks) < V:
        n = 2 * (V - len(toks)) + 64
        lens = _draw_lengths(rng, lengths, n)
        total = int(lens.sum())
        printable = rng.random(total) < p_printable
        pb = rng.integers(0x20, 0x7F, size=total)
        ab = rng.integers(0, 256, size=total)
        raw = np.where(printable, pb, ab).astype(np.uint8).tobytes()
        pos = 0
        for L in lens.tolist():
            tok = raw[pos:pos + L]
            pos += L
            if tok in seen:
                continue
            seen.add(tok)
            toks.append(tok)
            if len(toks) == V:
                break
    return vocab_from_tokens(toks)


def vocab_from_tokens(tokens) -> tuple:
    """CSR (offsets, bytes) of a list of byte strings, in list order."""
    lens = np.fromiter((len(t) for t in tokens), dtype=np.int64, count=len(tokens))
    offsets = np.zeros(len(tokens) + 1, dtype=np.int64)
    np.cumsum(lens, out=offsets[1:])
    assert offsets[-1] < 2**31
    data = np.frombuffer(b"".join(bytes(t) for t in tokens), dtype=np.uint8).copy()
    return offsets.astype(np.int32), data


def tokens_of(offsets, data):
    return [bytes(data[offsets[i]:offsets[i + 1]]) for i in range(len(offsets) - 1)]


def length_histogram(offsets) -> dict:
    lens = np.diff(np.asarray(offsets, dtype=np.int64))
    vals, counts = np.unique(lens, return_counts=True)
    return {int(v): int(c) for v, c in zip(vals, counts)}


# ------------------------------------------------------------------------ workloads

@functools.lru_cache(maxsize=8)
def dfa(workload: int):
    """(trans[S][256] int32, accepting[S] uint8) of a workload; start state 0."""
    w = WORKLOADS[workload]
    rng = rng_for(workload, COMPONENT_DFA)
    if w.kind == "union":
        trans, acc = union_dfa(rng, 40, w.S, w.subset, LEXER_ALPHABET)
    elif w.kind == "random":
        trans, acc = random_dfa(rng, w.S, w.subset, PRINTABLE)
    else:
        from . import grammars

        trans, acc = (a.copy() for a in grammars.AUTOMATA[w.kind][0]())
        if trans.shape[0] != w.S:
            raise RuntimeError(f"{w.name}: automaton has {trans.shape[0]} states, {w.S} expected")
    trans.setflags(write=False)
    acc.setflags(write=False)
    return trans, acc


def vocab(workload: int):
    """(offsets[V+1] int32, bytes uint8) of a workload."""
    w = WORKLOADS[workload]
    return _vocab_of(w.vocab_from or workload)


@functools.lru_cache(maxsize=8)
def _vocab_of(src: int):
    ws = WORKLOADS[src]
    if ws.lengths[0] == "bpe":
        from . import grammars

        offsets, data = vocab_from_tokens(grammars.bpe_vocab(rng_for(src, COMPONENT_VOCAB), ws.V))
    else:
        offsets, data = random_vocab(rng_for(src, COMPONENT_VOCAB), ws.V, ws.lengths, ws.p_printable)
    offsets.setflags(write=False)
    data.setflags(write=False)
    return offsets, data


def init_states(workload: int, batch: int | None = None) -> np.ndarray:
    w = WORKLOADS[workload]
    B = w.B if batch is None else batch
    if w.init == "zero":
        return np.zeros(B, dtype=np.int32)
    return rng_for(workload, COMPONENT_INIT).integers(0, w.S, size=B).astype(np.int32)


def logits(workload: int, step: int, device="cpu", batch: int | None = None, torch_dtype=None):
    """One step's [B][V] logits as a torch tensor on ``device`` (seeded per
    (workload, step)); fp32 N(0, sigma), rounded to bf16 for bf16 workloads."""
    import torch

    w = WORKLOADS[workload]
    B = w.B if batch is None else batch
    g = torch.Generator(device=device)
    g.manual_seed(seed_int(workload, COMPONENT_LOGITS, step))
    x = torch.randn((B, w.V), generator=g, device=device, dtype=torch.float32)
    x.mul_(w.sigma)
    dt = torch_dtype or (torch.float32 if w.dtype == "f32" else torch.bfloat16)
    return x.to(dt)


def logits_all(workload: int, device="cpu", steps: int | None = None, batch: int | None = None):
    """[steps][B][V] logits, each step drawn as ``logits(workload, step)``."""
    import torch

    w = WORKLOADS[workload]
    n = w.steps if steps is None else steps
    B = w.B if batch is None else batch
    dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    out = torch.empty((n, B, w.V), dtype=dt, device=device)
    for k in range(n):
        out[k].copy_(logits(workload, k, device=device, batch=B))
    return out


def sha256(a) -> str:
    a = np.ascontiguousarray(a)
    return hashlib.sha256(a.view(np.uint8).tobytes()).hexdigest()


# --------------------------------------------------------- the paper's worked examples

def dfa_from_spec(num_states: int, moves) -> np.ndarray:
    """trans[S][256] from a list of (from_state, bytes_string, to_state)."""
    trans = np.full((num_states, 256), DEAD, dtype=np.int32)
    for src, chars, dst in moves:
        for ch in chars.encode("latin-1"):
            trans[src, ch] = dst
    return trans
