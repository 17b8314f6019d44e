"""CPU oracle for vocabulary alignment and masked greedy decoding.

TEST INFRASTRUCTURE ONLY: the test suite, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg are the only callers.  The product path never
imports this package.  It shares no code with the HIP library; the arithmetic
lives in ``dv_oracle.c`` (plain scalar C loops), this module only marshals
numpy arrays into it.

What each function follows in the paper (DOMINO, "Guiding LLMs The Right
Way"):

* ``walk`` / ``align`` / ``align_rows``: Sec. 3.3 and Algorithm 2 -- every
  scanner state is walked through every vocabulary token; at full lookahead
  (Sec. 3.5, k = infinity) a token is allowed exactly when the walk survives.
* ``masked_step`` / ``masked_argmax``: Algorithm 1 (mask, apply, decode,
  update) with Algorithm 3's argmax over an admissible token set.
* ``align_eos``: the same table with an end-of-sequence column (Algorithm 1
  stops on EOS; Sec. 3.2 makes EOS a terminal), allowed in accepting states.
* ``masked_step_opportunistic``: opportunistic masking (Sec. 3.5, further
  optimizations) -- the model's unconstrained choice is checked first.
* ``masked_sample`` (with ``philox4x32_10``, ``ln_f32``, ``gumbel``): the
  sampled decode of Algorithm 1 at temperature T (Sec. 4 samples at T = 1)
  as a Gumbel-max draw over the allowed tokens, with counter-based noise.
* ``spec_walk`` / ``spec_verify``: the speculative chain check of Sec. 3.6 --
  how many proposed tokens the constraint admits, and greedy verification of
  the proposals against the model's logits at every proposed position.

All readings of the paper's silences (DEAD sentinel, byte alphabet, tie and
NaN rules, bitmask layout) are stated in ``dv_oracle.c``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

DEAD = -1
F32 = 0
BF16 = 1

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dv_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libdv_oracle.so")
SANITIZED_LIB_PATH = os.path.join(_HERE, "libdv_oracle_san.so")
_lib = None
BUILD_FLAGS = ("-O2", "-std=c11")
# AddressSanitizer + UndefinedBehaviorSanitizer build (host code only: gcc);
# a process loading it needs the two runtimes preloaded (sanitizer_env).
SANITIZE_FLAGS = ("-O1", "-g", "-std=c11", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                  "-fno-sanitize-recover=all")


def build(force: bool = False, out: str | None = None, defines: tuple = (), sanitize: bool = False) -> str:
    """Compile ``dv_oracle.c`` with gcc into a shared library; returns its path."""
    out = out or (SANITIZED_LIB_PATH if sanitize else _LIB_PATH)
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(_SRC):
        flags = SANITIZE_FLAGS if sanitize else BUILD_FLAGS
        cmd = ["gcc", *flags, "-shared", "-fPIC", "-o", out, _SRC, "-lm"]
        cmd += [f"-D{d}" for d in defines]
        subprocess.run(cmd, check=True)
    return out


def sanitizer_env() -> dict:
    """Environment for a child process that loads the sanitized oracle
    (``DV_ORACLE_LIBRARY``): the gcc sanitizer runtimes preloaded, leak
    checks off (the interpreter's own allocations), any report fatal."""
    runtimes = []
    for name in ("libasan.so", "libubsan.so"):
        path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True,
                              check=True).stdout.strip()
        runtimes.append(os.path.realpath(path))
    env = dict(os.environ)
    env["LD_PRELOAD"] = ":".join(runtimes)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["DV_ORACLE_LIBRARY"] = build(sanitize=True)
    return env


_i32p = ctypes.POINTER(ctypes.c_int32)
_u32p = ctypes.POINTER(ctypes.c_uint32)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_i64p = ctypes.POINTER(ctypes.c_int64)


def _bind(lib):
    lib.oracle_walk.restype = ctypes.c_int32
    lib.oracle_walk.argtypes = [_i32p, ctypes.c_int32, ctypes.c_int32, _u8p, ctypes.c_int64]
    lib.oracle_align_rows.restype = None
    lib.oracle_align_rows.argtypes = [_i32p, ctypes.c_int32, _i32p, _u8p, ctypes.c_int32,
                                      _i32p, ctypes.c_int64, _i32p, _u32p]
    lib.oracle_align_rows_eos.restype = None
    lib.oracle_align_rows_eos.argtypes = [_i32p, ctypes.c_int32, _i32p, _u8p, ctypes.c_int32,
                                          ctypes.c_void_p, ctypes.c_int32, _i32p, ctypes.c_int64,
                                          _i32p, _u32p]
    lib.oracle_align.restype = None
    lib.oracle_align.argtypes = [_i32p, ctypes.c_int32, _i32p, _u8p, ctypes.c_int32, _i32p, _u32p]
    lib.oracle_masked_argmax.restype = ctypes.c_int32
    lib.oracle_masked_argmax.argtypes = [_u32p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int32]
    lib.oracle_masked_step.restype = None
    lib.oracle_masked_step.argtypes = [_i32p, _u32p, ctypes.c_int32, ctypes.c_int32, _i32p,
                                       ctypes.c_void_p, ctypes.c_int, ctypes.c_int32,
                                       ctypes.c_int64, _i32p, _i32p]
    lib.oracle_spec_walk.restype = None
    lib.oracle_spec_walk.argtypes = [_i32p, _u32p, ctypes.c_int32, ctypes.c_int32, _i32p, _i32p,
                                     ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, _i32p, _i32p]
    lib.oracle_spec_verify.restype = None
    lib.oracle_spec_verify.argtypes = [_i32p, _u32p, ctypes.c_int32, ctypes.c_int32, _i32p, _i32p,
                                       ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int,
                                       ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, _i32p, _i32p,
                                       _i32p]
    lib.oracle_masked_step_opportunistic.restype = None
    lib.oracle_masked_step_opportunistic.argtypes = [_i32p, _u32p, ctypes.c_int32, ctypes.c_int32,
                                                     _i32p, ctypes.c_void_p, ctypes.c_int,
                                                     ctypes.c_int32, ctypes.c_int64, _i32p, _i32p,
                                                     ctypes.c_void_p]
    lib.oracle_philox4x32_10.restype = None
    lib.oracle_philox4x32_10.argtypes = [_u32p, _u32p, _u32p]
    lib.oracle_ln_f32.restype = ctypes.c_float
    lib.oracle_ln_f32.argtypes = [ctypes.c_float]
    lib.oracle_gumbel.restype = ctypes.c_float
    lib.oracle_gumbel.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32]
    lib.oracle_masked_sample.restype = None
    lib.oracle_masked_sample.argtypes = [_i32p, _u32p, ctypes.c_int32, ctypes.c_int32, _i32p,
                                         ctypes.c_void_p, ctypes.c_int, ctypes.c_int32, ctypes.c_int64,
                                         ctypes.c_float, ctypes.c_uint64, ctypes.c_uint64, _i32p, _i32p]
    lib.oracle_walk_lookups.restype = ctypes.c_int64
    lib.oracle_walk_lookups.argtypes = [_i32p, ctypes.c_int32, _i32p, _u8p, ctypes.c_int32,
                                        _i32p, ctypes.c_int64]
    lib.oracle_walk_length_hist.restype = None
    lib.oracle_walk_length_hist.argtypes = [_i32p, ctypes.c_int32, _i32p, _u8p, ctypes.c_int32,
                                            _i32p, ctypes.c_int64, _i64p, ctypes.c_int32]
    return lib


def load(path: str | None = None):
    """Load the oracle library (compiling it first if it is not built)."""
    global _lib
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _lib is None:
        chosen = os.environ.get("DV_ORACLE_LIBRARY")
        _lib = _bind(ctypes.CDLL(chosen if chosen else build()))
    return _lib


def _p(a, ct):
    return a.ctypes.data_as(ct)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def words(num_tokens: int) -> int:
    return (num_tokens + 31) // 32


def walk(trans, s: int, token: bytes, lib=None) -> int:
    lib = lib or load()
    trans = _c(trans, np.int32)
    buf = np.frombuffer(bytes(token), dtype=np.uint8) if len(token) else np.zeros(1, np.uint8)
    buf = _c(buf, np.uint8)
    return int(lib.oracle_walk(_p(trans, _i32p), trans.shape[0], int(s), _p(buf, _u8p), len(token)))


def align_rows(trans, offsets, tok_bytes, rows, lib=None):
    """(next_state[len(rows)][V], allow[len(rows)][ceil(V/32)]) for the given states."""
    lib = lib or load()
    trans = _c(trans, np.int32)
    offsets = _c(offsets, np.int32)
    tok_bytes = _c(tok_bytes if len(tok_bytes) else np.zeros(1, np.uint8), np.uint8)
    rows = _c(rows, np.int32)
    V = offsets.shape[0] - 1
    ns = np.empty((rows.shape[0], V), np.int32)
    al = np.empty((rows.shape[0], words(V)), np.uint32)
    lib.oracle_align_rows(_p(trans, _i32p), trans.shape[0], _p(offsets, _i32p),
                          _p(tok_bytes, _u8p), V, _p(rows, _i32p), rows.shape[0],
                          _p(ns, _i32p), _p(al, _u32p))
    return ns, al


def align_eos(trans, offsets, tok_bytes, accepting, eos_token: int, rows=None, lib=None):
    """Table rows with an end-of-sequence token: EOS is allowed exactly in the
    states flagged in ``accepting`` (None: no state) and keeps the state."""
    lib = lib or load()
    trans = _c(trans, np.int32)
    offsets = _c(offsets, np.int32)
    tok_bytes = _c(tok_bytes if len(tok_bytes) else np.zeros(1, np.uint8), np.uint8)
    S = trans.shape[0]
    rows = np.arange(S, dtype=np.int32) if rows is None else _c(rows, np.int32)
    acc = None if accepting is None else _c(accepting, np.uint8)
    V = offsets.shape[0] - 1
    ns = np.empty((rows.shape[0], V), np.int32)
    al = np.empty((rows.shape[0], words(V)), np.uint32)
    lib.oracle_align_rows_eos(_p(trans, _i32p), S, _p(offsets, _i32p), _p(tok_bytes, _u8p), V,
                              None if acc is None else acc.ctypes.data, int(eos_token),
                              _p(rows, _i32p), rows.shape[0], _p(ns, _i32p), _p(al, _u32p))
    return ns, al


def align(trans, offsets, tok_bytes, lib=None):
    """Full table: (next_state[S][V] int32, allow[S][ceil(V/32)] uint32)."""
    lib = lib or load()
    trans = _c(trans, np.int32)
    offsets = _c(offsets, np.int32)
    tok_bytes = _c(tok_bytes if len(tok_bytes) else np.zeros(1, np.uint8), np.uint8)
    S = trans.shape[0]
    V = offsets.shape[0] - 1
    ns = np.empty((S, V), np.int32)
    al = np.empty((S, words(V)), np.uint32)
    lib.oracle_align(_p(trans, _i32p), S, _p(offsets, _i32p), _p(tok_bytes, _u8p), V,
                     _p(ns, _i32p), _p(al, _u32p))
    return ns, al


def _logit_array(logits):
    """numpy fp32 array -> (array, F32); numpy uint16 (bf16 bit patterns) -> (array, BF16)."""
    if logits.dtype == np.float32:
        return logits, F32
    if logits.dtype == np.uint16:
        return logits, BF16
    raise TypeError(f"logits must be float32 or uint16 bf16 bits, got {logits.dtype}")


def masked_argmax(allow_row, logits_row, lib=None) -> int:
    lib = lib or load()
    allow_row = _c(allow_row, np.uint32)
    logits_row, dt = _logit_array(np.ascontiguousarray(logits_row))
    V = logits_row.shape[0]
    assert allow_row.shape[0] >= words(V)
    return int(lib.oracle_masked_argmax(_p(allow_row, _u32p), logits_row.ctypes.data, dt, V))


def masked_step(next_state, allow, states, logits, num_tokens: int | None = None, lib=None):
    """One batch step.  ``logits`` is [B][ld] (ld >= V) fp32 or bf16 bits (uint16)."""
    lib = lib or load()
    next_state = _c(next_state, np.int32)
    allow = _c(allow, np.uint32)
    states = _c(states, np.int32)
    logits, dt = _logit_array(np.ascontiguousarray(logits))
    S, V = next_state.shape
    if num_tokens is not None:
        assert num_tokens == V
    B = states.shape[0]
    ld = logits.shape[1] if B else V
    tok = np.empty(B, np.int32)
    nst = np.empty(B, np.int32)
    if B:
        lib.oracle_masked_step(_p(next_state, _i32p), _p(allow, _u32p), S, V, _p(states, _i32p),
                               logits.ctypes.data, dt, B, ld, _p(tok, _i32p), _p(nst, _i32p))
    return tok, nst


def masked_step_opportunistic(next_state, allow, states, logits, lib=None):
    """Opportunistic masking (Sec. 3.5): the unconstrained choice first, the
    mask only when it is not allowed.  Returns (token, new_state,
    unconstrained_ok[B] bool)."""
    lib = lib or load()
    next_state = _c(next_state, np.int32)
    allow = _c(allow, np.uint32)
    states = _c(states, np.int32)
    logits, dt = _logit_array(np.ascontiguousarray(logits))
    S, V = next_state.shape
    B = states.shape[0]
    ld = logits.shape[1] if B else V
    tok = np.empty(B, np.int32)
    nst = np.empty(B, np.int32)
    ok = np.zeros(B, np.uint8)
    if B:
        lib.oracle_masked_step_opportunistic(_p(next_state, _i32p), _p(allow, _u32p), S, V,
                                             _p(states, _i32p), logits.ctypes.data, dt, B, ld,
                                             _p(tok, _i32p), _p(nst, _i32p), ok.ctypes.data)
    return tok, nst, ok.astype(bool)


def philox4x32_10(ctr, key, lib=None):
    """Philox4x32-10 of a 4-word counter and a 2-word key -> 4 words."""
    lib = lib or load()
    c = np.ascontiguousarray(ctr, np.uint32)
    k = np.ascontiguousarray(key, np.uint32)
    out = np.empty(4, np.uint32)
    lib.oracle_philox4x32_10(_p(c, _u32p), _p(k, _u32p), _p(out, _u32p))
    return out


def ln_f32(x, lib=None) -> float:
    lib = lib or load()
    return float(np.float32(lib.oracle_ln_f32(float(np.float32(x)))))


def gumbel(seed: int, offset: int, row: int, token: int, lib=None) -> float:
    lib = lib or load()
    return float(np.float32(lib.oracle_gumbel(seed, offset, row, token)))


def masked_sample(next_state, allow, states, logits, inv_temperature: float, seed: int, offset: int,
                  lib=None):
    """One sampled masked step (Gumbel-max over the allowed tokens)."""
    lib = lib or load()
    next_state = _c(next_state, np.int32)
    allow = _c(allow, np.uint32)
    states = _c(states, np.int32)
    logits, dt = _logit_array(np.ascontiguousarray(logits))
    S, V = next_state.shape
    B = states.shape[0]
    ld = logits.shape[1] if B else V
    tok = np.empty(B, np.int32)
    nst = np.empty(B, np.int32)
    if B:
        lib.oracle_masked_sample(_p(next_state, _i32p), _p(allow, _u32p), S, V, _p(states, _i32p),
                                 logits.ctypes.data, dt, B, ld, float(np.float32(inv_temperature)),
                                 int(seed), int(offset), _p(tok, _i32p), _p(nst, _i32p))
    return tok, nst


def spec_walk(next_state, allow, states, proposals, lib=None):
    """Speculative chain check (Sec. 3.6): (accepted[B], final_state[B]) for
    ``proposals`` [B][s] int32 walked from ``states`` through the table."""
    lib = lib or load()
    next_state = _c(next_state, np.int32)
    allow = _c(allow, np.uint32)
    states = _c(states, np.int32)
    proposals = _c(proposals, np.int32).reshape(states.shape[0], -1)
    S, V = next_state.shape
    B, s = proposals.shape
    acc = np.empty(B, np.int32)
    fin = np.empty(B, np.int32)
    if B:
        lib.oracle_spec_walk(_p(next_state, _i32p), _p(allow, _u32p), S, V, _p(states, _i32p),
                             _p(proposals if proposals.size else np.zeros(1, np.int32), _i32p),
                             s, max(s, 1), B, _p(acc, _i32p), _p(fin, _i32p))
    return acc, fin


def spec_verify(next_state, allow, states, proposals, logits, lib=None):
    """Speculative verification with greedy decoding (Sec. 3.6, Algorithm 1).

    ``proposals`` is [B][s] int32; ``logits`` is [B][s+1][V'] (V' >= V) fp32
    or bf16 bits (uint16), any strides with a unit last one: position j of
    row b holds the logits scored after the first j proposals.  Returns
    (token[B][s+1], accepted[B], new_state[B])."""
    lib = lib or load()
    next_state = _c(next_state, np.int32)
    allow = _c(allow, np.uint32)
    states = _c(states, np.int32)
    B = states.shape[0]
    proposals = _c(proposals, np.int32).reshape(B, -1)
    s = proposals.shape[1]
    S, V = next_state.shape
    logits, dt = _logit_array(logits)
    if logits.ndim != 3 or logits.shape[0] != B or logits.shape[1] != s + 1 or logits.shape[2] < V:
        raise ValueError(f"logits must be [B][s+1][>=V], got {logits.shape}")
    if logits.strides[2] != logits.itemsize or any(x % logits.itemsize for x in logits.strides):
        logits = np.ascontiguousarray(logits)
    ld_row, ld_pos = (x // logits.itemsize for x in logits.strides[:2])
    tok = np.empty((B, s + 1), np.int32)
    acc = np.empty(B, np.int32)
    nst = np.empty(B, np.int32)
    if B:
        lib.oracle_spec_verify(_p(next_state, _i32p), _p(allow, _u32p), S, V, _p(states, _i32p),
                               _p(proposals if proposals.size else np.zeros(1, np.int32), _i32p),
                               s, max(s, 1), logits.ctypes.data, dt, ld_row, ld_pos, B,
                               _p(tok, _i32p), _p(acc, _i32p), _p(nst, _i32p))
    return tok, acc, nst


def walk_lookups(trans, offsets, tok_bytes, rows, lib=None) -> int:
    """Total DFA transitions taken over all (row state, token) walks."""
    lib = lib or load()
    trans = _c(trans, np.int32)
    offsets = _c(offsets, np.int32)
    tok_bytes = _c(tok_bytes if len(tok_bytes) else np.zeros(1, np.uint8), np.uint8)
    rows = _c(rows, np.int32)
    return int(lib.oracle_walk_lookups(_p(trans, _i32p), trans.shape[0], _p(offsets, _i32p),
                                       _p(tok_bytes, _u8p), offsets.shape[0] - 1,
                                       _p(rows, _i32p), rows.shape[0]))


def walk_length_hist(trans, offsets, tok_bytes, rows, lib=None) -> np.ndarray:
    """hist[k] = number of (row state, token) walks taking exactly k DFA
    transitions before they end or die; k runs to the longest token."""
    lib = lib or load()
    trans = _c(trans, np.int32)
    offsets = _c(offsets, np.int32)
    tok_bytes = _c(tok_bytes if len(tok_bytes) else np.zeros(1, np.uint8), np.uint8)
    rows = _c(rows, np.int32)
    max_len = int(np.diff(offsets).max()) if offsets.shape[0] > 1 else 0
    hist = np.zeros(max_len + 1, np.int64)
    lib.oracle_walk_length_hist(_p(trans, _i32p), trans.shape[0], _p(offsets, _i32p), _p(tok_bytes, _u8p),
                                offsets.shape[0] - 1, _p(rows, _i32p), rows.shape[0], _p(hist, _i64p), max_len)
    return hist


class RowCache:
    """Oracle table rows computed on demand, for full-size workloads whose whole
    table would be too slow or too large for the CPU (the rows are the same
    definition as ``align``)."""

    def __init__(self, trans, offsets, tok_bytes, lib=None):
        self.trans = _c(trans, np.int32)
        self.offsets = _c(offsets, np.int32)
        self.tok_bytes = _c(tok_bytes, np.uint8)
        self.lib = lib or load()
        self.rows: dict[int, tuple[np.ndarray, np.ndarray]] = {}

    def get(self, s: int):
        if s not in self.rows:
            ns, al = align_rows(self.trans, self.offsets, self.tok_bytes,
                                np.array([s], np.int32), lib=self.lib)
            self.rows[s] = (ns[0], al[0])
        return self.rows[s]


def masked_chain(cache: RowCache, init_state: int, logits_rows, lib=None):
    """Greedy chain of one batch row over several steps: ``logits_rows`` is
    [steps][V] for that row.  Returns (tokens[steps], states[steps + 1])."""
    lib = lib or cache.lib
    steps = logits_rows.shape[0]
    S = cache.trans.shape[0]
    toks = np.full(steps, -1, np.int32)
    sts = np.full(steps + 1, DEAD, np.int32)
    s = int(init_state) if 0 <= int(init_state) < S else DEAD
    sts[0] = s
    for k in range(steps):
        if s == DEAD:
            toks[k], sts[k + 1] = -1, DEAD
            continue
        ns_row, al_row = cache.get(s)
        t = masked_argmax(al_row, logits_rows[k], lib=lib)
        toks[k] = t
        s = DEAD if t == -1 else int(ns_row[t])
        sts[k + 1] = s
    return toks, sts


def spec_verify_rows(cache: RowCache, state: int, proposals, pos_logits, lib=None):
    """``spec_verify`` for one row of a workload whose full table is too large
    for the CPU: the table rows it needs come from ``cache`` (same definition
    as ``align``).  ``pos_logits`` is [s+1][V'] for that row.  Returns
    (token[s+1], accepted, new_state)."""
    lib = lib or cache.lib
    proposals = np.asarray(proposals, np.int32)
    s = proposals.shape[0]
    S = cache.trans.shape[0]
    V = cache.offsets.shape[0] - 1
    toks = np.full(s + 1, -1, np.int32)
    st = int(state) if 0 <= int(state) < S else DEAD
    acc, new = None, DEAD
    for j in range(s + 1):
        if st != DEAD:
            ns_row, al_row = cache.get(st)
            toks[j] = masked_argmax(al_row, pos_logits[j][:V], lib=lib)
        t = int(toks[j])
        if acc is None and (j == s or t == -1 or t != proposals[j]):
            acc, new = j, (DEAD if t == -1 else int(ns_row[t]))
        if j < s:
            p = int(proposals[j])
            if st != DEAD and 0 <= p < V and (al_row[p // 32] >> np.uint32(p % 32)) & 1:
                nx = int(ns_row[p])
                st = nx if 0 <= nx < S else DEAD
            else:
                st = DEAD
    return toks, acc, new
