"""Vocabulary alignment and masked greedy decoding on MI355X (gfx950).

Thin Python binding over ``libdv.so`` (C ABI in ``include/dv.h``).  It only
marshals torch tensors into device pointers and a HIP stream; every step of
the computation runs in the library's HIP kernels.  There is no CPU fallback:
importing this package fails if the library is not built.

    next_state, allow = align(trans, offsets, tok_bytes)
    token, new_state = masked_step(next_state, allow, states, logits)

``align`` is the offline vocabulary alignment of the DOMINO paper (Sec. 3.3,
Algorithm 2, walked to full depth as in Sec. 3.5) for a byte-level DFA;
``masked_step`` is one step of its Algorithm 1 with greedy decoding;
``spec_walk`` / ``spec_verify`` are the speculative chain check of Sec. 3.6.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = ["align", "validate_vocab", "masked_step", "masked_step_noalloc", "masked_sample", "spec_walk", "spec_verify", "align_workspace_bytes",
           "masked_step_workspace_bytes", "masked_sample_workspace_bytes", "spec_verify_workspace_bytes",
           "step_workspace", "sample_workspace", "spec_workspace", "DvError", "DEAD", "library_path", "lib"]

DEAD = -1
DV_OK = 0
DV_F32, DV_BF16 = 0, 1

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.environ.get("DV_LIBRARY", os.path.join(_HERE, "libdv.so"))


class DvError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(
            f"libdv.so not found at {_LIB_PATH}: build it first "
            "(python -c 'import __graft_entry__ as g; g.build()' or "
            "python paper_2403_06988_amd/_build.py); there is no CPU fallback")
    lib = ctypes.CDLL(_LIB_PATH)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.dv_version.restype = i32
    lib.dv_version.argtypes = []
    lib.dv_status_string.restype = ctypes.c_char_p
    lib.dv_status_string.argtypes = [i32]
    lib.dv_last_error.restype = ctypes.c_char_p
    lib.dv_last_error.argtypes = []
    lib.dv_align_workspace_bytes.restype = sz
    lib.dv_align_workspace_bytes.argtypes = [i32, i32]
    lib.dv_align.restype = ctypes.c_int
    lib.dv_align.argtypes = [vp, i32, vp, vp, i32, vp, vp, vp, sz, vp]
    lib.dv_validate_vocab.restype = ctypes.c_int
    lib.dv_validate_vocab.argtypes = [vp, i32, i64, vp, vp]
    lib.dv_align_eos.restype = ctypes.c_int
    lib.dv_align_eos.argtypes = [vp, i32, vp, vp, i32, vp, i32, vp, vp, vp, sz, vp]
    lib.dv_masked_step_workspace_bytes.restype = sz
    lib.dv_masked_step_workspace_bytes.argtypes = [i32, i32]
    lib.dv_masked_step.restype = ctypes.c_int
    lib.dv_masked_step.argtypes = [vp, vp, i32, i32, vp, vp, i32, i32, i64, vp, vp, vp, sz, vp]
    lib.dv_masked_step_noalloc.restype = ctypes.c_int
    lib.dv_masked_step_noalloc.argtypes = [vp, vp, i32, i32, vp, vp, i32, i32, i64, vp, vp, vp]
    lib.dv_masked_step_opportunistic.restype = ctypes.c_int
    lib.dv_masked_step_opportunistic.argtypes = [vp, vp, i32, i32, vp, vp, i32, i32, i64, vp, vp, vp, sz,
                                                 vp]
    lib.dv_masked_sample_workspace_bytes.restype = sz
    lib.dv_masked_sample_workspace_bytes.argtypes = [i32, i32]
    lib.dv_masked_sample.restype = ctypes.c_int
    lib.dv_masked_sample.argtypes = [vp, vp, i32, i32, vp, vp, i32, i32, i64, ctypes.c_float, ctypes.c_uint64,
                                     ctypes.c_uint64, vp, vp, vp, sz, vp]
    lib.dv_spec_walk.restype = ctypes.c_int
    lib.dv_spec_walk.argtypes = [vp, vp, i32, i32, vp, vp, i32, i64, i32, vp, vp, vp]
    lib.dv_spec_verify_workspace_bytes.restype = sz
    lib.dv_spec_verify_workspace_bytes.argtypes = [i32, i32, i32]
    lib.dv_spec_verify.restype = ctypes.c_int
    lib.dv_spec_verify.argtypes = [vp, vp, i32, i32, vp, vp, i32, i64, vp, i32, i64, i64, i32, vp, vp, vp,
                                   vp, sz, vp]
    return lib


lib = _load()
library_path = _LIB_PATH


def _check(status: int, what: str):
    if status != DV_OK:
        name = lib.dv_status_string(status).decode()
        detail = lib.dv_last_error().decode()
        raise DvError(status, f"{what}: {name}: {detail}")


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def _stream(stream, device) -> int:
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _want(t, name, dtype, device=None):
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def align_workspace_bytes(num_states: int, num_tokens: int) -> int:
    return int(lib.dv_align_workspace_bytes(num_states, num_tokens))


def masked_step_workspace_bytes(batch: int, num_tokens: int) -> int:
    return int(lib.dv_masked_step_workspace_bytes(batch, num_tokens))


def validate_vocab(offsets, tok_bytes, stream=None) -> int:
    """dv_validate_vocab: -1 when offsets [V+1] is a valid CSR layout over
    tok_bytes (starts at 0, non-decreasing, ends within tok_bytes), else the
    first index at which it is not.  Synchronizes the stream."""
    dev = offsets.device
    _want(offsets, "offsets", torch.int32, dev)
    _want(tok_bytes, "tok_bytes", torch.uint8, dev)
    out = torch.empty(1, dtype=torch.int32, device=dev)
    st = lib.dv_validate_vocab(_ptr(offsets), offsets.numel() - 1, tok_bytes.numel(), _ptr(out),
                               _stream(stream, dev))
    _check(st, "dv_validate_vocab")
    return int(out.item())


def align(trans, offsets, tok_bytes, next_state=None, allow=None, workspace=None, stream=None,
          accepting=None, eos_token=None, validate=True):
    """Alignment table of a byte DFA and a vocabulary (device tensors).

    trans [S][256] int32, offsets [V+1] int32, tok_bytes [offsets[V]] uint8.
    With ``eos_token`` (and optionally ``accepting`` [S] uint8), that token is
    allowed exactly in accepting states (dv_align_eos).  ``validate``: check
    the vocabulary's layout first (validate_vocab; one synchronization) and
    raise ValueError if it is malformed.
    Returns (next_state [S][V] int32, allow [S][ceil(V/32)] int32 holding the
    uint32 bit pattern)."""
    dev = trans.device
    _want(trans, "trans", torch.int32, dev)
    _want(offsets, "offsets", torch.int32, dev)
    _want(tok_bytes, "tok_bytes", torch.uint8, dev)
    if validate and offsets.numel() >= 2:
        bad = validate_vocab(offsets, tok_bytes, stream)
        if bad >= 0:
            raise ValueError(f"malformed vocabulary: offsets break the CSR layout at index {bad}")
    if trans.dim() != 2 or trans.shape[1] != 256:
        raise ValueError("trans must be [S][256]")
    S, V = trans.shape[0], offsets.shape[0] - 1
    Wd = (V + 31) // 32
    if next_state is None:
        next_state = torch.empty((S, V), dtype=torch.int32, device=dev)
    if allow is None:
        allow = torch.empty((S, Wd), dtype=torch.int32, device=dev)
    _want(next_state, "next_state", torch.int32, dev)
    _want(allow, "allow", torch.int32, dev)
    if next_state.numel() != S * V or allow.numel() != S * Wd:
        raise ValueError("next_state / allow have the wrong size")
    need = align_workspace_bytes(S, max(V, 1))
    workspace, ws_bytes = _workspace(workspace, need, dev,
                                     lambda: torch.empty(max(need, 1), dtype=torch.uint8, device=dev))
    bytes_ptr = _ptr(tok_bytes) if tok_bytes.numel() else None
    if eos_token is None:
        if accepting is not None:
            raise ValueError("accepting is only meaningful with eos_token")
        st = lib.dv_align(_ptr(trans), S, _ptr(offsets), bytes_ptr, V, _ptr(next_state), _ptr(allow),
                          _ptr(workspace), ws_bytes, _stream(stream, dev))
        _check(st, "dv_align")
    else:
        if accepting is not None:
            _want(accepting, "accepting", torch.uint8, dev)
            if accepting.numel() != S:
                raise ValueError("accepting must have one flag per state")
        st = lib.dv_align_eos(_ptr(trans), S, _ptr(offsets), bytes_ptr, V, _ptr(accepting),
                              int(eos_token), _ptr(next_state), _ptr(allow), _ptr(workspace),
                              ws_bytes, _stream(stream, dev))
        _check(st, "dv_align_eos")
    return next_state, allow


def step_workspace(batch: int, num_tokens: int, device) -> torch.Tensor:
    """A zero-filled workspace for ``masked_step`` with up to ``batch`` rows;
    every call leaves it zero, so calls ordered on one stream can reuse it."""
    n = masked_step_workspace_bytes(batch, num_tokens)
    return torch.zeros(max(n, 1), dtype=torch.uint8, device=device)


def _out(t, name, n, dev):
    """A caller-supplied int32 output of n elements (or a new one)."""
    if t is None:
        return torch.empty(n, dtype=torch.int32, device=dev)
    _want(t, name, torch.int32, dev)
    if t.numel() != n:
        raise ValueError(f"{name} must have {n} elements, got {t.numel()}")
    return t


def _workspace(ws, need, dev, make):
    """A caller-supplied workspace of at least ``need`` bytes (or a new one);
    returns (tensor, its size in bytes)."""
    if ws is None:
        ws = make()
    if not ws.is_cuda or ws.device != dev:
        raise ValueError(f"workspace must be a device tensor on {dev}")
    if not ws.is_contiguous():
        raise ValueError("workspace must be contiguous")
    nbytes = ws.numel() * ws.element_size()
    if nbytes < need:
        raise ValueError(f"workspace holds {nbytes} bytes, {need} needed")
    return ws, nbytes


def _step_args(next_state, allow, states, logits):
    """Checks shared by the step calls; returns (S, V, B, ld, dtype code)."""
    dev = states.device
    _want(next_state, "next_state", torch.int32, dev)
    _want(allow, "allow", torch.int32, dev)
    _want(states, "states", torch.int32, dev)
    dt = _dtype_code(logits)
    if not logits.is_cuda or logits.device != dev:
        raise ValueError("logits must be on the same device as states")
    if next_state.dim() != 2:
        raise ValueError("next_state must be [S][V]")
    S, V = next_state.shape
    if allow.numel() != S * ((V + 31) // 32):
        raise ValueError("allow must be [S][ceil(V/32)]")
    B = states.shape[0]
    if states.dim() != 1:
        raise ValueError("states must be [B]")
    if logits.dim() != 2 or logits.shape[0] != B or logits.shape[1] != V:
        raise ValueError(f"logits must be [{B}][{V}] (a wider row stride is allowed)")
    if B and logits.stride(1) != 1:
        raise ValueError("logits must have unit stride along the vocabulary")
    ld = logits.stride(0) if B > 1 else max(V, logits.stride(0))
    return S, V, B, ld, dt


def masked_step(next_state, allow, states, logits, token=None, new_state=None, workspace=None,
                stream=None, opportunistic=False):
    """One greedy masked decoding step.  logits [B][ld] (fp32 or bf16, unit
    stride along the vocabulary).  Returns (token [B] int32, new_state [B] int32).
    ``opportunistic``: check the model's own choice against the mask first
    (dv_masked_step_opportunistic; same results)."""
    dev = states.device
    S, V, B, ld, dt = _step_args(next_state, allow, states, logits)
    token = _out(token, "token", B, dev)
    new_state = _out(new_state, "new_state", B, dev)
    workspace, nbytes = _workspace(workspace, masked_step_workspace_bytes(B, V), dev,
                                   lambda: step_workspace(B, V, dev))
    fn = lib.dv_masked_step_opportunistic if opportunistic else lib.dv_masked_step
    st = fn(_ptr(next_state), _ptr(allow), S, V, _ptr(states), _ptr(logits), dt, B, ld, _ptr(token),
            _ptr(new_state), _ptr(workspace), nbytes, _stream(stream, dev))
    _check(st, "dv_masked_step_opportunistic" if opportunistic else "dv_masked_step")
    return token, new_state


NOALLOC_MAX_BATCH = 65536


def masked_step_noalloc(next_state, allow, states, logits, token, new_state, stream=None):
    """``masked_step`` through dv_masked_step_noalloc: no workspace; split
    rows meet in the library's own scratch array on the device (batch at
    most NOALLOC_MAX_BATCH).  The outputs are caller-supplied, so the call
    allocates nothing.  Calls that may overlap on one GPU race."""
    dev = states.device
    S, V, B, ld, dt = _step_args(next_state, allow, states, logits)
    if token is None or new_state is None:
        raise ValueError("masked_step_noalloc writes into caller-supplied token and new_state")
    token = _out(token, "token", B, dev)
    new_state = _out(new_state, "new_state", B, dev)
    st = lib.dv_masked_step_noalloc(_ptr(next_state), _ptr(allow), S, V, _ptr(states), _ptr(logits), dt, B, ld,
                                    _ptr(token), _ptr(new_state), _stream(stream, dev))
    _check(st, "dv_masked_step_noalloc")
    return token, new_state


def masked_sample_workspace_bytes(batch: int, num_tokens: int) -> int:
    return int(lib.dv_masked_sample_workspace_bytes(batch, num_tokens))


def sample_workspace(batch: int, num_tokens: int, device) -> torch.Tensor:
    """A zero-filled workspace for ``masked_sample`` (left zero by every call;
    reusable by calls ordered on one stream)."""
    n = masked_sample_workspace_bytes(batch, num_tokens)
    return torch.zeros(max(n, 1), dtype=torch.uint8, device=device)


def masked_sample(next_state, allow, states, logits, seed: int, offset: int, inv_temperature: float = 1.0,
                  token=None, new_state=None, workspace=None, stream=None):
    """One sampled masked decoding step: each row draws from softmax(logits *
    inv_temperature) over its allowed tokens (Gumbel-max with Philox noise of
    (seed, offset, row, token); use a new offset for every step).  logits
    [B][ld] fp32 or bf16.  Returns (token [B], new_state [B])."""
    dev = states.device
    S, V, B, ld, dt = _step_args(next_state, allow, states, logits)
    token = _out(token, "token", B, dev)
    new_state = _out(new_state, "new_state", B, dev)
    workspace, nbytes = _workspace(workspace, masked_sample_workspace_bytes(B, V), dev,
                                   lambda: sample_workspace(B, V, dev))
    st = lib.dv_masked_sample(_ptr(next_state), _ptr(allow), S, V, _ptr(states), _ptr(logits), dt, B, ld,
                              float(inv_temperature), int(seed) & (2**64 - 1), int(offset) & (2**64 - 1),
                              _ptr(token), _ptr(new_state), _ptr(workspace), nbytes,
                              _stream(stream, dev))
    _check(st, "dv_masked_sample")
    return token, new_state


def _dtype_code(logits):
    if logits.dtype == torch.float32:
        return DV_F32
    if logits.dtype == torch.bfloat16:
        return DV_BF16
    raise TypeError(f"logits must be float32 or bfloat16, got {logits.dtype}")


def _proposals(proposals, B, dev):
    if proposals.dtype != torch.int32 or not proposals.is_cuda or proposals.device != dev:
        raise TypeError("proposals must be an int32 device tensor on the states' device")
    if proposals.dim() != 2 or proposals.shape[0] != B:
        raise ValueError(f"proposals must be [{B}][s]")
    s = proposals.shape[1]
    if B and s and proposals.stride(1) != 1:
        raise ValueError("proposals must have unit stride along a row")
    ld = proposals.stride(0) if B > 1 else s
    return s, max(ld, s)


def spec_walk(next_state, allow, states, proposals, accepted=None, final_state=None, stream=None):
    """Speculative chain check: (accepted [B], final_state [B]) -- how many of
    each row's proposals [B][s] the table admits in turn, and where they lead."""
    dev = states.device
    _want(next_state, "next_state", torch.int32, dev)
    _want(allow, "allow", torch.int32, dev)
    _want(states, "states", torch.int32, dev)
    S, V = next_state.shape
    B = states.shape[0]
    s, ld = _proposals(proposals, B, dev)
    accepted = _out(accepted, "accepted", B, dev)
    final_state = _out(final_state, "final_state", B, dev)
    st = lib.dv_spec_walk(_ptr(next_state), _ptr(allow), S, V, _ptr(states),
                          _ptr(proposals) if proposals.numel() else None, s, ld, B, _ptr(accepted),
                          _ptr(final_state), _stream(stream, dev))
    _check(st, "dv_spec_walk")
    return accepted, final_state


def spec_verify_workspace_bytes(batch: int, num_proposed: int, num_tokens: int) -> int:
    return int(lib.dv_spec_verify_workspace_bytes(batch, num_proposed, num_tokens))


def spec_workspace(batch: int, num_proposed: int, num_tokens: int, device) -> torch.Tensor:
    """A zero-filled workspace for ``spec_verify`` (left zero by every call;
    reusable by calls ordered on one stream)."""
    n = spec_verify_workspace_bytes(batch, num_proposed, num_tokens)
    return torch.zeros(max(n, 1), dtype=torch.uint8, device=device)


def spec_verify(next_state, allow, states, proposals, logits, token=None, accepted=None,
                new_state=None, workspace=None, stream=None):
    """Greedy verification of proposed tokens (Sec. 3.6).

    proposals [B][s] int32; logits [B][s+1][V] fp32 or bf16 with any strides
    except a unit one along the vocabulary (position j of row b: the model's
    logits after the first j proposals).  Returns (token [B][s+1],
    accepted [B], new_state [B]): the emitted tokens are token[b][:accepted[b]+1]."""
    dev = states.device
    _want(next_state, "next_state", torch.int32, dev)
    _want(allow, "allow", torch.int32, dev)
    _want(states, "states", torch.int32, dev)
    dt = _dtype_code(logits)
    S, V = next_state.shape
    B = states.shape[0]
    s, ld = _proposals(proposals, B, dev)
    if not logits.is_cuda or logits.device != dev:
        raise ValueError("logits must be on the same device as states")
    if logits.dim() != 3 or logits.shape[0] != B or logits.shape[1] != s + 1 or logits.shape[2] != V:
        raise ValueError(f"logits must be [{B}][{s + 1}][{V}] (wider strides are allowed)")
    if B and logits.stride(2) != 1:
        raise ValueError("logits must have unit stride along the vocabulary")
    ld_row, ld_pos = logits.stride(0), logits.stride(1)
    if token is None:
        token = torch.empty((B, s + 1), dtype=torch.int32, device=dev)
    token = _out(token, "token", B * (s + 1), dev)
    accepted = _out(accepted, "accepted", B, dev)
    new_state = _out(new_state, "new_state", B, dev)
    workspace, nbytes = _workspace(workspace, spec_verify_workspace_bytes(B, s, V), dev,
                                   lambda: spec_workspace(B, s, V, dev))
    st = lib.dv_spec_verify(_ptr(next_state), _ptr(allow), S, V, _ptr(states),
                            _ptr(proposals) if proposals.numel() else None, s, ld, _ptr(logits), dt,
                            ld_row, ld_pos, B, _ptr(token), _ptr(accepted), _ptr(new_state),
                            _ptr(workspace), nbytes, _stream(stream, dev))
    _check(st, "dv_spec_verify")
    return token, accepted, new_state
