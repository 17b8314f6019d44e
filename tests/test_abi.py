"""The C ABI on the host (no GPU needed): the library loads, exports every
function include/dv.h declares, and rejects bad arguments before any HIP call.

Pointer arguments here are fake non-NULL addresses: each call is built so that
a host-side check rejects it, so nothing is ever launched or dereferenced."""
import ctypes
import os
import re

import pytest

import paper_2403_06988_amd as dv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dv.h")
lib = dv.lib

OK, INVALID, SHAPE, DTYPE, ALIAS, WORKSPACE, HIP = range(7)
P = 0x7F0000000000  # fake device address (never dereferenced)
GB = 1 << 30


PROBE_LIB = os.path.join(ROOT, "paper_2403_06988_amd", "libdv_probes.so")


def declared_functions(header):
    text = open(os.path.join(ROOT, "include", header)).read()
    return re.findall(r"^(?:DV_API|DVPROBE_API)\s+[\w\s\*]+?\b(dv\w+)\s*\(", text, flags=re.M)


def test_every_declared_symbol_is_exported():
    """dv.h's functions from libdv.so; the probes of dv_probes.h from their
    own library, and none of them from libdv.so."""
    names = declared_functions("dv.h")
    assert {"dv_align_workspace_bytes", "dv_align", "dv_masked_step_workspace_bytes",
            "dv_masked_step", "dv_status_string", "dv_last_error", "dv_version"} <= set(names)
    raw = ctypes.CDLL(dv.library_path)
    for n in names:
        assert hasattr(raw, n), n
    probes = declared_functions("dv_probes.h")
    assert {"dvprobe_stream_read", "dvprobe_stream_write", "dvprobe_gather", "dvprobe_lds_gather",
            "dvprobe_step_floor", "dvprobe_walk_gather"} <= set(probes)
    plib = ctypes.CDLL(PROBE_LIB)
    for n in probes:
        assert hasattr(plib, n), n
        assert not hasattr(raw, n), f"{n} is measurement code: it belongs in libdv_probes.so only"


def test_step_floor_probe_rejects_bad_arguments():
    plib = ctypes.CDLL(PROBE_LIB)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    f = plib.dvprobe_step_floor
    f.restype = i32
    f.argtypes = [i32, vp, i32, i64, vp, i32, vp, i32, vp, vp, vp, i64, vp]

    def call(mode=1, logits=P, V=1000, ld=1000, allow=P + GB, S=16, states=P + 2 * GB, B=8, tok=P + 3 * GB,
             new=P + 4 * GB, sink=P + 5 * GB, sink_words=8 * 64):
        return f(mode, logits, V, ld, allow, S, states, B, tok, new, sink, sink_words, None)

    for kw in (dict(mode=3), dict(mode=-1), dict(logits=None), dict(mode=2, allow=None), dict(states=None),
               dict(B=0), dict(ld=999), dict(logits=P + 8), dict(ld=1001), dict(sink_words=7), dict(V=4)):
        assert call(**kw) == 1, kw


def test_status_strings_and_version():
    assert lib.dv_status_string(OK) == b"DV_OK"
    assert lib.dv_status_string(ALIAS) == b"DV_ERR_ALIAS"
    assert lib.dv_status_string(99) == b"DV_ERR_UNKNOWN"
    assert lib.dv_version() >= 100


def test_workspace_queries():
    assert lib.dv_align_workspace_bytes(0, 10) == 0
    assert lib.dv_align_workspace_bytes(70000, 10) == 0
    a = lib.dv_align_workspace_bytes(8192, 128256)
    assert a >= 8192 * 256 * 2  # compacted table of at most 256 uint16 columns
    assert lib.dv_masked_step_workspace_bytes(-1, 10) == 0
    assert lib.dv_masked_step_workspace_bytes(256, 128256) >= 256 * 12
    assert lib.dv_masked_step_workspace_bytes(0, 10) > 0


def test_step_workspace_fits_the_noalloc_array():
    """dv_masked_step_noalloc passes its scratch array as the workspace, sized
    for DV_NOALLOC_MAX_BATCH rows meeting through a maximum and a count (12
    bytes a row): every batch it accepts must need no more, including the
    batches whose rows meet in pairs (up to 24 bytes a row)."""
    cap = 768 * 1024
    for V in (1, 1000, 32000, 70001, 128256, 256000, 1 << 24):
        for B in list(range(1, 300)) + [511, 512, 1000, 4096, 65535, 65536]:
            need = lib.dv_masked_step_workspace_bytes(B, V)
            assert 0 < need <= cap, (B, V, need)


def _align(trans=P, S=16, offsets=P + GB, bytes_=P + 2 * GB, V=1000, ns=P + 3 * GB,
           allow=P + 4 * GB, ws=P + 5 * GB, ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = lib.dv_align_workspace_bytes(max(S, 1), max(V, 1))
    return lib.dv_align(trans, S, offsets, bytes_, V, ns, allow, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(trans=None), INVALID),
    (dict(offsets=None), INVALID),
    (dict(ns=None), INVALID),
    (dict(allow=None), INVALID),
    (dict(S=0), SHAPE),
    (dict(S=65536), SHAPE),
    (dict(V=0), SHAPE),
    (dict(V=-5), SHAPE),
    (dict(allow=P + 3 * GB + 4), ALIAS),          # allow inside next_state
    (dict(ns=P), ALIAS),                          # next_state over trans
    (dict(allow=P + GB), ALIAS),                  # allow over offsets
    (dict(ws=None), WORKSPACE),
    (dict(ws_bytes=100), WORKSPACE),
    (dict(ws=P + 5 * GB + 8), WORKSPACE),         # not 256-byte aligned
    (dict(ws=P + 3 * GB), ALIAS),                 # workspace over next_state
])
def test_align_rejects_before_launch(kw, status):
    assert _align(**kw) == status
    assert lib.dv_last_error().startswith(b"dv_align")


def _step(ns=P, allow=P + GB, S=16, V=1000, states=P + 2 * GB, logits=P + 3 * GB, dtype=0, B=8,
          ld=1000, tok=P + 4 * GB, new=P + 5 * GB, ws=P + 6 * GB, ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = lib.dv_masked_step_workspace_bytes(max(B, 0), max(V, 1))
    return lib.dv_masked_step(ns, allow, S, V, states, logits, dtype, B, ld, tok, new, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(ns=None), INVALID),
    (dict(states=None), INVALID),
    (dict(logits=None), INVALID),
    (dict(tok=None), INVALID),
    (dict(S=0), SHAPE),
    (dict(V=0), SHAPE),
    (dict(B=-1), SHAPE),
    (dict(ld=999), SHAPE),
    (dict(dtype=2), DTYPE),
    (dict(dtype=-1), DTYPE),
    (dict(new=P + 4 * GB + 4), ALIAS),            # token / new_state overlap
    (dict(new=P + 2 * GB), ALIAS),                # in-place state update
    (dict(tok=P + 3 * GB + 100), ALIAS),          # output inside logits
    (dict(tok=P + 8), ALIAS),                     # output inside next_state
    (dict(ws=None), WORKSPACE),
    (dict(ws_bytes=8), WORKSPACE),
    (dict(ws=P + 6 * GB + 64), WORKSPACE),
    (dict(ws=P + 2 * GB), ALIAS),
    (dict(logits=P + 3 * GB + 2), INVALID),       # fp32 logits not 4-byte aligned
    (dict(logits=P + 3 * GB + 1, dtype=1), INVALID),  # bf16 logits at an odd address
])
def test_masked_step_rejects_before_launch(kw, status):
    assert _step(**kw) == status
    assert lib.dv_last_error().startswith(b"dv_masked_step")


def _noalloc(ns=P, allow=P + GB, S=16, V=1000, states=P + 2 * GB, logits=P + 3 * GB, dtype=0, B=8,
             ld=1000, tok=P + 4 * GB, new=P + 5 * GB):
    return lib.dv_masked_step_noalloc(ns, allow, S, V, states, logits, dtype, B, ld, tok, new, None)


@pytest.mark.parametrize("kw,status", [
    (dict(ns=None), INVALID),
    (dict(logits=None), INVALID),
    (dict(S=0), SHAPE),
    (dict(B=-1), SHAPE),
    (dict(B=65537), SHAPE),                       # beyond the scratch array
    (dict(ld=999), SHAPE),
    (dict(dtype=2), DTYPE),
    (dict(new=P + 2 * GB), ALIAS),                # in-place state update
    (dict(logits=P + 3 * GB + 1, dtype=1), INVALID),
])
def test_masked_step_noalloc_rejects_before_any_hip_call(kw, status):
    """Every check of the scratch-backed step runs before it looks up or
    clears its scratch array (no GPU here: a HIP call would fail)."""
    assert _noalloc(**kw) == status
    assert lib.dv_last_error().startswith(b"dv_masked_step_noalloc")


def test_masked_step_noalloc_empty_batch_is_a_noop():
    assert _noalloc(B=0, states=None, logits=None, tok=None, new=None) == OK
    assert lib.dv_last_error() == b""


@pytest.mark.parametrize("kw,status", [
    (dict(offsets=None), INVALID),
    (dict(out=None), INVALID),
    (dict(V=0), SHAPE),
    (dict(V=1 << 25), SHAPE),
    (dict(nbytes=-1), SHAPE),
    (dict(out=P + 40), ALIAS),                    # the result inside offsets
])
def test_validate_vocab_rejects_before_launch(kw, status):
    a = dict(offsets=P, V=1000, nbytes=5000, out=P + GB)
    a.update(kw)
    assert lib.dv_validate_vocab(a["offsets"], a["V"], a["nbytes"], a["out"], None) == status
    assert lib.dv_last_error().startswith(b"dv_validate_vocab")


def test_last_error_is_per_thread():
    """The detail string belongs to the calling thread: threads failing in
    different entry points, and one whose calls succeed, each read their
    own last error while the others keep calling (ctypes releases the
    interpreter lock around the calls)."""
    import threading
    errors = []
    barrier = threading.Barrier(3)

    def run(call, want, prefix):
        barrier.wait()
        for _ in range(300):
            st = call()
            msg = lib.dv_last_error()
            if st != want or not msg.startswith(prefix) or (prefix == b"" and msg != b""):
                errors.append((want, st, prefix, msg))
                return

    threads = [threading.Thread(target=run, args=a) for a in (
        (lambda: _align(S=0), SHAPE, b"dv_align"),
        (lambda: _step(dtype=2), DTYPE, b"dv_masked_step"),
        (lambda: _step(B=0), OK, b""),
    )]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors[:3]


def test_masked_step_empty_batch_is_a_noop():
    assert _step(B=0) == OK
    assert lib.dv_last_error() == b""
    # empty tensors have NULL data pointers
    assert _step(B=0, states=None, logits=None, tok=None, new=None) == OK
    assert _step(B=0, ns=None) == INVALID


def test_binding_type_checks():
    import torch
    with pytest.raises((TypeError, ValueError)):
        dv.align(torch.zeros((2, 256), dtype=torch.int64), torch.zeros(3, dtype=torch.int32),
                 torch.zeros(1, dtype=torch.uint8))
    with pytest.raises((TypeError, ValueError)):
        dv.align(torch.zeros((2, 256), dtype=torch.int32), torch.zeros(3, dtype=torch.int32),
                 torch.zeros(1, dtype=torch.uint8))  # CPU tensors are refused


def test_align_eos_rejects_bad_token_before_launch():
    ws_bytes = lib.dv_align_workspace_bytes(16, 1000)
    for eos in (-1, 1000, 5000):
        st = lib.dv_align_eos(P, 16, P + GB, P + 2 * GB, 1000, P + 6 * GB, eos, P + 3 * GB, P + 4 * GB,
                              P + 5 * GB, ws_bytes, None)
        assert st == SHAPE
        assert lib.dv_last_error().startswith(b"dv_align_eos")
    # accepting flags overlapping an output
    st = lib.dv_align_eos(P, 16, P + GB, P + 2 * GB, 1000, P + 3 * GB + 8, 3, P + 3 * GB, P + 4 * GB,
                          P + 5 * GB, ws_bytes, None)
    assert st == ALIAS


def _walk(ns=P, allow=P + GB, S=16, V=1000, states=P + 2 * GB, props=P + 3 * GB, s=4, ld=4, B=8,
          acc=P + 4 * GB, fin=P + 5 * GB):
    return lib.dv_spec_walk(ns, allow, S, V, states, props, s, ld, B, acc, fin, None)


@pytest.mark.parametrize("kw,status", [
    (dict(ns=None), INVALID),
    (dict(props=None), INVALID),
    (dict(acc=None), INVALID),
    (dict(S=0), SHAPE),
    (dict(B=-1), SHAPE),
    (dict(s=-1), SHAPE),
    (dict(s=1025, ld=2000), SHAPE),
    (dict(ld=3), SHAPE),
    (dict(B=300000, s=4), SHAPE),                 # B * (s + 1) above the batch limit
    (dict(fin=P + 4 * GB + 4), ALIAS),
    (dict(acc=P + 3 * GB + 16), ALIAS),           # output inside the proposals
    (dict(fin=P + 2 * GB), ALIAS),                # final state written over the states
])
def test_spec_walk_rejects_before_launch(kw, status):
    assert _walk(**kw) == status
    assert lib.dv_last_error().startswith(b"dv_spec_walk")


def test_spec_walk_empty_and_no_proposals():
    assert _walk(B=0, states=None, props=None, acc=None, fin=None) == OK
    assert _walk(B=0, ns=None) == INVALID


def _verify(ns=P, allow=P + GB, S=16, V=1000, states=P + 2 * GB, props=P + 3 * GB, s=4, ldp=4,
            logits=P + 4 * GB, dtype=1, ld_row=5000, ld_pos=1000, B=8, tok=P + 5 * GB,
            acc=P + 6 * GB, new=P + 7 * GB, ws=P + 8 * GB, ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = lib.dv_spec_verify_workspace_bytes(max(B, 0), max(s, 0), max(V, 1))
    return lib.dv_spec_verify(ns, allow, S, V, states, props, s, ldp, logits, dtype, ld_row, ld_pos, B,
                              tok, acc, new, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(allow=None), INVALID),
    (dict(logits=None), INVALID),
    (dict(tok=None), INVALID),
    (dict(new=None), INVALID),
    (dict(V=0), SHAPE),
    (dict(s=-2), SHAPE),
    (dict(ldp=2), SHAPE),
    (dict(ld_row=-1), SHAPE),
    (dict(ld_pos=1 << 41), SHAPE),
    (dict(B=(1 << 20) // 5 + 1), SHAPE),
    (dict(dtype=7), DTYPE),
    (dict(acc=P + 5 * GB + 8), ALIAS),            # accepted inside token [B][s+1]
    (dict(tok=P + 4 * GB + 64), ALIAS),           # token inside the logits
    (dict(new=P + 2 * GB), ALIAS),                # new state written over the states
    (dict(ws=None), WORKSPACE),
    (dict(ws_bytes=16), WORKSPACE),
    (dict(ws=P + 8 * GB + 128), WORKSPACE),
    (dict(ws=P + 3 * GB), ALIAS),
    (dict(logits=P + 4 * GB + 3), INVALID),       # bf16 logits at an odd address
])
def test_spec_verify_rejects_before_launch(kw, status):
    assert _verify(**kw) == status
    assert lib.dv_last_error().startswith(b"dv_spec_verify")


def test_spec_verify_workspace_and_empty_batch():
    assert lib.dv_spec_verify_workspace_bytes(-1, 4, 10) == 0
    assert lib.dv_spec_verify_workspace_bytes(8, 2000, 10) == 0
    assert lib.dv_spec_verify_workspace_bytes(256, 8, 128256) >= 2 * 256 * 9 * 4
    assert _verify(B=0, states=None, props=None, logits=None, tok=None, acc=None, new=None) == OK


@pytest.mark.parametrize("kw,status", [
    (dict(ns=None), INVALID),
    (dict(ld=999), SHAPE),
    (dict(dtype=2), DTYPE),
    (dict(new=P + 2 * GB), ALIAS),
    (dict(ws_bytes=8), WORKSPACE),
])
def test_opportunistic_step_rejects_before_launch(kw, status):
    args = dict(ns=P, allow=P + GB, S=16, V=1000, states=P + 2 * GB, logits=P + 3 * GB, dtype=1, B=300,
                ld=1000, tok=P + 4 * GB, new=P + 5 * GB, ws=P + 6 * GB, ws_bytes=None)
    args.update(kw)
    if args["ws_bytes"] is None:
        args["ws_bytes"] = lib.dv_masked_step_workspace_bytes(300, 1000)
    st = lib.dv_masked_step_opportunistic(args["ns"], args["allow"], args["S"], args["V"], args["states"],
                                          args["logits"], args["dtype"], args["B"], args["ld"], args["tok"],
                                          args["new"], args["ws"], args["ws_bytes"], None)
    assert st == status
    assert lib.dv_last_error().startswith(b"dv_masked_step_opportunistic")


@pytest.mark.parametrize("kw,status", [
    (dict(ns=None), INVALID),
    (dict(ld=999), SHAPE),
    (dict(inv_t=0.0), SHAPE),
    (dict(inv_t=-1.0), SHAPE),
    (dict(inv_t=float("nan")), SHAPE),
    (dict(inv_t=float("inf")), SHAPE),
    (dict(dtype=5), DTYPE),
    (dict(new=P + 2 * GB), ALIAS),
    (dict(ws_bytes=8), WORKSPACE),
    (dict(ws=P + 6 * GB + 8), WORKSPACE),
    (dict(logits=P + 3 * GB + 1), INVALID),
])
def test_masked_sample_rejects_before_launch(kw, status):
    args = dict(ns=P, allow=P + GB, S=16, V=1000, states=P + 2 * GB, logits=P + 3 * GB, dtype=1, B=8,
                ld=1000, inv_t=1.0, tok=P + 4 * GB, new=P + 5 * GB, ws=P + 6 * GB, ws_bytes=None)
    args.update(kw)
    if args["ws_bytes"] is None:
        args["ws_bytes"] = lib.dv_masked_sample_workspace_bytes(8, 1000)
    st = lib.dv_masked_sample(args["ns"], args["allow"], args["S"], args["V"], args["states"], args["logits"],
                              args["dtype"], args["B"], args["ld"], args["inv_t"], 1, 2, args["tok"], args["new"],
                              args["ws"], args["ws_bytes"], None)
    assert st == status
    assert lib.dv_last_error().startswith(b"dv_masked_sample")


def test_masked_sample_workspace_query():
    assert lib.dv_masked_sample_workspace_bytes(-1, 10) == 0
    assert lib.dv_masked_sample_workspace_bytes(256, 128256) >= 256 * 8
