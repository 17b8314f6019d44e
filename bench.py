#!/usr/bin/env python3
"""Throughput of the constrained-decoding hot path on one MI355X.

One benchmark step is one whole job of the hot path on one batch of
synthetic input: build the alignment table of the DFA and the vocabulary
(dv_align), then run the workload's greedy decoding chain (one dv_masked_step
per decoding step, each step's states feeding the next).  Inputs (DFA,
vocabulary, every step's logits) are resident in HBM before timing starts.

Reported (one JSON line):
  value        masked decode steps / s over the timed decode launches
  align        (state, token) alignments / s of dv_align
  ms_per_step  wall time of one whole job (align + all decode steps)
  roofline     the dominant kernel (the masked step) against HBM bandwidth:
               algorithmic bytes per launch / mean launch time (HIP events
               around the replay of the job's decode steps, captured once as
               a HIP graph, on the launch stream; divided by the step count)
               (with the probes: frac_of_measured_read, the same rate against
               this box's streaming-read probe)
  roofline_align  dv_align against the HBM write roofline (4.125 B / pair)
               (frac_of_measured_write: against the streaming-write probe)
  opportunistic  the decode chain with the model's own choice checked first
               (Sec. 3.5), on the workload's logits and on adherent logits
  sample       the decode chain sampled at temperature 1 (Sec. 4), ALU roofline
  spec_verify  greedy verification of s = 8 proposed tokens per row (Sec. 3.6)
               over windows of the job's decode chain, with its own roofline
  floors       the masked step's measured floors at its own launch shape
               (probes in libdv_probes.so): an empty step, a loads-only pass
               over whole rows and one over exactly the lines the step reads
  extra        decode legs of the other bandwidth-sized workloads (3 and 5):
               us per step, touched-line roofline, traffic, floors
  cpu_baseline the CPU oracle on a bounded sample of the same workload
  inputs       SHA-256 of the DFA, the vocabulary and the initial states, and
               the realised token lengths

Usage: python bench.py [--steps K] [--warmup W] [--workload 1..10] [--no-cpu]
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "(state,token) alignments/sec for dv_align; masked decode steps/sec at V=128k"
HBM_PEAK_GBS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_2403_06988_amd", "csrc")
KERNEL_SOURCES = {"masked_step": ("dv_step.hip", "dv_internal.h"),
                  "align": ("dv_align.hip", "dv_internal.h"),
                  "spec_verify": ("dv_step.hip", "dv_spec.hip", "dv_internal.h"),
                  "sample": ("dv_sample.hip", "dv_sample.h", "dv_internal.h")}
TRAFFIC_FILES = {
    ("masked_step", 3): "masked_step_bf16_kernel__llm-tokenizer-scale_S1024_V128256_B64.traffic.txt",
    ("masked_step", 4): "masked_step_bf16_kernel__grammar-lexer-union_S8192_V128256_B256.traffic.txt",
    ("masked_step", 5): "masked_step_bf16_kernel__large-vocab-high-batch_S4096_V256000_B1024.traffic.txt",
    ("align", 4): "walk_prefix_kernel__grammar-lexer-union_S8192_V128256.traffic.txt",
    ("spec_verify", 4): "spec_verify__grammar-lexer-union_S8192_V128256_B256_s8.traffic.txt",
}
PROBE_LIB = os.path.join(ROOT, "paper_2403_06988_amd", "libdv_probes.so")
EXTRA_WORKLOADS = (3, 5)


def kernel_source_hash(which):
    """Hash of the kernel sources without their comments and blank lines, so
    that a recorded measurement stays attached to the code it was taken on
    through edits of the comments alone."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[which]:
        for line in open(os.path.join(CSRC, f), encoding="utf-8"):
            code = line.split("//", 1)[0].rstrip()
            if code:
                h.update(code.encode() + b"\n")
    return h.hexdigest()[:16]


def inputs_record(trans, offsets, data, init):
    """SHA-256 of the workload's inputs (the DFA, the vocabulary, the
    initial states) and the realised token lengths, so that a result names
    exactly what it was measured on."""
    import numpy as np

    def sha(*arrays):
        h = hashlib.sha256()
        for a in arrays:
            h.update(np.ascontiguousarray(a).tobytes())
        return h.hexdigest()

    lens = np.diff(np.asarray(offsets, dtype=np.int64))
    return {"dfa_sha256": sha(trans), "vocab_sha256": sha(offsets, data), "init_states_sha256": sha(init),
            "token_len_mean": float(lens.mean()) if lens.size else 0.0, "token_len_max": int(lens.max(initial=0)),
            "token_bytes": int(lens.sum())}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10, help="timed jobs")
    ap.add_argument("--warmup", type=int, default=2, help="untimed jobs")
    ap.add_argument("--workload", type=int, default=4)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU-oracle baseline")
    ap.add_argument("--no-probes", action="store_true", help="skip the roofline probes")
    ap.add_argument("--no-spec", action="store_true", help="skip the speculative-verification leg")
    ap.add_argument("--no-opportunistic", action="store_true", help="skip the opportunistic-masking leg")
    ap.add_argument("--no-sample", action="store_true", help="skip the masked-sampling leg")
    ap.add_argument("--no-floors", action="store_true", help="skip the masked step's floor probes")
    ap.add_argument("--no-extra", action="store_true", help="skip the decode legs of workloads 3 and 5")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


LINE = 128  # bytes the memory system fetches at a time


def touched_line_bytes(al, states, base_ptr, ld, V, elt):
    """Logit bytes a masked step must read: the 128-byte lines that hold at
    least one allowed token, over the rows whose state is live (a line with
    no allowed token cannot change the result).  Row r (state states[r])
    starts at byte base_ptr + r * ld * elt; lines are aligned in memory, so a
    row that does not start on a line boundary counts the lines it touches."""
    import torch

    rows = torch.nonzero(states >= 0)[:, 0]
    if rows.numel() == 0:
        return 0
    tpl = LINE // elt
    total = 0
    for part in torch.split(rows, max(1, (1 << 26) // max(V, 1))):   # bounded temporaries
        words = al[states[part].long()]                                  # [m, W] int32
        shift = torch.arange(32, device=words.device, dtype=torch.int32)
        bits = ((words[..., None] >> shift) & 1).reshape(part.numel(), -1)[:, :V]
        off = ((base_ptr + part.long() * ld * elt) % LINE) // elt          # [m]
        lid = (off[:, None] + torch.arange(V, device=words.device)) // tpl
        hit = torch.zeros((part.numel(), (V + tpl - 1) // tpl + 1), dtype=torch.int32, device=words.device)
        hit.scatter_reduce_(1, lid, bits, reduce="amax")
        total += int(hit.sum())
    return total * LINE


def step_bytes(w, logit_bytes, live_rows, B):
    """Algorithmic HBM bytes of one masked step: the logit lines the live rows
    must read (touched_line_bytes), each live row's allow row (4 ceil(V/32) B)
    and one gathered next_state entry; every row reads its state and writes
    token and new state."""
    return logit_bytes + live_rows * (4 * w.words + 4) + 12 * B


def align_walk_kind(trans):
    """Which walk dv_align runs for this table (the library decides on the
    device from the same quantities): the whole compacted table staged in
    LDS, the prefix-table walk (at most 98 compacted columns), or the tile
    walk.  Reporting only: it names the kernel the roofline figures cover."""
    import numpy as np
    S = trans.shape[0]
    C = int(((trans >= 0) & (trans < S)).any(axis=0).sum())
    Cp = (C + 2) & ~1 if C < 256 else 256
    lds_table = 16 * 256 * 2
    if S <= 512:
        lds_table = max(lds_table, min(S * 256 * 2, 64 * 1024))
    if S * Cp * 2 <= lds_table:
        return "walk_kernel (whole table in LDS)"
    return "walk_prefix_kernel" if Cp <= 98 else "walk_kernel"


def traffic_record(which, workload_id):
    """Calibrated HBM bytes per launch from the committed rocprofv3 --pmc
    summary (FETCH_SIZE + WRITE_SIZE, each scaled by what the counter reads
    for a streaming probe of known size), if it covers this workload and was
    taken on the current kernel source; else None."""
    name = TRAFFIC_FILES.get((which, workload_id))
    if name is None:
        return None
    path = os.path.join(PROFILES, name)
    if not os.path.exists(path):
        return None
    rec = {}
    for line in open(path):
        if ":" in line and not line.startswith(" "):
            k, v = line.split(":", 1)
            rec[k.strip()] = v.strip()
    if rec.get("kernel_source_hash") != kernel_source_hash(which):
        return None
    return float(rec["hbm_bytes_per_launch"])


def cpu_baseline(w, wid, trans, offsets, data, init, x_dev, budget_s):
    """The oracle as it stands, single-threaded, on a bounded sample: the
    oracle's own greedy chain over every row of the batch for the first steps
    (at most 32, or half the budget; table rows built beforehand, untimed, as
    the decode throughput excludes the table build), then alignment rows for
    the rest of the budget."""
    import numpy as np

    import oracle
    from tests.gpu_common import to_oracle

    lib = oracle.load()
    # decode: all B rows, step after step, until half the budget is spent
    max_steps = int(max(1, min(x_dev.shape[0], 32, 2e9 // (w.B * w.V * w.elt))))
    cache = oracle.RowCache(trans, offsets, data, lib=lib)
    cur = [int(s) for s in init]
    row_steps = 0
    t_dec = 0.0
    done_steps = 0
    for k in range(max_steps):
        xs = to_oracle(x_dev[k])
        rows = [cache.get(s) if s >= 0 else None for s in cur]   # untimed: table build
        t0 = time.perf_counter()
        for b in range(w.B):
            if rows[b] is None:
                continue
            tok = oracle.masked_argmax(rows[b][1], xs[b], lib=lib)
            cur[b] = -1 if tok < 0 else int(rows[b][0][tok])
            row_steps += 1
        t_dec += time.perf_counter() - t0
        done_steps += 1
        if t_dec > budget_s / 2:
            break
    dec_steps_per_s = (row_steps / w.B) / t_dec if t_dec > 0 else None
    # alignment: whole rows of the table
    rng = np.random.default_rng(0)
    pairs = 0
    t_al = 0.0
    while t_al < budget_s - t_dec:
        rows = rng.integers(0, w.S, 4).astype(np.int32)
        t0 = time.perf_counter()
        oracle.align_rows(trans, offsets, data, rows, lib=lib)
        t_al += time.perf_counter() - t0
        pairs += len(rows) * w.V
    # workload statistic for the alignment's L2 roofline: table moves per pair,
    # in all and past the first one and two bytes (the tile walk and the
    # prefix-table walk take those from LDS)
    srows = rng.integers(0, w.S, 256).astype(np.int32)
    hist = oracle.walk_length_hist(trans, offsets, data, srows, lib=lib)
    k = np.arange(len(hist))
    npairs = len(srows) * w.V
    moves = float((k * hist).sum()) / npairs
    past = {d: float((np.maximum(k - d, 0) * hist).sum()) / npairs for d in (1, 2)}
    every = all_cores(w, lib, cache, init, x_dev, done_steps, trans, offsets, data, budget_s / 3)
    return {
        "value": dec_steps_per_s, "unit": "steps/s", "cores": 1, "kind": "oracle",
        "moves_per_pair": moves,
        "moves_past_byte_1_per_pair": past[1],
        "moves_past_byte_2_per_pair": past[2],
        "sample": (f"{row_steps} row-steps: the oracle's greedy chain over all {w.B} rows for "
                   f"{done_steps} steps; table rows built untimed"),
        "align_value": pairs / t_al, "align_unit": "alignments/s",
        "align_sample": f"{pairs} (state, token) pairs in whole table rows",
        "seconds": round(t_dec + t_al, 2),
        "all_cores": every,
        "cpu_model": cpu_model(),
        "oracle_build": " ".join(oracle.BUILD_FLAGS),
    }


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def all_cores(w, lib, cache, init, x_dev, steps, trans, offsets, data, budget_s):
    """The same oracle calls spread over the process's CPU share (at most 16
    threads; the C calls run without the interpreter lock): the first
    ``steps`` steps of the greedy chain with the rows of each step split over
    the threads, then whole table rows of the alignment, one call per thread
    at a time."""
    import concurrent.futures as cf

    import numpy as np

    import oracle
    from tests.gpu_common import to_oracle

    n = max(1, min(16, len(os.sched_getaffinity(0))))
    parts = [list(range(i, w.B, n)) for i in range(n)]
    cur = [int(s) for s in init]
    t_dec, row_steps = 0.0, 0
    with cf.ThreadPoolExecutor(n) as pool:
        for k in range(steps):
            xs = to_oracle(x_dev[k])
            rows = [cache.get(s) if s >= 0 else None for s in cur]   # untimed (built by the 1-thread leg)

            def run(part):
                out = []
                for b in part:
                    if rows[b] is None:
                        continue
                    tok = oracle.masked_argmax(rows[b][1], xs[b], lib=lib)
                    out.append((b, -1 if tok < 0 else int(rows[b][0][tok])))
                return out

            t0 = time.perf_counter()
            results = list(pool.map(run, parts))
            t_dec += time.perf_counter() - t0
            for out in results:
                for b, nxt in out:
                    cur[b] = nxt
                    row_steps += 1
        rng = np.random.default_rng(1)
        pairs, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < budget_s:
            batches = [rng.integers(0, w.S, 2).astype(np.int32) for _ in range(n)]
            list(pool.map(lambda r: oracle.align_rows(trans, offsets, data, r, lib=lib), batches))
            pairs += sum(len(r) for r in batches) * w.V
        t_al = time.perf_counter() - t0
    return {"cores": n, "value": (row_steps / w.B) / t_dec if t_dec > 0 else None, "unit": "steps/s",
            "align_value": pairs / t_al, "align_unit": "alignments/s",
            "sample": f"{row_steps} row-steps over {steps} steps, then {pairs} (state, token) pairs",
            "seconds": round(t_dec + t_al, 2)}


def probe_lib():
    """The roofline probes (libdv_probes.so, include/dv_probes.h): measurement
    code kept out of libdv.so."""
    import ctypes

    if not os.path.exists(PROBE_LIB):
        raise SystemExit(f"{PROBE_LIB} not built (python -c 'import __graft_entry__ as g; g.build()')")
    lib = ctypes.CDLL(PROBE_LIB)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.dvprobe_stream_read.argtypes = [vp, sz, vp, vp]
    lib.dvprobe_stream_write.argtypes = [vp, sz, vp]
    lib.dvprobe_gather.argtypes = [vp, i32, i32, i32, i32, vp, vp]
    lib.dvprobe_lds_gather.argtypes = [vp, i32, i32, i32, i32, vp, vp]
    lib.dvprobe_step_floor.argtypes = [i32, vp, i32, i64, vp, i32, vp, i32, vp, vp, vp, i64, vp]
    lib.dvprobe_walk_gather.argtypes = [vp, i32, i32, i32, i32, i32, vp, vp]
    for f in (lib.dvprobe_stream_read, lib.dvprobe_stream_write, lib.dvprobe_gather,
              lib.dvprobe_lds_gather, lib.dvprobe_step_floor, lib.dvprobe_walk_gather):
        f.restype = i32
    return lib


_HIP_RT = None


def _hip_runtime():
    """The HIP runtime library (already loaded by torch), for its own graph calls."""
    import ctypes

    global _HIP_RT
    if _HIP_RT is None:
        lib = ctypes.CDLL("libamdhip64.so")
        vp, i32 = ctypes.c_void_p, ctypes.c_int
        lib.hipStreamBeginCapture.argtypes = [vp, i32]
        lib.hipStreamEndCapture.argtypes = [vp, ctypes.POINTER(vp)]
        lib.hipGraphInstantiate.argtypes = [ctypes.POINTER(vp), vp, vp, ctypes.c_char_p, ctypes.c_size_t]
        lib.hipGraphLaunch.argtypes = [vp, vp]
        lib.hipGraphExecDestroy.argtypes = [vp]
        lib.hipGraphDestroy.argtypes = [vp]
        for f in (lib.hipStreamBeginCapture, lib.hipStreamEndCapture, lib.hipGraphInstantiate,
                  lib.hipGraphLaunch, lib.hipGraphExecDestroy, lib.hipGraphDestroy):
            f.restype = i32
        lib.hipGetErrorString.argtypes = [i32]
        lib.hipGetErrorString.restype = ctypes.c_char_p
        _HIP_RT = lib
    return _HIP_RT


class HipGraph:
    """``launches()`` captured into a HIP graph by the HIP runtime's own stream
    capture (global mode, so any allocation or synchronization inside fails
    the capture instead of running outside the graph) on a side stream, and
    replayed with hipGraphLaunch on the current stream.

    torch.cuda.graph is not used for timing: on this PyTorch build for ROCm,
    once a process has made one torch capture, every later kernel of that
    process runs longer (the same loads-only kernel over 256 rows of 128,256
    bf16: 11.0 us per dispatch before and 11.8 us after, in rocprofv3 kernel
    traces; captures made through the HIP API, in any capture mode, leave it
    at 11.0)."""

    def __init__(self, launches, dev):
        import ctypes
        import torch

        self._lib = lib = _hip_runtime()
        self._dev = dev
        side = torch.cuda.Stream(dev)
        side.wait_stream(torch.cuda.current_stream(dev))
        torch.cuda.synchronize()
        graph = ctypes.c_void_p()
        self._check(lib.hipStreamBeginCapture(side.cuda_stream, 0), "hipStreamBeginCapture")
        try:
            with torch.cuda.stream(side):
                launches()
        finally:
            rc = lib.hipStreamEndCapture(side.cuda_stream, ctypes.byref(graph))
        self._check(rc, "hipStreamEndCapture")
        self._graph = graph
        self._exec = ctypes.c_void_p()
        self._check(lib.hipGraphInstantiate(ctypes.byref(self._exec), graph, None, None, 0), "hipGraphInstantiate")
        self._side = side

    def _check(self, rc, what):
        if rc != 0:
            raise RuntimeError(f"{what}: {self._lib.hipGetErrorString(rc).decode()}")

    def replay(self):
        import torch

        self._check(self._lib.hipGraphLaunch(self._exec, torch.cuda.current_stream(self._dev).cuda_stream),
                    "hipGraphLaunch")

    def close(self):
        import torch

        if self._exec:
            torch.cuda.synchronize()
            self._lib.hipGraphExecDestroy(self._exec)
            self._lib.hipGraphDestroy(self._graph)
            self._exec = None


def capture(launches, dev):
    """Run ``launches()`` once on a side stream (lazy set-up happens outside
    the capture), then capture it (HipGraph)."""
    import torch

    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        launches()
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()
    return HipGraph(launches, dev)


def graph_seconds(launches, dev, reps=3):
    """Seconds per replay of a HIP graph of ``launches()`` (run once eagerly
    on a side stream first, then captured), timed with HIP events on the
    replaying stream; the minimum over ``reps`` replays."""
    import torch

    graph = capture(launches, dev)
    stream = torch.cuda.current_stream(dev)
    best = None
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        graph.replay()
        b.record(stream)
        torch.cuda.synchronize()
        t = a.elapsed_time(b) / 1e3
        best = t if best is None else min(best, t)
    graph.close()
    return best


def step_floors(probes, w, al, x, states_all, dev, step_us, bytes_per_launch):
    """The masked step's floors at its own launch shape (same blocks and block
    size), each over the job's steps with the job's own states, graph-replayed:
    an empty step (launch + state read + outputs), a loads-only pass over
    whole rows, and a loads-only pass over exactly the 128-byte lines holding
    an allowed token (the bytes the roofline counts; mask bytes read first)."""
    import torch

    if w.dtype != "bf16":
        return None
    tok = torch.empty(w.B, dtype=torch.int32, device=dev)
    new = torch.empty(w.B, dtype=torch.int32, device=dev)
    sink_words = w.B * 64
    sink = torch.empty(sink_words, dtype=torch.int32, device=dev)
    out = {}
    for mode, key in ((0, "empty_step_us"), (1, "loads_whole_rows_us"), (2, "loads_touched_lines_us")):
        def launches():
            sh = torch.cuda.current_stream(dev).cuda_stream
            for k in range(w.steps):
                rc = probes.dvprobe_step_floor(mode, x[k].data_ptr(), w.V, w.V, al.data_ptr(), w.S,
                                               states_all[k].data_ptr(), w.B, tok.data_ptr(), new.data_ptr(),
                                               sink.data_ptr(), sink_words, sh)
                if rc != 0:
                    raise RuntimeError(f"dvprobe_step_floor mode {mode} failed with status {rc}")
        out[key] = graph_seconds(launches, dev) / w.steps * 1e6
    touched = out["loads_touched_lines_us"]
    out["step_us"] = step_us
    out["step_over_touched_floor"] = step_us / touched
    out["frac_at_touched_floor"] = bytes_per_launch / (touched * 1e-6) / 1e9 / HBM_PEAK_GBS
    out["note"] = ("probes at the step's grid and block size, graph-replayed over the job's steps and states; "
                   "frac_at_touched_floor = the roofline fraction a step as fast as the loads-only pass over "
                   "its touched lines would reach")
    return out


def run_probes(probes, dev, table_bytes):
    """Measured rates of the memory paths the kernels use (libdv_probes.so):
    HBM stream read / write, dependent random gathers from a table the size
    of the workload's compacted DFA (L1/L2), the alignment walk's own gather
    pattern (2-byte reads at state * classes + class), and gathers from LDS."""
    import torch

    lib = probes
    stream = torch.cuda.current_stream(dev)
    sh = stream.cuda_stream

    def timed(fn, reps=5):
        best = None
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            rc = fn()
            b.record(stream)
            torch.cuda.synchronize()
            if rc != 0:
                raise RuntimeError(f"probe failed with status {rc}")
            ms = a.elapsed_time(b)
            best = ms if best is None else min(best, ms)
        return best / 1e3

    out = {}
    n = 2 << 30
    buf = torch.empty(n, dtype=torch.uint8, device=dev)
    sink = torch.empty(1 << 20, dtype=torch.int32, device=dev)
    lib.dvprobe_stream_write(buf.data_ptr(), n, sh)
    out["hbm_read_GBs"] = n / timed(lambda: lib.dvprobe_stream_read(buf.data_ptr(), n, sink.data_ptr(), sh)) / 1e9
    out["hbm_write_GBs"] = n / timed(lambda: lib.dvprobe_stream_write(buf.data_ptr(), n, sh)) / 1e9
    del buf
    entries = max(1024, table_bytes // 4)
    perm = torch.randperm(entries, device=dev, dtype=torch.int64).to(torch.int32)
    lanes, chains, steps = 524288, 4, 32
    sink = torch.empty(lanes, dtype=torch.int32, device=dev)
    t = timed(lambda: lib.dvprobe_gather(perm.data_ptr(), entries, lanes, chains, steps, sink.data_ptr(), sh))
    out["gather_table_bytes"] = entries * 4
    out["l2_gather_per_s"] = lanes * chains * steps / t
    # the alignment walk's own later moves: 2-byte reads st = table[st * Cp + c]
    # through a state table of the compacted size, 3 chases per lane (the
    # prefix walk's states per block), two 1024-lane blocks per compute unit
    S_tab, Cp = max(1, table_bytes // (98 * 2)), 98
    g = torch.Generator(device=dev)
    g.manual_seed(98)
    tab16 = torch.randint(0, S_tab, (S_tab * Cp,), generator=g, device=dev, dtype=torch.int32).to(torch.int16)
    lanes, steps = 2 * 256 * 1024, 32
    sink = torch.empty(lanes, dtype=torch.int32, device=dev)
    t = timed(lambda: lib.dvprobe_walk_gather(tab16.data_ptr(), S_tab, Cp, lanes, 3, steps, sink.data_ptr(), sh))
    out["walk_gather_table_bytes"] = S_tab * Cp * 2
    out["walk_gather_per_s"] = lanes * 3 * steps / t
    lds_entries = 16384
    sink = torch.empty(131072, dtype=torch.int32, device=dev)
    perm = torch.randperm(lds_entries, device=dev, dtype=torch.int64).to(torch.int32)
    lanes, steps = 131072, 256
    t = timed(lambda: lib.dvprobe_lds_gather(perm.data_ptr(), lds_entries, lanes, chains, steps,
                                             sink.data_ptr(), sh))
    out["lds_gather_per_s"] = lanes * chains * steps / t
    return out


def extra_leg(dv, probes, wid, dev, floors=True):
    """Decode leg of another bandwidth-sized workload: its table built once,
    then its whole greedy chain graph-replayed (inputs resident in HBM),
    with the touched-line roofline, the traffic record and the floors."""
    import numpy as np
    import torch

    import workloads as W

    w = W.WORKLOADS[wid]
    log(f"extra workload: {w.describe()}")
    trans, _ = W.dfa(wid)
    offsets, data = W.vocab(wid)
    init = W.init_states(wid)
    trans_d, offsets_d, data_d, init_d = (torch.from_numpy(np.require(a, requirements=["C", "W"])).to(dev)
                                          for a in (trans, offsets, data, init))
    ns = torch.empty((w.S, w.V), dtype=torch.int32, device=dev)
    al = torch.empty((w.S, w.words), dtype=torch.int32, device=dev)
    ws_align = torch.empty(dv.align_workspace_bytes(w.S, w.V), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    align_ms = []
    if dv.validate_vocab(offsets_d, data_d) != -1:
        raise SystemExit("malformed workload vocabulary")
    for _ in range(4):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        dv.align(trans_d, offsets_d, data_d, next_state=ns, allow=al, workspace=ws_align, validate=False)
        b.record(stream)
        torch.cuda.synchronize()
        align_ms.append(a.elapsed_time(b))
    x = W.logits_all(wid, device=dev)
    ws = dv.step_workspace(w.B, w.V, dev)
    states_all = torch.empty((w.steps + 1, w.B), dtype=torch.int32, device=dev)
    tokens_all = torch.empty((w.steps, w.B), dtype=torch.int32, device=dev)
    states_all[0].copy_(init_d)

    def launches():
        for k in range(w.steps):
            dv.masked_step(ns, al, states_all[k], x[k], token=tokens_all[k], new_state=states_all[k + 1],
                           workspace=ws)

    t = graph_seconds(launches, dev) / w.steps
    live_per_step = (states_all[:-1] >= 0).sum(dim=1).cpu().numpy()
    logit_bytes = [touched_line_bytes(al, states_all[k], x[k].data_ptr(), w.V, w.V, w.elt) for k in range(w.steps)]
    bytes_per_launch = float(np.mean([step_bytes(w, lb, int(n), w.B) for lb, n in zip(logit_bytes, live_per_step)]))
    whole_rows = float(np.mean(live_per_step)) * w.V * w.elt
    achieved = bytes_per_launch / t / 1e9
    out = {"workload": w.describe(), "align_ms": float(np.median(align_ms[1:])),
           "align_per_s": w.S * w.V / (float(np.median(align_ms[1:])) / 1e3),
           "us_per_step": t * 1e6, "steps_per_s": 1.0 / t, "rows_steps_per_s": w.B / t,
           "roofline": {"kernel": "masked_step_bf16_kernel" if w.dtype == "bf16" else "masked_step_kernel",
                        "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": achieved / HBM_PEAK_GBS, "bytes_per_launch": bytes_per_launch,
                        "logit_lines_read_fraction": float(np.mean(logit_bytes)) / whole_rows if whole_rows else None,
                        "traffic": traffic_record("masked_step", wid)}}
    if floors:
        out["floors"] = step_floors(probes, w, al, x, states_all, dev, t * 1e6, bytes_per_launch)
    return out


def bench_spec(dv, w, wid, ns, al, x, tokens_all, states_all, dev, s=8, keep=0.9, reps=3):
    """Speculative verification (Sec. 3.6) over the job's decode chain: window
    k proposes the chain's tokens of steps k(s+1) .. k(s+1)+s-1, each kept with
    probability ``keep`` (else replaced by the next token id), and verifies
    them against the logits of those s + 1 steps, seen as [B][s+1][V] through
    strides.  All windows are captured in one HIP graph; HIP events around
    its replay give the time per verification call."""
    import numpy as np
    import torch

    n_win = w.steps // (s + 1)
    g = torch.Generator(device=dev)
    g.manual_seed(2024)
    props, starts, views = [], [], []
    for k in range(n_win):
        k0 = k * (s + 1)
        p = tokens_all[k0:k0 + s].t().contiguous()
        repl = torch.rand(p.shape, generator=g, device=dev) >= keep
        props.append(torch.where(repl, (p + 1) % w.V, p).to(torch.int32).contiguous())
        starts.append(states_all[k0].clone())
        views.append(x[k0:k0 + s + 1].transpose(0, 1))       # [B][s+1][V], ld_row = V, ld_pos = B V
    tok = torch.empty((n_win, w.B, s + 1), dtype=torch.int32, device=dev)
    acc = torch.empty((n_win, w.B), dtype=torch.int32, device=dev)
    nst = torch.empty((n_win, w.B), dtype=torch.int32, device=dev)
    ws = dv.spec_workspace(w.B, s, w.V, dev)

    def launches():
        for k in range(n_win):
            dv.spec_verify(ns, al, starts[k], props[k], views[k], token=tok[k], accepted=acc[k],
                           new_state=nst[k], workspace=ws)

    launches()
    torch.cuda.synchronize()
    ref = (tok.clone(), acc.clone(), nst.clone())
    graph = capture(launches, dev)
    stream = torch.cuda.current_stream(dev)
    times = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        graph.replay()
        b.record(stream)
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b) / 1e3 / n_win)
    graph.close()
    same = bool(torch.equal(tok, ref[0]) and torch.equal(acc, ref[1]) and torch.equal(nst, ref[2]))
    t = float(np.median(times))
    emitted = float((acc + (tok.gather(2, acc.to(torch.int64)[..., None])[..., 0] != -1)).sum()) / n_win
    # each position's state: the window's start advanced by its first j
    # proposals (DEAD after an illegal one); live positions read logits
    logit_bytes, live = 0, 0
    for k in range(n_win):
        st = starts[k].clone()
        k0 = k * (s + 1)
        for j in range(s + 1):
            logit_bytes += touched_line_bytes(al, st, x[k0 + j].data_ptr(), w.V, w.V, w.elt)
            live += int((st >= 0).sum())
            if j < s:
                p = props[k][:, j].long()
                ok = (st >= 0) & (p >= 0) & (p < w.V)
                nxt = ns[st.clamp(min=0).long(), p.clamp(0, w.V - 1)]
                st = torch.where(ok, nxt, torch.full_like(st, -1))
    live_pos = live / n_win
    bytes_call = (logit_bytes / n_win + live_pos * (4 * w.words + 4)
                  + w.B * (s * 12 + (s + 1) * 4 + 12))
    achieved = bytes_call / t / 1e9
    return {
        "proposed_per_row": s, "keep_probability": keep, "calls": n_win,
        "us_per_call": t * 1e6, "calls_per_s": 1.0 / t,
        "emitted_tokens_per_s": emitted / t, "positions_per_s": w.B * (s + 1) / t,
        "mean_accepted": float(acc.float().mean()), "live_positions_per_call": live_pos,
        "graph_matches_eager": same,
        "roofline": {"kernel": "masked_step_bf16_kernel over B(s+1) positions + spec_accept_kernel"
                     if w.dtype == "bf16" else "masked_step_kernel over B(s+1) positions",
                     "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "bytes_per_launch": bytes_call,
                     "traffic": traffic_record("spec_verify", wid) if s == 8 else None},
    }


def bench_opportunistic(dv, w, ns, al, x, tokens_all, states_all, dev, adherent=(0.9, 1.0), reps=3):
    """Opportunistic masking (Sec. 3.5): the job's decode chain with the model's
    own choice checked first, on the workload's logits and on copies in which
    a fraction ``adherent`` of the row-steps favour the chain's own (allowed)
    choice -- raising the chosen logit leaves the chain unchanged.  With every
    row-step adherent no row is read twice: the time is that of the
    unconstrained greedy pass alone.  Each chain
    is captured as a HIP graph and replayed; the check's hit rate is the
    fraction of live row-steps whose overall argmax is allowed."""
    import numpy as np
    import torch

    steps = tokens_all.shape[0]
    ws = dv.step_workspace(w.B, w.V, dev)
    sts = torch.empty_like(states_all)
    tks = torch.empty_like(tokens_all)
    stream = torch.cuda.current_stream(dev)

    def timed_chain(xv):
        def launches():
            for k in range(steps):
                dv.masked_step(ns, al, sts[k], xv[k], token=tks[k], new_state=sts[k + 1], workspace=ws,
                               opportunistic=True)
        sts[0].copy_(states_all[0])
        launches()
        torch.cuda.synchronize()
        same_eager = bool(torch.equal(tks, tokens_all))
        graph = capture(launches, dev)
        times = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            graph.replay()
            b.record(stream)
            torch.cuda.synchronize()
            times.append(a.elapsed_time(b) / 1e3 / steps)
        graph.close()
        same = same_eager and bool(torch.equal(tks, tokens_all))
        free = torch.stack([xv[k].float().argmax(dim=1) for k in range(steps)]).to(torch.int64)
        st = states_all[:-1].to(torch.int64)
        live = st >= 0
        word = al[st.clamp(min=0), free // 32].to(torch.int64) & 0xFFFFFFFF
        hit = ((word >> (free % 32)) & 1).bool() & live
        return {"us_per_step": float(np.median(times)) * 1e6, "matches_masked_step": same,
                "check_hit_rate": float(hit.sum()) / max(int(live.sum()), 1)}

    out = {"random_logits": timed_chain(x)}
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    u = torch.rand(tokens_all.shape, generator=g, device=dev)
    for frac in adherent:
        pick = (u < frac) & (tokens_all >= 0)
        k_idx, b_idx = torch.nonzero(pick, as_tuple=True)
        xa = x.clone()
        xa[k_idx, b_idx, tokens_all[k_idx, b_idx].to(torch.int64)] = 30.0
        out[f"adherent_{frac:g}"] = timed_chain(xa)
        del xa
    return out


# Algorithmic VALU work of a sampled step, in full-rate lane-op slots: a
# Gumbel-noised allowed token costs two binary32 logarithms (25 each: the
# exponent split, a four-step Newton reciprocal, the series, the final fma),
# the uniform (4) and the key (3); a Philox4x32-10 call, per 4-token group
# with an allowed token, costs 10 rounds of two 32x32->64 multiplies (quarter
# rate: 4 slots each) and 4 other operations.
SAMPLE_OPS_PER_TOKEN = 57
SAMPLE_OPS_PER_GROUP = 120
VALU_PEAK_OPS = 256 * 64 * 2.4e9   # CUs x lanes per clock x clock (no packed math)


def bench_sample(dv, w, ns, al, x, init_d, dev, seed=2024, reps=3):
    """Masked sampling at temperature 1 (Sec. 4): the job's decode chain with
    dv_masked_sample in place of the greedy step (step k uses offset k),
    captured as a HIP graph and replayed."""
    import numpy as np
    import torch

    steps = x.shape[0]
    ws = dv.sample_workspace(w.B, w.V, dev)
    sts = torch.empty((steps + 1, w.B), dtype=torch.int32, device=dev)
    tks = torch.empty((steps, w.B), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def launches():
        for k in range(steps):
            dv.masked_sample(ns, al, sts[k], x[k], seed, k, token=tks[k], new_state=sts[k + 1], workspace=ws)

    sts[0].copy_(init_d)
    launches()
    torch.cuda.synchronize()
    ref = (tks.clone(), sts.clone())
    graph = capture(launches, dev)
    times = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        graph.replay()
        b.record(stream)
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b) / 1e3 / steps)
    graph.close()
    same = bool(torch.equal(tks, ref[0]) and torch.equal(sts, ref[1]))
    t = float(np.median(times))
    # work along the chain: allowed tokens and 4-token groups holding one
    pop8 = torch.tensor([bin(i).count("1") for i in range(256)], dtype=torch.int64, device=dev)
    allowed = groups = 0
    for k in range(steps):
        st = sts[k].to(torch.int64)
        rows = al[st.clamp(min=0)][st >= 0].to(torch.int64) & 0xFFFFFFFF
        for sh in (0, 8, 16, 24):
            allowed += int(pop8[(rows >> sh) & 0xFF].sum())
        nz = (rows | (rows >> 1) | (rows >> 2) | (rows >> 3)) & 0x11111111
        for sh in (0, 8, 16, 24):
            groups += int(pop8[(nz >> sh) & 0xFF].sum())
    ops = (allowed * SAMPLE_OPS_PER_TOKEN + groups * SAMPLE_OPS_PER_GROUP) / steps
    achieved = ops / t
    return {"us_per_step": t * 1e6, "steps_per_s": 1.0 / t, "temperature": 1.0,
            "allowed_tokens_per_step": allowed / steps, "groups_per_step": groups / steps,
            "graph_matches_eager": same,
            "roofline": {"kernel": "masked_sample_kernel", "bound": "alu",
                         "achieved": achieved / 1e9, "peak": VALU_PEAK_OPS / 1e9, "unit": "Gop/s",
                         "frac": achieved / VALU_PEAK_OPS, "ops_per_launch": ops,
                         "note": f"{SAMPLE_OPS_PER_TOKEN} ops per noised token + {SAMPLE_OPS_PER_GROUP} per "
                                 "Philox call, full-rate lane-op slots; peak = 256 CUs x 64 lanes x 2.4 GHz"}}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the multi-GPU "
              "sharding of this path is a design, not a measurement.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2403_06988_amd as dv
    import workloads as W

    wid = args.workload
    w = W.WORKLOADS[wid]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)

    log(f"inputs: {w.describe()}")
    trans, _ = W.dfa(wid)
    offsets, data = W.vocab(wid)
    init = W.init_states(wid)
    # the workload arrays are cached read-only; torch wants writable ones
    trans_d, offsets_d, data_d, init_d = (torch.from_numpy(np.require(a, requirements=["C", "W"])).to(dev)
                                          for a in (trans, offsets, data, init))
    x = W.logits_all(wid, device=dev)
    ns = torch.empty((w.S, w.V), dtype=torch.int32, device=dev)
    al = torch.empty((w.S, w.words), dtype=torch.int32, device=dev)
    ws_align = torch.empty(dv.align_workspace_bytes(w.S, w.V), dtype=torch.uint8, device=dev)
    ws_step = dv.step_workspace(w.B, w.V, dev)
    states_all = torch.empty((w.steps + 1, w.B), dtype=torch.int32, device=dev)
    tokens_all = torch.empty((w.steps, w.B), dtype=torch.int32, device=dev)
    torch.cuda.synchronize()
    log("inputs resident in HBM")

    def decode_launches():
        for k in range(w.steps):
            dv.masked_step(ns, al, states_all[k], x[k], token=tokens_all[k],
                           new_state=states_all[k + 1], workspace=ws_step)

    if dv.validate_vocab(offsets_d, data_d) != -1:      # checked once, outside the timed region
        raise SystemExit("malformed workload vocabulary")

    def align_launch():
        dv.align(trans_d, offsets_d, data_d, next_state=ns, allow=al, workspace=ws_align, validate=False)

    # Eager warm-up (also the reference the graph replays are checked against).
    for _ in range(args.warmup):
        align_launch()
        states_all[0].copy_(init_d)
        decode_launches()
    torch.cuda.synchronize()
    eager_tokens = tokens_all.clone()
    eager_states = states_all.clone()

    # The per-token decode loop is launch-bound from Python (a ctypes call per
    # step costs more host time than the kernel takes), so it is captured once
    # in a HIP graph and replayed, as a serving loop would run it.
    states_all[0].copy_(init_d)
    graph = capture(decode_launches, dev)
    stream = torch.cuda.current_stream(dev)

    def mk():
        return torch.cuda.Event(enable_timing=True)

    ev = [(mk(), mk(), mk(), mk()) for _ in range(args.steps)]
    graph_ok = True
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for j in range(args.steps):
        a0, a1, d0, d1 = ev[j]
        a0.record(stream)
        align_launch()
        a1.record(stream)
        states_all[0].copy_(init_d)
        d0.record(stream)
        graph.replay()
        d1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    graph.close()
    graph_ok = bool(torch.equal(tokens_all, eager_tokens) and torch.equal(states_all, eager_states))

    align_ms = [a0.elapsed_time(a1) for (a0, a1, _, _) in ev]
    decode_ms = [d0.elapsed_time(d1) for (_, _, d0, d1) in ev]
    live_per_step = (states_all[:-1] >= 0).sum(dim=1).cpu().numpy()
    dead_final = int((states_all[-1] < 0).sum())

    pairs = w.S * w.V
    align_s = float(np.mean(align_ms)) / 1e3
    dec_s = float(np.mean(decode_ms)) / 1e3
    logit_bytes = [touched_line_bytes(al.view(torch.int32), states_all[k], x[k].data_ptr(), w.V, w.V, w.elt)
                   for k in range(w.steps)]
    bytes_per_launch = float(np.mean([step_bytes(w, lb, int(n), w.B)
                                      for lb, n in zip(logit_bytes, live_per_step)]))
    whole_rows = float(np.mean(live_per_step)) * w.V * w.elt
    mean_launch_s = dec_s / w.steps
    achieved = bytes_per_launch / mean_launch_s / 1e9
    align_bytes = pairs * 4.125
    align_achieved = align_bytes / align_s / 1e9

    out = {
        "metric": METRIC,
        "value": w.steps / dec_s,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded DFA, vocabulary and logits; no model weights)",
        "config": {"workload": w.describe(), "S": w.S, "V": w.V, "B": w.B,
                   "decode_steps_per_job": w.steps, "logits_dtype": w.dtype},
        "align": {"value": pairs / align_s, "unit": "alignments/s", "ms": align_s * 1e3},
        "decode": {"us_per_step_mean": mean_launch_s * 1e6,
                   "us_per_job_min": float(np.min(decode_ms)) * 1e3,
                   "launch": "HIP graph of the job's decode steps, replayed",
                   "graph_matches_eager": graph_ok,
                   "rows_steps_per_s": w.B * w.steps / dec_s,
                   "live_rows_first_last": [int(live_per_step[0]), int(live_per_step[-1])],
                   "dead_rows_at_end": dead_final},
        "roofline": {"kernel": "masked_step_bf16_kernel" if w.dtype == "bf16" else "masked_step_kernel",
                     "bound": "hbm", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "bytes_per_launch": bytes_per_launch,
                     "logit_lines_read_fraction": float(np.mean(logit_bytes)) / whole_rows if whole_rows else None,
                     "traffic": traffic_record("masked_step", wid)},
        "roofline_align": {"kernel": f"dv_align ({align_walk_kind(trans)}, with the prep kernels)", "bound": "hbm",
                           "achieved": align_achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                           "frac": align_achieved / HBM_PEAK_GBS, "bytes_per_launch": align_bytes,
                           "traffic": traffic_record("align", wid)},
        "kernel_source_hash": {k: kernel_source_hash(k) for k in KERNEL_SOURCES},
        "inputs": inputs_record(trans, offsets, data, init),
    }
    probes = probe_lib() if not (args.no_probes and args.no_floors) else None
    if not args.no_floors and w.dtype == "bf16":
        log("masked-step floors")
        out["floors"] = step_floors(probes, w, al, x, states_all, dev, mean_launch_s * 1e6, bytes_per_launch)
    if not args.no_opportunistic and w.dtype == "bf16":
        log("opportunistic masking")
        out["opportunistic"] = bench_opportunistic(dv, w, ns, al, x, tokens_all, states_all, dev)
        out["opportunistic"]["masked_us_per_step"] = mean_launch_s * 1e6
    if not args.no_sample:
        log("masked sampling")
        out["sample"] = bench_sample(dv, w, ns, al, x, init_d, dev)
    if not args.no_spec:
        log("speculative verification")
        out["spec_verify"] = bench_spec(dv, w, wid, ns, al, x, tokens_all, states_all, dev)
    if not args.no_probes:
        log("roofline probes")
        out["probes"] = run_probes(probes, dev, w.S * 96 * 2)
        # the same achieved rates against what this box's streaming probes reach
        out["roofline"]["frac_of_measured_read"] = achieved / out["probes"]["hbm_read_GBs"]
        out["roofline_align"]["frac_of_measured_write"] = align_achieved / out["probes"]["hbm_write_GBs"]
    if not args.no_cpu:
        log("cpu baseline (oracle, 1 thread)")
        out["cpu_baseline"] = cpu_baseline(w, wid, trans, offsets, data, init, x, args.cpu_seconds)
    kind = align_walk_kind(trans)
    if "probes" in out and "cpu_baseline" in out and "whole" not in kind:
        # dv_align's gathers for random DFAs: every move past the part of the
        # walk served from LDS is a random read of the L2-resident table
        depth = 2 if kind == "walk_prefix_kernel" else 1
        later = out["cpu_baseline"][f"moves_past_byte_{depth}_per_pair"] * pairs / align_s
        peak = out["probes"]["walk_gather_per_s"]
        out["roofline_align_l2"] = {"kernel": kind, "bound": "l2_gather", "achieved": later,
                                    "peak": peak, "unit": "gathers/s", "frac": later / peak,
                                    "note": f"gathers = table moves past byte {depth} (the LDS part of the walk); "
                                            "peak = measured rate of the walk-pattern gather probe (2-byte reads "
                                            "st = table[st * Cp + c] through a table of the compacted size, "
                                            "3 chases per lane, two 1024-lane blocks per compute unit); "
                                            "gathers that hit L1 can push frac above 1"}
    if not args.no_extra:
        out["extra"] = {}
        for e in EXTRA_WORKLOADS:
            if e != wid:
                out["extra"][str(e)] = extra_leg(dv, probes or probe_lib(), e, dev, floors=not args.no_floors)
                torch.cuda.empty_cache()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
