"""GPU parity at the two largest workloads, in full, against the oracle.

Workload 4 (grammar-lexer union: S = 8,192, V = 128,256, B = 256 x 256
steps) and workload 5 (large vocabulary: S = 4,096, V = 256,000, B = 1,024
x 128 steps) hold about 10^9 (state, token) pairs each.  Compared bit for
bit, in the benchmark's launch configuration:

* every state row of the alignment table (next_state and allow words,
  padding bits included; Sec. 3.3, Algorithm 2);
* every row-step of the greedy decoding chain (token and new state at each
  step, the oracle using its own table and its own previous states;
  Algorithm 1);
* one full batch of the speculative verification (Sec. 3.6), of the
  opportunistic step (Sec. 3.5) and a short sampled chain (Algorithm 1's
  decode by sampling, T = 1).

The oracle runs as it stands: its own functions, called on blocks of 512
table rows or on slices of the batch, spread over a thread pool (ctypes
releases the interpreter lock around each C call).  Sampling draws row b's
noise from the row's position in the batch, so each sampled step is one
oracle call over the whole batch."""
import concurrent.futures as cf
import dataclasses
import os

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from tests.gpu_common import run_chain, to_oracle, u32

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
BLOCK = 512
THREADS = max(1, min(16, len(os.sched_getaffinity(0))))
SEED = 0x5EED_0000_0000_2403


def _say(msg):
    print(msg, flush=True)


def _dev(a):
    return torch.from_numpy(np.require(a, requirements=["C", "W"])).to(DEV)


def _pmap(fn, items):
    with cf.ThreadPoolExecutor(THREADS) as pool:
        return list(pool.map(fn, items))


def _slices(n, parts=4 * THREADS):
    step = max(1, -(-n // parts))
    return [slice(i, min(n, i + step)) for i in range(0, n, step)]


@pytest.fixture(scope="module")
def dv():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2403_06988_amd as dv_mod
    return dv_mod


@dataclasses.dataclass
class Big:
    wid: int
    w: W.Workload
    trans: np.ndarray
    offsets: np.ndarray
    data: np.ndarray
    ns: torch.Tensor          # the device's table
    al: torch.Tensor
    ns_o: np.ndarray          # the oracle's table
    al_o: np.ndarray


@pytest.fixture(scope="module", params=[4, 5], ids=lambda wid: f"workload{wid}")
def big(request, dv):
    wid = request.param
    w = W.WORKLOADS[wid]
    _say(f"[large] {w.describe()}: device table, then the oracle's in blocks of {BLOCK} rows "
         f"on {THREADS} threads")
    torch.cuda.empty_cache()
    trans, _ = W.dfa(wid)
    offsets, data = W.vocab(wid)
    ns, al = dv.align(_dev(trans), _dev(offsets), _dev(data))
    torch.cuda.synchronize()
    ns_o = np.empty((w.S, w.V), np.int32)
    al_o = np.empty((w.S, w.words), np.uint32)

    def block(r0):
        rows = np.arange(r0, min(r0 + BLOCK, w.S), dtype=np.int32)
        a, b = oracle.align_rows(trans, offsets, data, rows)
        ns_o[r0:r0 + rows.size] = a
        al_o[r0:r0 + rows.size] = b

    _pmap(block, range(0, w.S, BLOCK))
    yield Big(wid, w, trans, offsets, data, ns, al, ns_o, al_o)
    del ns, al
    torch.cuda.empty_cache()


def _oracle_step(b: Big, states, xs):
    """The oracle's greedy step over the batch, slices of rows in parallel."""
    B = states.shape[0]
    tok = np.empty(B, np.int32)
    new = np.empty(B, np.int32)

    def part(sl):
        tok[sl], new[sl] = oracle.masked_step(b.ns_o, b.al_o, states[sl], xs[sl])

    _pmap(part, _slices(B))
    return tok, new


def _first_difference(got, want):
    bad = np.argwhere(got != want)
    i = tuple(bad[0])
    return f"{bad.shape[0]} differences, first at {i}: device {got[i]} oracle {want[i]}"


def test_align_table_full(big):
    """Every state row of next_state and allow."""
    w = big.w
    for r0 in range(0, w.S, BLOCK):
        r1 = min(w.S, r0 + BLOCK)
        g = big.ns[r0:r1].cpu().numpy()
        o = big.ns_o[r0:r1]
        assert np.array_equal(g, o), f"workload {big.wid} next_state rows {r0}-{r1}: {_first_difference(g, o)}"
        g = u32(big.al[r0:r1])
        o = big.al_o[r0:r1]
        assert np.array_equal(g, o), f"workload {big.wid} allow rows {r0}-{r1}: {_first_difference(g, o)}"
    _say(f"[large] workload {big.wid}: {w.S} x {w.V} table bit-exact")


def test_greedy_chain_full(dv, big):
    """Every row at every step of the benchmark's decode chain."""
    w = big.w
    init = W.init_states(big.wid)
    x = W.logits_all(big.wid, device=DEV)
    ws = dv.step_workspace(w.B, w.V, DEV)
    toks, sts = run_chain(dv, big.ns, big.al, _dev(init), x, ws)
    torch.cuda.synchronize()
    toks_h, sts_h = toks.cpu().numpy(), sts.cpu().numpy()
    cur = init
    for k in range(w.steps):
        t_o, n_o = _oracle_step(big, cur, to_oracle(x[k]))
        assert np.array_equal(toks_h[k], t_o), f"workload {big.wid} step {k} token: " \
                                               f"{_first_difference(toks_h[k], t_o)}"
        assert np.array_equal(sts_h[k + 1], n_o), f"workload {big.wid} step {k} new_state: " \
                                                  f"{_first_difference(sts_h[k + 1], n_o)}"
        cur = n_o
    del x
    _say(f"[large] workload {big.wid}: {w.B} rows x {w.steps} steps bit-exact, "
         f"{int((cur == -1).sum())} rows died")


def _perturb(rng, greedy, V, keep):
    other = rng.integers(-2, V + 2, greedy.shape).astype(np.int32)
    return np.where(rng.random(greedy.shape) < keep, greedy, other).astype(np.int32)


def test_spec_verify_full_batch(dv, big):
    """Speculative verification of every row (s = 8 at workload 4, the
    benchmark's, s = 4 at workload 5): proposals follow the oracle's greedy
    choices with probability 0.85 per position, else random ids."""
    w = big.w
    s = 8 if big.wid == 4 else 4
    x = W.logits_all(big.wid, device=DEV, steps=s + 1).transpose(0, 1).contiguous()   # [B][s+1][V]
    xs = to_oracle(x)
    init = W.init_states(big.wid)
    rng = np.random.default_rng(700 + big.wid)
    greedy = np.empty((w.B, s), np.int32)
    cur = init
    for j in range(s):
        greedy[:, j], cur = _oracle_step(big, cur, np.ascontiguousarray(xs[:, j]))
    props = _perturb(rng, greedy, w.V, 0.85)
    tok, acc, nst = dv.spec_verify(big.ns, big.al, _dev(init), _dev(props), x)
    torch.cuda.synchronize()
    t_o = np.empty((w.B, s + 1), np.int32)
    a_o = np.empty(w.B, np.int32)
    n_o = np.empty(w.B, np.int32)

    def part(sl):
        t_o[sl], a_o[sl], n_o[sl] = oracle.spec_verify(big.ns_o, big.al_o, init[sl], props[sl], xs[sl])

    _pmap(part, _slices(w.B))
    g = tok.cpu().numpy()
    assert np.array_equal(g, t_o), f"workload {big.wid} spec tokens: {_first_difference(g, t_o)}"
    assert np.array_equal(acc.cpu().numpy(), a_o)
    assert np.array_equal(nst.cpu().numpy(), n_o)
    _say(f"[large] workload {big.wid}: spec verify s={s}, {w.B} rows bit-exact, "
         f"mean accepted {a_o.mean():.2f}")


@pytest.mark.parametrize("adherent", [0.0, 0.9])
def test_opportunistic_full_batch(dv, big, adherent):
    """The check-first step over every row, against the oracle's
    opportunistic step; ``adherent``: the fraction of rows whose logits
    favour an allowed token (one taken from the oracle's table row)."""
    w = big.w
    init = W.init_states(big.wid)
    x = W.logits(big.wid, 0, device=DEV)
    rng = np.random.default_rng(800 + big.wid)
    if adherent:
        pick = np.nonzero(rng.random(w.B) < adherent)[0]
        cols = []
        for r in pick:
            ok = np.nonzero(big.ns_o[init[r]] != -1)[0]
            cols.append(int(ok[rng.integers(0, ok.size)]) if ok.size else 0)
        x[torch.from_numpy(pick).to(DEV), torch.from_numpy(np.array(cols, np.int64)).to(DEV)] = 30.0
    tok, new = dv.masked_step(big.ns, big.al, _dev(init), x, opportunistic=True)
    torch.cuda.synchronize()
    xs = to_oracle(x)
    t_o = np.empty(w.B, np.int32)
    n_o = np.empty(w.B, np.int32)
    hit = np.empty(w.B, bool)

    def part(sl):
        t_o[sl], n_o[sl], hit[sl] = oracle.masked_step_opportunistic(big.ns_o, big.al_o, init[sl], xs[sl])

    _pmap(part, _slices(w.B))
    assert np.array_equal(tok.cpu().numpy(), t_o)
    assert np.array_equal(new.cpu().numpy(), n_o)
    _say(f"[large] workload {big.wid}: opportunistic step, {w.B} rows bit-exact, check passed for "
         f"{hit.mean():.3f} of rows")


def test_sampled_chain_full_batch(dv, big):
    """A sampled chain at T = 1 (offset = step) over every row: 4 steps at
    workload 4, 2 at workload 5."""
    w = big.w
    steps = 4 if big.wid == 4 else 2
    init = W.init_states(big.wid)
    x = W.logits_all(big.wid, device=DEV, steps=steps)
    ws = dv.sample_workspace(w.B, w.V, DEV)
    states = _dev(init)
    cur = init
    for k in range(steps):
        tok, new = dv.masked_sample(big.ns, big.al, states, x[k], SEED + big.wid, k, workspace=ws)
        torch.cuda.synchronize()
        t_o, n_o = oracle.masked_sample(big.ns_o, big.al_o, cur, to_oracle(x[k]), 1.0, SEED + big.wid, k)
        g = tok.cpu().numpy()
        assert np.array_equal(g, t_o), f"workload {big.wid} sampled step {k}: {_first_difference(g, t_o)}"
        assert np.array_equal(new.cpu().numpy(), n_o)
        states, cur = new, n_o
    _say(f"[large] workload {big.wid}: sampled chain, {w.B} rows x {steps} steps bit-exact")
