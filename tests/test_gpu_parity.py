"""GPU parity: the HIP path against the CPU oracle, bit for bit.

Alignment tables (next_state, allow with padding bits) and greedy decoding
chains (token, new_state at every step) are compared with the oracle, which
computes from the same seeded inputs with its own table and its own previous
states.  Workloads 1-3 and 6-10 are compared in full here; workloads 4-5
(10^9-pair tables) in full in test_gpu_parity_large.py.  The launch
configuration is the benchmark's (same shapes, same calls)."""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from tests.gpu_common import run_chain, to_oracle, u32

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module")
def dv():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2403_06988_amd as dv_mod
    return dv_mod


DEV = torch.device("cuda:0")


def _dev(a):
    # a copy only where the array is not contiguous or is read-only (cached tables)
    return torch.from_numpy(np.require(a, requirements=["C", "W"])).to(DEV)


def _align(dv, trans, offsets, data):
    ns, al = dv.align(_dev(trans), _dev(offsets), _dev(data if len(data) else np.zeros(1, np.uint8)))
    torch.cuda.synchronize()
    return ns, al


def _say(msg):
    print(msg, flush=True)


# ------------------------------------------------------------- worked examples

@pytest.mark.parametrize("name", ["fig_nfa_int.json", "fig_overview_scanner.json"])
def test_align_paper_examples(dv, name):
    g = json.load(open(os.path.join(GOLDEN, name)))
    trans = W.dfa_from_spec(len(g["states"]), g["moves"])
    offsets, data = W.vocab_from_tokens([t.encode() for t in g["vocab"]])
    ns, al = _align(dv, trans, offsets, data)
    ns_o, al_o = oracle.align(trans, offsets, data)
    np.testing.assert_array_equal(ns.cpu().numpy(), ns_o)
    np.testing.assert_array_equal(u32(al), al_o)
    if "expected_next_state" in g:
        np.testing.assert_array_equal(ns.cpu().numpy(), np.array(g["expected_next_state"]))


# ------------------------------------------------------------ alignment edges

def _random_case(seed, S, V, max_len, p_empty=0.0, junk=True, alphabet=None):
    rng = np.random.default_rng(seed)
    alphabet = alphabet if alphabet is not None else np.arange(256)
    trans = np.full((S, 256), -1, np.int32)
    for s in range(S):
        k = int(rng.integers(1, len(alphabet) + 1))
        cols = rng.choice(alphabet, size=k, replace=False)
        trans[s, cols] = rng.integers(0, S, size=k)
    if junk:
        mask = rng.random(trans.shape) < 0.05
        trans[mask] = rng.choice(np.array([S, S + 7, -2, -(1 << 30), 1 << 30], np.int32), mask.sum())
    toks = []
    for _ in range(V):
        L = 0 if rng.random() < p_empty else int(rng.integers(1, max_len + 1))
        toks.append(bytes(rng.choice(alphabet, size=L).astype(np.uint8)))
    offsets, data = W.vocab_from_tokens(toks)
    return trans, offsets, data


@pytest.mark.parametrize("S,V,max_len,p_empty", [
    (1, 1, 3, 0.0), (3, 31, 4, 0.0), (5, 33, 4, 0.1), (7, 63, 5, 0.0), (9, 64, 5, 0.0),
    (33, 65, 6, 0.0), (40, 1023, 6, 0.05), (64, 1025, 8, 0.0), (100, 4097, 12, 0.02),
    (37, 3000, 200, 0.0),                   # a few very long tokens
])
def test_align_edge_shapes(dv, S, V, max_len, p_empty):
    _say(f"align edge S={S} V={V} max_len={max_len}")
    trans, offsets, data = _random_case(S * 1000 + V, S, V, max_len, p_empty,
                                        alphabet=np.arange(0x20, 0x30))
    ns, al = _align(dv, trans, offsets, data)
    ns_o, al_o = oracle.align(trans, offsets, data)
    np.testing.assert_array_equal(ns.cpu().numpy(), ns_o)
    np.testing.assert_array_equal(u32(al), al_o)


@pytest.mark.parametrize("S,V,max_len,p_empty,alphabet,eos", [
    (513, 2100, 12, 0.02, 48, None),      # odd S: the last state tile has one state
    (1025, 1500, 9, 0.0, 256, None),      # every byte live: Cp = 256
    (700, 4097, 40, 0.05, 100, 17),       # long tokens (bytes past the eighth), EOS column
    (600, 999, 2, 0.3, 126, 998),         # Cp = 128 (126 live classes + the dead class)
    (700, 4097, 40, 0.05, 90, 17),        # prefix-table walk: long tokens, empty tokens, EOS
    (900, 3000, 10, 0.01, 97, None),      # Cp = 98, the largest prefix table
    (900, 3000, 10, 0.01, 98, 5),         # Cp = 100: the tile walk, beside an idle prefix walk
    (600, 70000, 6, 0.0, 200, None),      # tile walk on a strided grid (more tiles than blocks)
    (400, 140000, 5, 0.0, 30, None),      # whole table in LDS, strided grid
    (400, 5000, 8, 0.0, 94, 4999),        # S <= 512 but too large whole: prefix walk, 3 token ranges
    (3000, 5000, 40, 0.01, 2, 4999),      # prefix walk, Cp = 4: most walks survive past the eighth byte
    (2000, 3000, 60, 0.0, 3, None),       # prefix walk, Cp = 4, tokens up to 60 bytes
    (65535, 300, 12, 0.02, 90, 7),        # the largest state count: prefix walk, DEAD = 0xFFFF = S
    (65535, 300, 12, 0.0, 200, None),     # the largest state count: tile walk
])
def test_align_large_dfa(dv, S, V, max_len, p_empty, alphabet, eos):
    """DFAs too large to stage whole in LDS: the prefix-table walk (tables of
    at most 98 columns: the states two byte classes away come from LDS) or
    the tile walk (its row tile in LDS), both reading later moves from the
    L2-resident table; and the whole-table walk on a strided grid."""
    _say(f"align large S={S} V={V} max_len={max_len} alphabet={alphabet} eos={eos}")
    trans, offsets, data = _random_case(S * 7 + V, S, V, max_len, p_empty, alphabet=np.arange(alphabet))
    if eos is None:
        ns, al = _align(dv, trans, offsets, data)
        ns_o, al_o = oracle.align(trans, offsets, data)
    else:
        acc = (np.random.default_rng(S).random(S) < 0.3).astype(np.uint8)
        ns, al = dv.align(_dev(trans), _dev(offsets), _dev(data), accepting=_dev(acc), eos_token=eos)
        torch.cuda.synchronize()
        ns_o, al_o = oracle.align_eos(trans, offsets, data, acc, eos)
    np.testing.assert_array_equal(ns.cpu().numpy(), ns_o)
    np.testing.assert_array_equal(u32(al), al_o)


@pytest.mark.parametrize("S,live_lo,eos", [(2000, 128, None), (1500, 200, 11)])
def test_align_wide_alphabet_long_walks(dv, S, live_lo, eos):
    """A DFA too large to stage whole with most of the 256 bytes live from
    every state, over BPE-like tokens: walks survive for several bytes (3-4
    moves per pair), so the tile walk's lockstep groups run long."""
    _say(f"align wide alphabet S={S} live>={live_lo} eos={eos}")
    rng = np.random.default_rng(S + live_lo)
    trans = np.full((S, 256), -1, np.int32)
    for s in range(S):
        k = int(rng.integers(live_lo, 257))
        cols = rng.choice(256, size=k, replace=False)
        trans[s, cols] = rng.integers(0, S, size=k)
    offsets, data = W.vocab(8)
    V = 4000
    offsets, data = offsets[:V + 1].copy(), data[:offsets[V]].copy()
    if eos is None:
        ns, al = _align(dv, trans, offsets, data)
        ns_o, al_o = oracle.align(trans, offsets, data)
    else:
        acc = (rng.random(S) < 0.2).astype(np.uint8)
        ns, al = dv.align(_dev(trans), _dev(offsets), _dev(data), accepting=_dev(acc), eos_token=eos)
        torch.cuda.synchronize()
        ns_o, al_o = oracle.align_eos(trans, offsets, data, acc, eos)
    np.testing.assert_array_equal(ns.cpu().numpy(), ns_o)
    np.testing.assert_array_equal(u32(al), al_o)


def test_align_all_tokens_empty(dv):
    trans = np.zeros((4, 256), np.int32)
    offsets = np.zeros(70, np.int32)
    ns, al = _align(dv, trans, offsets, np.zeros(0, np.uint8))
    ns_o, al_o = oracle.align(trans, offsets, np.zeros(0, np.uint8))
    np.testing.assert_array_equal(ns.cpu().numpy(), ns_o)
    np.testing.assert_array_equal(u32(al), al_o)


def test_align_all_transitions_dead(dv):
    trans = np.full((5, 256), -1, np.int32)
    trans[2, 7] = 99  # out of range: still dead
    offsets, data = W.vocab(1)
    ns, al = _align(dv, trans, offsets, data)
    assert (ns.cpu().numpy() == -1).all() and (u32(al) == 0).all()


@pytest.mark.parametrize("dead_byte", [None, 0xFF, 0x00, 0x80])
def test_align_every_byte_value(dv, dead_byte):
    """All 256 bytes live (C = 256 classes, no spare class for dead bytes), or
    all but one (C = 255: the dead byte's class is the last one).  Every
    single-byte token and tokens through the dead byte are walked."""
    rng = np.random.default_rng(5)
    S = 50
    trans = rng.integers(0, S, size=(S, 256)).astype(np.int32)
    if dead_byte is not None:
        trans[:, dead_byte] = -1
    toks = [bytes([b]) for b in range(256)] + [bytes(rng.integers(0, 256, 3).astype(np.uint8))
                                               for _ in range(700)]
    toks += [bytes([0x41, b, 0x42]) for b in (0x00, 0x80, 0xFF)]
    offsets, data = W.vocab_from_tokens(toks)
    ns, al = _align(dv, trans, offsets, data)
    ns_o, al_o = oracle.align(trans, offsets, data)
    np.testing.assert_array_equal(ns.cpu().numpy(), ns_o)
    np.testing.assert_array_equal(u32(al), al_o)


def test_validate_vocab_and_decreasing_offsets(dv):
    """dv_validate_vocab finds the first index at which the CSR layout breaks;
    align refuses such a vocabulary; a decreasing pair whose bytes all lie in
    the buffer, aligned without the check, is an empty token on both sides
    (the oracle walks the empty range)."""
    trans, _ = W.dfa(2)
    offsets, data = W.vocab(2)
    V = offsets.shape[0] - 1
    assert dv.validate_vocab(_dev(offsets), _dev(data)) == -1
    bad = offsets.copy()
    bad[0] = 1
    assert dv.validate_vocab(_dev(bad), _dev(data)) == 0
    bad = offsets.copy()
    bad[700] = bad[699] - 1
    assert dv.validate_vocab(_dev(bad), _dev(data)) == 700
    assert dv.validate_vocab(_dev(offsets), _dev(data[:-1])) == V       # ends past the bytes
    bad = offsets.copy()
    bad[V - 5:] = offsets[V] + 7
    assert dv.validate_vocab(_dev(bad), _dev(data)) == V - 5               # the first entry past the bytes
    with pytest.raises(ValueError):
        dv.align(_dev(trans), _dev(bad), _dev(data))
    # a decreasing pair inside the buffer: token 1000 spans [o[1000], o[999]) backwards
    dec = offsets.copy()
    dec[1000] = offsets[998]
    assert dv.validate_vocab(_dev(dec), _dev(data)) == 1000
    ns, al = dv.align(_dev(trans), _dev(dec), _dev(data), validate=False)
    torch.cuda.synchronize()
    ns_o, al_o = oracle.align(trans, dec, data)
    np.testing.assert_array_equal(ns.cpu().numpy(), ns_o)
    np.testing.assert_array_equal(u32(al), al_o)
    assert (ns_o[:, 999] == np.arange(trans.shape[0])).all()          # empty: the state is kept


def test_align_is_deterministic(dv):
    trans, _ = W.dfa(2)
    offsets, data = W.vocab(2)
    a = _align(dv, trans, offsets, data)
    b = _align(dv, trans, offsets, data)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


# --------------------------------------------------------- workload tables

class _Cache:
    wid = None
    data = None


def _workload_table(dv, wid):
    if _Cache.wid != wid:
        _Cache.wid, _Cache.data = None, None
        torch.cuda.empty_cache()
        trans, _ = W.dfa(wid)
        offsets, data = W.vocab(wid)
        ns, al = _align(dv, trans, offsets, data)
        _Cache.wid, _Cache.data = wid, (trans, offsets, data, ns, al)
    return _Cache.data


@pytest.mark.parametrize("wid", [1, 2, 3, 6, 7, 8, 9, 10])
def test_align_workload_full(dv, wid):
    _say(f"align workload {W.WORKLOADS[wid].describe()}")
    trans, offsets, data, ns, al = _workload_table(dv, wid)
    ns_o, al_o = oracle.align(trans, offsets, data)
    np.testing.assert_array_equal(ns.cpu().numpy(), ns_o)
    np.testing.assert_array_equal(u32(al), al_o)


# ------------------------------------------------------------ greedy chains

def _chain_check(dv, wid, sample_rows):
    w = W.WORKLOADS[wid]
    trans, offsets, data, ns, al = _workload_table(dv, wid)
    init = W.init_states(wid)
    x = W.logits_all(wid, device=DEV)
    ws = dv.step_workspace(w.B, w.V, DEV)
    toks, sts = run_chain(dv, ns, al, _dev(init), x, ws)
    torch.cuda.synchronize()
    toks_h, sts_h = toks.cpu().numpy(), sts.cpu().numpy()
    rows = np.arange(w.B) if sample_rows is None else sample_rows
    cache = oracle.RowCache(trans, offsets, data)
    xr = to_oracle(x[:, torch.from_numpy(rows.astype(np.int64)).to(DEV)])
    del x
    dead = 0
    for i, b in enumerate(rows):
        t_o, s_o = oracle.masked_chain(cache, init[b], xr[:, i])
        np.testing.assert_array_equal(toks_h[:, b], t_o, err_msg=f"workload {wid} row {b}")
        np.testing.assert_array_equal(sts_h[1:, b], s_o[1:], err_msg=f"workload {wid} row {b}")
        dead += int(s_o[-1] == -1)
    _say(f"chain workload {wid}: {len(rows)} rows x {w.steps} steps bit-exact, {dead} rows died")
    # every emitted token is allowed from the state it was chosen in (all rows)
    st = sts[:-1].to(torch.int64)
    tk = toks.to(torch.int64)
    live = (st >= 0) & (tk >= 0)
    word = al[st.clamp(min=0), (tk.clamp(min=0) // 32)].to(torch.int64) & 0xFFFFFFFF
    assert bool((((word >> (tk.clamp(min=0) % 32)) & 1) == 1)[live].all())
    assert bool(((tk == -1) == (sts[1:] == -1)).all())


@pytest.mark.parametrize("wid", [1, 2, 3, 6, 7, 8, 9, 10])
def test_chain_workload_full(dv, wid):
    _say(f"chain workload {W.WORKLOADS[wid].describe()}")
    _chain_check(dv, wid, None)


# ---------------------------------------------------------- masked step edges

def _one_row_table(V, allowed):
    ns = np.full((1, V), -1, np.int32)
    ns[0, list(allowed)] = 0
    alive = ns != -1
    Wd = (V + 31) // 32
    pad = np.zeros((1, Wd * 32), bool)
    pad[:, :V] = alive
    al = np.packbits(pad, axis=1, bitorder="little").view("<u4").reshape(1, Wd)
    return ns, al


PLANTED_F32 = [
    ([100, 9, 9, 5, 1, 9, 0, 9, 0, 0.5], [1, 2, 5, 7, 9], 1),
    ([0, 1, -0.0, 7, 7, 0.0, 9], [2, 5], 2),
    ([0, 1, 0.0, 7, 7, -0.0, 9], [2, 5], 2),
    ([5, float("nan"), 3, 3, -np.inf], [1, 4], 1),
    ([float("nan"), 2.0, 1.0], [0, 1, 2], 1),
    ([float("nan")] * 6, [3, 5], 3),
    ([np.inf, 1e30, np.inf, 2, 3], [1, 3], 1),
    ([-np.inf, -np.inf, -3e38], [0, 1], 0),
    ([-1e-45, 0.0, 1e-45, -0.0], [0, 2, 3], 2),
    ([1, 2, 3], [], -1),
]


@pytest.mark.parametrize("spread", [1, 37, 20011])
@pytest.mark.parametrize("case", range(len(PLANTED_F32)))
def test_step_planted_specials_f32(dv, case, spread):
    """Planted values at indices i * spread, so large spreads cross vector,
    wave, block and chunk boundaries (multi-block rows)."""
    vals, allowed, expect = PLANTED_F32[case]
    V = len(vals) * spread + 5
    x = np.full((1, V), 1e38, np.float32)       # disallowed everywhere else
    x[0, np.arange(len(vals)) * spread] = np.array(vals, np.float32)
    ns, al = _one_row_table(V, [a * spread for a in allowed])
    tok, new = dv.masked_step(_dev(ns), _dev(al.view(np.int32)), _dev(np.zeros(1, np.int32)), _dev(x))
    tok_o, new_o = oracle.masked_step(ns, al, np.zeros(1, np.int32), x)
    assert int(tok.item()) == int(tok_o[0]) == (expect * spread if expect >= 0 else -1)
    assert int(new.item()) == int(new_o[0])


@pytest.mark.parametrize("bits,allowed,expect", [
    ([0x3F80, 0x3F80, 0x3F80], [1, 2], 1),
    ([0x8000, 0x0000, 0x0001], [0, 1], 0),
    ([0x8000, 0x0000, 0x0001], [0, 1, 2], 2),
    ([0x7FC1, 0xFF80, 0xFFC1], [0, 1, 2], 0),
    ([0x7FC1, 0xC000, 0x7F80], [0, 1], 1),
    ([0xFFC1, 0xFF7F], [0, 1], 1),
    ([0xBF80, 0xC000, 0xBF80], [0, 1, 2], 0),
])
@pytest.mark.parametrize("spread", [1, 9, 50021])
def test_step_planted_specials_bf16(dv, bits, allowed, expect, spread):
    V = len(bits) * spread + 3
    x = np.full((1, V), 0x7F00, np.uint16)
    x[0, np.arange(len(bits)) * spread] = np.array(bits, np.uint16)
    ns, al = _one_row_table(V, [a * spread for a in allowed])
    xt = _dev(x.view(np.int16)).view(torch.bfloat16)
    tok, _ = dv.masked_step(_dev(ns), _dev(al.view(np.int32)), _dev(np.zeros(1, np.int32)), xt)
    tok_o, _ = oracle.masked_step(ns, al, np.zeros(1, np.int32), x)
    assert int(tok.item()) == int(tok_o[0]) == expect * spread


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,V,extra_ld,offset", [
    (1, 1, 0, 0), (3, 7, 0, 0), (5, 33, 3, 0), (4, 1000, 0, 1), (17, 4099, 5, 1),
    (2, 70001, 0, 0), (9, 70001, 11, 3), (300, 2048, 0, 0), (3000, 129, 0, 0),
])
def test_step_shapes_ld_and_alignment(dv, dtype, B, V, extra_ld, offset):
    """Random tables and states (including dead and out-of-range states),
    row strides wider than V and row starts that are not 16-byte aligned."""
    _say(f"step shapes B={B} V={V} ld=V+{extra_ld} offset={offset} {dtype}")
    rng = np.random.default_rng(B * 7 + V)
    S = 13
    alive = rng.random((S, V)) < rng.choice([0.0, 0.002, 0.05, 0.5, 1.0], size=(S, 1))
    ns = np.where(alive, rng.integers(0, S, (S, V)), -1).astype(np.int32)
    Wd = (V + 31) // 32
    pad = np.zeros((S, Wd * 32), bool)
    pad[:, :V] = alive
    al = np.packbits(pad, axis=1, bitorder="little").view("<u4").reshape(S, Wd)
    states = rng.integers(-2, S + 2, B).astype(np.int32)
    ld = V + extra_ld
    buf = torch.from_numpy((rng.standard_normal(B * ld + offset + 8) * 4).astype(np.float32))
    buf = buf.to(dtype)
    special = torch.tensor([float("nan"), float("inf"), -float("inf"), -0.0, 0.0], dtype=dtype)
    pos = torch.from_numpy(rng.integers(0, buf.numel(), 64))
    buf[pos] = special[torch.from_numpy(rng.integers(0, 5, 64))]
    buf_d = buf.to(DEV)
    x = buf_d[offset:offset + B * ld].view(B, ld)[:, :V]
    tok, new = dv.masked_step(_dev(ns), _dev(al.view(np.int32)), _dev(states), x)
    xo = to_oracle(buf[offset:offset + B * ld].view(B, ld))
    tok_o, new_o = oracle.masked_step(ns, al, states, xo)
    np.testing.assert_array_equal(tok.cpu().numpy(), tok_o)
    np.testing.assert_array_equal(new.cpu().numpy(), new_o)


@pytest.mark.parametrize("B,V,extra_ld", [
    (1, 5, 0), (2, 13, 1), (3, 4100, 3), (2, 70001, 0), (1, 70001, 5), (260, 1030, 1), (64, 50257, 0),
])
@pytest.mark.parametrize("dtype,head", [(torch.bfloat16, h) for h in range(8)] +
                         [(torch.float32, h) for h in range(4)])
def test_step_every_row_alignment(dv, B, V, extra_ld, dtype, head):
    """Rows starting at every element offset within 16 bytes: the first
    row's head (elements before its first 16-byte boundary) is `head`, later
    rows vary with the row stride.  Few distinct values (many ties across
    the head, vector and tail regions), planted NaN and signed zeros, random
    masks of every density; greedy and opportunistic steps both checked."""
    _say(f"step alignment {dtype} B={B} V={V} ld=V+{extra_ld} head={head}")
    rng = np.random.default_rng(1000 * head + V + B)
    S = 7
    alive = rng.random((S, V)) < rng.choice([0.002, 0.05, 0.5, 0.97, 1.0], size=(S, 1))
    ns = np.where(alive, rng.integers(0, S, (S, V)), -1).astype(np.int32)
    Wd = (V + 31) // 32
    pad = np.zeros((S, Wd * 32), bool)
    pad[:, :V] = alive
    al = np.packbits(pad, axis=1, bitorder="little").view("<u4").reshape(S, Wd)
    states = rng.integers(-1, S, B).astype(np.int32)
    ld = V + extra_ld
    esz = 2 if dtype == torch.bfloat16 else 4
    per = 16 // esz                  # elements per 16-byte vector
    offset = (per - head) % per      # elements from a 16-byte boundary
    vals = rng.integers(-2, 3, B * ld + offset + 8).astype(np.float32)
    buf = torch.from_numpy(vals).to(dtype)
    special = torch.tensor([float("nan"), -0.0, 0.0, 2.0], dtype=dtype)
    pos = torch.from_numpy(rng.integers(0, buf.numel(), 40))
    buf[pos] = special[torch.from_numpy(rng.integers(0, 4, 40))]
    base = torch.empty(buf.numel() + 64, dtype=dtype, device=DEV)
    shift = (-(base.data_ptr() // esz)) % per    # first 16-byte boundary of base
    buf_d = base[shift:shift + buf.numel()]
    buf_d.copy_(buf.to(DEV))
    x = buf_d[offset:offset + B * ld].view(B, ld)[:, :V]
    assert (x.data_ptr() // esz + head) % per == 0
    xo = to_oracle(buf[offset:offset + B * ld].view(B, ld))
    tok_o, new_o = oracle.masked_step(ns, al, states, xo)
    for opp in (False, True):
        tok, new = dv.masked_step(_dev(ns), _dev(al.view(np.int32)), _dev(states), x, opportunistic=opp)
        np.testing.assert_array_equal(tok.cpu().numpy(), tok_o)
        np.testing.assert_array_equal(new.cpu().numpy(), new_o)


@pytest.mark.parametrize("B,V,offset,extra_ld", [
    (600, 40000, 0, 0), (520, 30011, 0, 1), (530, 33333, 3, 2), (1030, 24577, 0, 7),
    # two to four blocks per compute unit, long rows: mask bytes two batches ahead
    (600, 140000, 0, 0), (530, 133333, 3, 2), (1024, 70000, 0, 0),
    # fewer than two blocks per compute unit, long chunks: every line is read
    (256, 128256, 0, 0), (300, 66000, 3, 1), (128, 140000, 0, 0), (64, 260000, 5, 3),
])
def test_step_skips_lines_without_allowed_tokens(dv, B, V, offset, extra_ld):
    """Vectors whose 8 tokens are all disallowed are not read (from the
    third batch of a chunk on) by launches of two or more blocks per compute
    unit (mask bytes staged in LDS) and by chunks of at least 8 batches at up
    to four blocks per unit (mask bytes two batches ahead); shorter chunks at
    one block per unit read every line, the same masks deciding.  Sparse masks
    (whole runs of disallowed vectors), few distinct values, planted NaN and
    signed zeros, aligned and misaligned rows, rows of one, two and four
    chunks; greedy and opportunistic steps against the oracle."""
    _say(f"step line skipping B={B} V={V} offset={offset} ld=V+{extra_ld}")
    rng = np.random.default_rng(B + V)
    S = 9
    dens = np.array([0.0005, 0.003, 0.02, 0.1, 0.5, 0.9, 1.0, 0.01, 0.05])[:, None]
    alive = rng.random((S, V)) < dens
    alive[7, : V // 2] = False                    # long empty runs, then dense
    alive[7, V // 2:] = True
    alive[8] = False
    alive[8, ::4099] = True                       # isolated allowed tokens
    ns = np.where(alive, rng.integers(0, S, (S, V)), -1).astype(np.int32)
    Wd = (V + 31) // 32
    pad = np.zeros((S, Wd * 32), bool)
    pad[:, :V] = alive
    al = np.packbits(pad, axis=1, bitorder="little").view("<u4").reshape(S, Wd)
    states = rng.integers(-1, S, B).astype(np.int32)
    ld = V + extra_ld
    vals = rng.integers(-3, 4, B * ld + offset + 8).astype(np.float32)
    buf = torch.from_numpy(vals).to(torch.bfloat16)
    special = torch.tensor([float("nan"), -0.0, 0.0, 3.0], dtype=torch.bfloat16)
    pos = torch.from_numpy(rng.integers(0, buf.numel(), 4000))
    buf[pos] = special[torch.from_numpy(rng.integers(0, 4, 4000))]
    buf_d = buf.to(DEV)
    x = buf_d[offset:offset + B * ld].view(B, ld)[:, :V]
    xo = to_oracle(buf[offset:offset + B * ld].view(B, ld))
    tok_o, new_o = oracle.masked_step(ns, al, states, xo)
    for opp in (False, True):
        tok, new = dv.masked_step(_dev(ns), _dev(al.view(np.int32)), _dev(states), x, opportunistic=opp)
        np.testing.assert_array_equal(tok.cpu().numpy(), tok_o)
        np.testing.assert_array_equal(new.cpu().numpy(), new_o)


def test_calls_on_two_streams_do_not_interfere(dv):
    """Two streams, each with its own workspaces, interleave greedy steps on
    rows split over many blocks (which meet in the workspace), sampled steps
    and an alignment, never waiting for each other: every result equals the
    oracle's (the library keeps no device state between calls)."""
    _say("two streams, interleaved calls")
    rng = np.random.default_rng(2024)
    S, V, B, steps = 13, 100_000, 3, 6
    alive = rng.random((S, V)) < rng.choice([0.001, 0.05, 0.6], size=(S, 1))
    ns = np.where(alive, rng.integers(0, S, (S, V)), -1).astype(np.int32)
    Wd = (V + 31) // 32
    pad = np.zeros((S, Wd * 32), bool)
    pad[:, :V] = alive
    al = np.packbits(pad, axis=1, bitorder="little").view("<u4").reshape(S, Wd)
    ns_d, al_d = _dev(ns), _dev(al.view(np.int32))
    trans, offsets, data = _random_case(31, 700, 5000, 10, 0.01, alphabet=np.arange(0x20, 0x7F))
    runs = []
    for _ in range(2):
        x = torch.from_numpy((rng.standard_normal((steps, B, V)) * 3).astype(np.float32)).to(torch.bfloat16)
        st = rng.integers(-1, S, (steps, B)).astype(np.int32)
        runs.append(dict(x=x, x_d=x.to(DEV), st=st, st_d=_dev(st),
                         tok=torch.empty((steps, B), dtype=torch.int32, device=DEV),
                         new=torch.empty((steps, B), dtype=torch.int32, device=DEV),
                         stok=torch.empty((steps, B), dtype=torch.int32, device=DEV),
                         snew=torch.empty((steps, B), dtype=torch.int32, device=DEV),
                         ws=dv.step_workspace(B, V, DEV), sws=dv.sample_workspace(B, V, DEV),
                         stream=torch.cuda.Stream(DEV)))
    tr_d, of_d, da_d = _dev(trans), _dev(offsets), _dev(data)
    nsa = torch.empty((700, 5000), dtype=torch.int32, device=DEV)
    ala = torch.empty((700, (5000 + 31) // 32), dtype=torch.int32, device=DEV)
    wsa = torch.empty(dv.align_workspace_bytes(700, 5000), dtype=torch.uint8, device=DEV)
    torch.cuda.synchronize()
    for k in range(steps):
        for i, r in enumerate(runs):
            with torch.cuda.stream(r["stream"]):
                dv.masked_step(ns_d, al_d, r["st_d"][k], r["x_d"][k], token=r["tok"][k], new_state=r["new"][k],
                               workspace=r["ws"])
                dv.masked_sample(ns_d, al_d, r["st_d"][k], r["x_d"][k], seed=7 + i, offset=k,
                                 token=r["stok"][k], new_state=r["snew"][k], workspace=r["sws"])
                if i == 1 and k == 2:
                    dv.align(tr_d, of_d, da_d, next_state=nsa, allow=ala, workspace=wsa)
    torch.cuda.synchronize()
    for i, r in enumerate(runs):
        for k in range(steps):
            xo = to_oracle(r["x"][k])
            tok_o, new_o = oracle.masked_step(ns, al, r["st"][k], xo)
            np.testing.assert_array_equal(r["tok"][k].cpu().numpy(), tok_o)
            np.testing.assert_array_equal(r["new"][k].cpu().numpy(), new_o)
            stok_o, snew_o = oracle.masked_sample(ns, al, r["st"][k], xo, 1.0, 7 + i, k)
            np.testing.assert_array_equal(r["stok"][k].cpu().numpy(), stok_o)
            np.testing.assert_array_equal(r["snew"][k].cpu().numpy(), snew_o)
    ns_o, al_o = oracle.align(trans, offsets, data)
    np.testing.assert_array_equal(nsa.cpu().numpy(), ns_o)
    np.testing.assert_array_equal(u32(ala), al_o)


def test_step_empty_batch(dv):
    ns = torch.zeros((2, 10), dtype=torch.int32, device=DEV)
    al = torch.full((2, 1), 0x3FF, dtype=torch.int32, device=DEV)
    tok, new = dv.masked_step(ns, al, torch.zeros(0, dtype=torch.int32, device=DEV),
                              torch.zeros((0, 10), device=DEV))
    assert tok.numel() == 0 and new.numel() == 0


def test_step_workspace_reuse_and_determinism(dv):
    trans, offsets, data, ns, al = _workload_table(dv, 2)
    w = W.WORKLOADS[2]
    ws = dv.step_workspace(64, w.V, DEV)
    rng = np.random.default_rng(0)
    outs = []
    for B in (64, 8, 64, 1, 33):
        st = _dev(rng.integers(0, w.S, B).astype(np.int32))
        x = W.logits(2, 7, device=DEV, batch=B)
        a = dv.masked_step(ns, al, st, x, workspace=ws)
        b = dv.masked_step(ns, al, st, x, workspace=ws)
        assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
        fresh = dv.masked_step(ns, al, st, x)  # its own zeroed workspace
        assert torch.equal(a[0], fresh[0]) and torch.equal(a[1], fresh[1])
        outs.append(a)
    torch.cuda.synchronize()


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_split_rows_leave_the_workspace_zero(dv, dtype):
    """Rows split over several blocks meet in the workspace; the block that
    arrives last puts the row's entries back to zero.  After split-row calls
    of every kind (greedy, sampled, speculative, all sizes) the shared
    workspace is all zero again, and each call matches the oracle."""
    rng = np.random.default_rng(5)
    S, Vmax = 6, 70001
    ws = torch.zeros(max(dv.spec_verify_workspace_bytes(64, 4, Vmax), dv.masked_step_workspace_bytes(64, Vmax),
                         dv.masked_sample_workspace_bytes(64, Vmax)), dtype=torch.uint8, device=DEV)
    for B, V in ((1, 70001), (7, 40000), (64, 4099), (3, 70001)):
        _say(f"split rows B={B} V={V} {dtype}")
        alive = rng.random((S, V)) < np.array([0.001, 0.02, 0.3, 1.0, 0.5, 0.0])[:, None]
        ns = np.where(alive, rng.integers(0, S, (S, V)), -1).astype(np.int32)
        Wd = (V + 31) // 32
        pad = np.zeros((S, Wd * 32), bool)
        pad[:, :V] = alive
        al = np.packbits(pad, axis=1, bitorder="little").view("<u4").reshape(S, Wd)
        states = rng.integers(-1, S, B).astype(np.int32)
        x = torch.from_numpy(rng.integers(-4, 5, (B, V)).astype(np.float32)).to(dtype).to(DEV)
        xo = to_oracle(x)
        nsd, ald = _dev(ns), _dev(al.view(np.int32))
        tok, new = dv.masked_step(nsd, ald, _dev(states), x, workspace=ws)
        t_o, n_o = oracle.masked_step(ns, al, states, xo)
        np.testing.assert_array_equal(tok.cpu().numpy(), t_o)
        np.testing.assert_array_equal(new.cpu().numpy(), n_o)
        assert int(ws.count_nonzero()) == 0
        tok, new = dv.masked_sample(nsd, ald, _dev(states), x, 11, B, workspace=ws)
        t_o, n_o = oracle.masked_sample(ns, al, states, xo, 1.0, 11, B)
        np.testing.assert_array_equal(tok.cpu().numpy(), t_o)
        np.testing.assert_array_equal(new.cpu().numpy(), n_o)
        assert int(ws.count_nonzero()) == 0
        props = rng.integers(0, V, (B, 4)).astype(np.int32)
        lg = torch.from_numpy(rng.integers(-4, 5, (B, 5, V)).astype(np.float32)).to(dtype).to(DEV)
        t, a, n = dv.spec_verify(nsd, ald, _dev(states), _dev(props), lg, workspace=ws)
        t_o, a_o, n_o = oracle.spec_verify(ns, al, states, props, to_oracle(lg))
        np.testing.assert_array_equal(t.cpu().numpy(), t_o)
        np.testing.assert_array_equal(a.cpu().numpy(), a_o)
        np.testing.assert_array_equal(n.cpu().numpy(), n_o)
        assert int(ws.count_nonzero()) == 0


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_step_and_sample_at_the_largest_vocabulary(dv, dtype):
    """V = 2^24 (the largest vocabulary the library accepts): rows split into
    more chunks than at any workload (the chunk size cap for the staged mask
    bytes applies), so many blocks meet on one row.  Greedy and sampled
    steps against the oracle; one planted maximum near the end of the row."""
    V, B, S = 1 << 24, 2, 2
    _say(f"largest vocabulary V={V} B={B} {dtype}")
    rng = np.random.default_rng(24)
    Wd = V // 32
    al = np.zeros((S, Wd), np.uint32)
    al[0] = rng.integers(0, 1 << 32, Wd, dtype=np.uint64).astype(np.uint32) & 0x01010101   # sparse
    al[1] = 0xFFFFFFFF
    alive = np.unpackbits(al.view(np.uint8), axis=1, bitorder="little").astype(bool)
    ns = np.where(alive, (np.arange(V) % S)[None, :], -1).astype(np.int32)
    del alive
    states = np.array([0, 1], np.int32)
    x = torch.from_numpy(rng.integers(-8, 9, (B, V)).astype(np.float32))
    x[0, V - 9] = 100.0   # allowed in state 0 or not: the oracle decides
    x[1, V - 3] = 100.0   # state 1 allows every token: this one wins
    x = x.to(dtype)
    xd = x.to(DEV)
    xo = to_oracle(x)
    nsd, ald = _dev(ns), _dev(al.view(np.int32))
    tok, new = dv.masked_step(nsd, ald, _dev(states), xd)
    t_o, n_o = oracle.masked_step(ns, al, states, xo)
    np.testing.assert_array_equal(tok.cpu().numpy(), t_o)
    np.testing.assert_array_equal(new.cpu().numpy(), n_o)
    assert int(t_o[1]) == V - 3
    tok, new = dv.masked_sample(nsd, ald, _dev(states), xd, 3, 9)
    t_o, n_o = oracle.masked_sample(ns, al, states, xo, 1.0, 3, 9)
    np.testing.assert_array_equal(tok.cpu().numpy(), t_o)
    np.testing.assert_array_equal(new.cpu().numpy(), n_o)


def test_step_rejects_in_place_update(dv):
    ns = torch.zeros((2, 10), dtype=torch.int32, device=DEV)
    al = torch.zeros((2, 1), dtype=torch.int32, device=DEV)
    st = torch.zeros(4, dtype=torch.int32, device=DEV)
    with pytest.raises(dv.DvError) as e:
        dv.masked_step(ns, al, st, torch.zeros((4, 10), device=DEV), new_state=st)
    assert e.value.status == 4


@pytest.mark.parametrize("capture", ["torch", "hip"])
@pytest.mark.parametrize("wid", [2, 3, 4])
def test_step_graph_replay_matches_eager(dv, wid, capture):
    """The decode loop captured as a HIP graph gives the eager results on
    every replay, with eager work in between: captured by torch.cuda.graph,
    and by the HIP API's own stream capture as the benchmark captures it."""
    w = W.WORKLOADS[wid]
    trans, offsets, data, ns, al = _workload_table(dv, wid)
    steps = 16
    x = W.logits_all(wid, device=DEV, steps=steps)
    ws = dv.step_workspace(w.B, w.V, DEV)
    init = _dev(W.init_states(wid))
    st = torch.empty((steps + 1, w.B), dtype=torch.int32, device=DEV)
    tk = torch.empty((steps, w.B), dtype=torch.int32, device=DEV)

    def launches():
        for k in range(steps):
            dv.masked_step(ns, al, st[k], x[k], token=tk[k], new_state=st[k + 1], workspace=ws)

    st[0].copy_(init)
    launches()
    torch.cuda.synchronize()
    ref_t, ref_s = tk.clone(), st.clone()
    side = torch.cuda.Stream(DEV)
    side.wait_stream(torch.cuda.current_stream(DEV))
    with torch.cuda.stream(side):
        launches()
    torch.cuda.current_stream(DEV).wait_stream(side)
    torch.cuda.synchronize()
    if capture == "torch":
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            launches()
    else:
        import bench
        g = bench.HipGraph(launches, DEV)
    for rep in range(3):
        tk.fill_(-7)
        st[1:].fill_(-7)
        _ = (x[0].float().sum() + rep).item()  # eager work and a sync between replays
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(tk, ref_t) and torch.equal(st, ref_s), f"replay {rep}"
    if capture == "hip":
        g.close()


# ------------------------------------------------------- end-of-sequence column

def test_align_eos_paper_example(dv):
    g = json.load(open(os.path.join(GOLDEN, "fig_nfa_int.json")))
    e = g["eos"]
    trans = W.dfa_from_spec(len(g["states"]), g["moves"])
    offsets, data = W.vocab_from_tokens([t.encode() for t in g["vocab"]] + [b"</s>"])
    acc = np.array(e["accepting"], np.uint8)
    ns, al = dv.align(_dev(trans), _dev(offsets), _dev(data), accepting=_dev(acc), eos_token=e["eos_token"])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(ns.cpu().numpy()[:, e["eos_token"]], e["expected_eos_column"])
    np.testing.assert_array_equal(u32(al)[:, 0], np.array([int(x, 16) for x in e["expected_allow"]], np.uint32))


@pytest.mark.parametrize("wid", [1, 2, 3, 7, 8, 10])
@pytest.mark.parametrize("where", ["first", "middle", "last"])
def test_align_eos_workloads(dv, wid, where):
    w = W.WORKLOADS[wid]
    trans, acc = W.dfa(wid)
    offsets, data = W.vocab(wid)
    eos = {"first": 0, "middle": w.V // 2 + 3, "last": w.V - 1}[where]
    ns, al = dv.align(_dev(trans), _dev(offsets), _dev(data), accepting=_dev(acc), eos_token=eos)
    torch.cuda.synchronize()
    rows = np.arange(w.S, dtype=np.int32) if w.S <= 256 else np.unique(
        np.concatenate([[0, w.S - 1], np.random.default_rng(wid).integers(0, w.S, 40)])).astype(np.int32)
    ns_o, al_o = oracle.align_eos(trans, offsets, data, acc, eos, rows=rows)
    idx = torch.from_numpy(rows.astype(np.int64)).to(DEV)
    np.testing.assert_array_equal(ns.index_select(0, idx).cpu().numpy(), ns_o)
    np.testing.assert_array_equal(u32(al.index_select(0, idx)), al_o)


def test_align_eos_without_accepting_flags(dv):
    trans, _ = W.dfa(1)
    offsets, data = W.vocab(1)
    ns, al = dv.align(_dev(trans), _dev(offsets), _dev(data), eos_token=7)
    torch.cuda.synchronize()
    ns_o, al_o = oracle.align_eos(trans, offsets, data, None, 7)
    np.testing.assert_array_equal(ns.cpu().numpy(), ns_o)
    np.testing.assert_array_equal(u32(al), al_o)


def test_chain_stops_on_eos(dv):
    """A greedy chain whose logits favour EOS stops (picks EOS) exactly in
    accepting states, as the oracle's chain does."""
    w = W.WORKLOADS[2]
    trans, acc = W.dfa(2)
    offsets, data = W.vocab(2)
    eos = w.V - 1
    ns, al = dv.align(_dev(trans), _dev(offsets), _dev(data), accepting=_dev(acc), eos_token=eos)
    ns_o, al_o = oracle.align_eos(trans, offsets, data, acc, eos)
    steps = 32
    x = W.logits_all(2, device=DEV, steps=steps)
    x[:, :, eos] = 50.0  # the model always wants to stop: EOS wins wherever it is allowed
    ws = dv.step_workspace(w.B, w.V, DEV)
    init = W.init_states(2)
    toks, sts = run_chain(dv, ns, al, _dev(init), x, ws)
    xs = to_oracle(x)
    cur = init
    for k in range(steps):
        t_o, n_o = oracle.masked_step(ns_o, al_o, cur, xs[k])
        np.testing.assert_array_equal(toks[k].cpu().numpy(), t_o)
        np.testing.assert_array_equal(sts[k + 1].cpu().numpy(), n_o)
        # EOS is chosen exactly where the constraint may end
        live = cur >= 0
        np.testing.assert_array_equal(t_o[live] == eos, acc[cur[live]].astype(bool))
        cur = n_o
    assert (toks == eos).any()


# ------------------------------------------- speculative chain check (Sec. 3.6)

def _perturb(rng, greedy, V, keep):
    """Proposals that follow ``greedy`` with probability ``keep`` per position,
    else a random id (possibly outside [0, V))."""
    other = rng.integers(-2, V + 2, greedy.shape).astype(np.int32)
    return np.where(rng.random(greedy.shape) < keep, greedy, other).astype(np.int32)


def _greedy_proposals(ns_o, al_o, states, xs_pos, s):
    """The oracle's greedy chain over the first s positions: [B][s]."""
    out = np.empty((states.shape[0], s), np.int32)
    cur = states
    for j in range(s):
        t, cur = oracle.masked_step(ns_o, al_o, cur, xs_pos[:, j])
        out[:, j] = t
    return out


def _check_spec(dv, ns, al, ns_o, al_o, states, props, x_dev, label):
    tok, acc, nst = dv.spec_verify(ns, al, _dev(states), _dev(props), x_dev)
    a_w, f_w = dv.spec_walk(ns, al, _dev(states), _dev(props))
    torch.cuda.synchronize()
    xs = to_oracle(x_dev)
    tok_o, acc_o, nst_o = oracle.spec_verify(ns_o, al_o, states, props, xs)
    np.testing.assert_array_equal(tok.cpu().numpy(), tok_o, err_msg=label)
    np.testing.assert_array_equal(acc.cpu().numpy(), acc_o, err_msg=label)
    np.testing.assert_array_equal(nst.cpu().numpy(), nst_o, err_msg=label)
    a_o, f_o = oracle.spec_walk(ns_o, al_o, states, props)
    np.testing.assert_array_equal(a_w.cpu().numpy(), a_o, err_msg=label)
    np.testing.assert_array_equal(f_w.cpu().numpy(), f_o, err_msg=label)
    return acc_o


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_spec_paper_example(dv, dtype):
    g = json.load(open(os.path.join(GOLDEN, "fig_nfa_int.json")))
    e, sp = g["eos"], g["spec"]
    trans = W.dfa_from_spec(len(g["states"]), g["moves"])
    offsets, data = W.vocab_from_tokens([t.encode() for t in g["vocab"]] + [b"</s>"])
    acc = np.array(e["accepting"], np.uint8)
    ns, al = dv.align(_dev(trans), _dev(offsets), _dev(data), accepting=_dev(acc), eos_token=e["eos_token"])
    lg = np.array([[[float(v) for v in r] for r in rows] for rows in sp["logits"]], np.float32)
    x = _dev(lg).to(dtype)
    states, props = np.array(sp["states"], np.int32), np.array(sp["proposals"], np.int32)
    tok, a, nst = dv.spec_verify(ns, al, _dev(states), _dev(props), x)
    a_w, f_w = dv.spec_walk(ns, al, _dev(states), _dev(props))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(tok.cpu().numpy(), sp["expected_token"])
    np.testing.assert_array_equal(a.cpu().numpy(), sp["expected_accepted"])
    np.testing.assert_array_equal(nst.cpu().numpy(), sp["expected_new_state"])
    np.testing.assert_array_equal(a_w.cpu().numpy(), sp["expected_walk_accepted"])
    np.testing.assert_array_equal(f_w.cpu().numpy(), sp["expected_walk_final_state"])


@pytest.mark.parametrize("wid,s", [(1, 4), (2, 4), (2, 8), (3, 6), (6, 8), (7, 8), (8, 8), (9, 8), (10, 8)])
@pytest.mark.parametrize("layout", ["rows", "steps"])
def test_spec_workload_full(dv, wid, s, layout):
    """Every row and position against the oracle.  ``rows``: the model's
    [B][s+1][V] output; ``steps``: positions stored as [s+1][B][V] and passed
    through strides."""
    w = W.WORKLOADS[wid]
    _say(f"spec verify workload {w.describe()} s={s} layout={layout}")
    trans, offsets, data, ns, al = _workload_table(dv, wid)
    ns_o, al_o = oracle.align(trans, offsets, data)
    x = W.logits_all(wid, device=DEV, steps=s + 1)           # [s+1][B][V]
    x_rows = x.transpose(0, 1)                                # [B][s+1][V] view
    if layout == "rows":
        x_rows = x_rows.contiguous()
    states = W.init_states(wid)
    states[::7] = -1
    rng = np.random.default_rng(200 + wid * 10 + s)
    greedy = _greedy_proposals(ns_o, al_o, states, to_oracle(x_rows), s)
    props = _perturb(rng, greedy, w.V, 0.85)
    acc = _check_spec(dv, ns, al, ns_o, al_o, states, props, x_rows, f"workload {wid} s={s} {layout}")
    _say(f"  accepted histogram {np.bincount(acc, minlength=s + 1).tolist()}")


def test_spec_zero_proposals_is_a_step(dv):
    w = W.WORKLOADS[3]
    trans, offsets, data, ns, al = _workload_table(dv, 3)
    x = W.logits(3, 0, device=DEV)                            # [B][V]
    states = _dev(W.init_states(3))
    tok, acc, nst = dv.spec_verify(ns, al, states, torch.empty((w.B, 0), dtype=torch.int32, device=DEV),
                                   x[:, None, :])
    t, n = dv.masked_step(ns, al, states, x)
    a_w, f_w = dv.spec_walk(ns, al, states, torch.empty((w.B, 0), dtype=torch.int32, device=DEV))
    torch.cuda.synchronize()
    assert torch.equal(tok[:, 0], t) and torch.equal(nst, n)
    assert int(acc.abs().sum()) == 0 and int(a_w.abs().sum()) == 0
    assert torch.equal(f_w, torch.where((states >= 0) & (states < w.S), states, torch.full_like(states, -1)))


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,s,V,pad_prop,misalign", [
    (1, 1, 1, 0, 0),            # a one-token vocabulary
    (1, 64, 1000, 3, 0),        # one long row of proposals: positions split over chunks
    (3, 5, 33, 0, 1),           # a ragged word; rows not 16-byte aligned (scalar path)
    (40, 7, 4099, 2, 0),        # 320 positions: one block per position
    (300, 2, 20000, 0, 1),      # many rows, odd position stride
])
def test_spec_shapes_strides_and_edges(dv, dtype, B, s, V, pad_prop, misalign):
    rng = np.random.default_rng(B * 1000 + s * 10 + V)
    S = 12
    trans = rng.integers(-1, S + 1, (S, 256)).astype(np.int32)       # includes out-of-range targets
    trans[:, rng.random(256) < 0.5] = -1
    lens = rng.integers(1, 4, V)
    offsets = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    data = rng.integers(0, 256, int(offsets[-1])).astype(np.uint8)
    ns, al = _align(dv, trans, offsets, data)
    ns_o, al_o = oracle.align(trans, offsets, data)
    states = rng.integers(-2, S + 2, B).astype(np.int32)
    ld_pos = V + misalign
    buf = torch.randn(B * (s + 1) * ld_pos + 8, device=DEV).to(dtype)
    x = buf.as_strided((B, s + 1, V), ((s + 1) * ld_pos, ld_pos, 1), misalign)
    greedy = _greedy_proposals(ns_o, al_o, states, to_oracle(x), s)
    props_full = np.zeros((B, s + pad_prop), np.int32)
    props_full[:, :s] = _perturb(rng, greedy, V, 0.8)
    props_full[:, :s][rng.random((B, s)) < 0.05] = np.int32(2 ** 31 - 1)
    props_full[:, :s][rng.random((B, s)) < 0.05] = np.int32(-2 ** 31)
    props_dev = _dev(props_full)[:, :s]                      # row stride s + pad_prop
    tok, acc, nst = dv.spec_verify(ns, al, _dev(states), props_dev, x)
    a_w, f_w = dv.spec_walk(ns, al, _dev(states), props_dev)
    torch.cuda.synchronize()
    props = props_full[:, :s]
    tok_o, acc_o, nst_o = oracle.spec_verify(ns_o, al_o, states, props, to_oracle(x))
    a_o, f_o = oracle.spec_walk(ns_o, al_o, states, props)
    np.testing.assert_array_equal(tok.cpu().numpy(), tok_o)
    np.testing.assert_array_equal(acc.cpu().numpy(), acc_o)
    np.testing.assert_array_equal(nst.cpu().numpy(), nst_o)
    np.testing.assert_array_equal(a_w.cpu().numpy(), a_o)
    np.testing.assert_array_equal(f_w.cpu().numpy(), f_o)


def test_spec_empty_batch_and_aliasing(dv):
    trans, offsets, data, ns, al = _workload_table(dv, 1)
    e = torch.empty((0,), dtype=torch.int32, device=DEV)
    tok, acc, nst = dv.spec_verify(ns, al, e, torch.empty((0, 3), dtype=torch.int32, device=DEV),
                                   torch.empty((0, 4, ns.shape[1]), device=DEV))
    assert tok.shape == (0, 4) and acc.numel() == 0
    states = _dev(np.zeros(2, np.int32))
    props = _dev(np.zeros((2, 3), np.int32))
    x = torch.randn((2, 4, ns.shape[1]), device=DEV)
    with pytest.raises(dv.DvError):
        dv.spec_verify(ns, al, states, props, x, new_state=states)
    with pytest.raises(dv.DvError):
        dv.spec_walk(ns, al, states, props, accepted=props[0][:2])   # an output inside the proposals
    with pytest.raises(ValueError):
        dv.spec_walk(ns, al, states, props, accepted=props[0])       # the wrong size: refused by the binding


# ------------------------------------- opportunistic masking (Sec. 3.5, optimizations)

OPP_BF16 = [  # (bits, allowed, expect): the free maximum allowed, not allowed, special keys on top
    ([0x3F80, 0x4000, 0x3F80], [0, 1, 2], 1),
    ([0x3F80, 0x4000, 0x3F80], [0, 2], 0),
    ([0x7FC1, 0xC000, 0x7F80], [0, 1], 1),       # NaN first, +inf not allowed
    ([0x7FC1, 0xC000, 0x7F80], [0, 1, 2], 2),
    ([0x8000, 0x0000, 0xFFC1], [0, 1, 2], 0),    # -0.0 ties +0.0: lowest index
    ([0xFFC1, 0xFF80, 0xFF7F], [0, 1], 0),       # -NaN and -inf tie at -inf
    ([0x4000, 0x4000, 0x4000], [1, 2], 1),       # a tie whose lowest index is not allowed
]


@pytest.mark.parametrize("case", range(len(OPP_BF16)))
@pytest.mark.parametrize("spread", [1, 9, 50021])
def test_opportunistic_planted_specials_bf16(dv, case, spread):
    """256 rows (one block per row, so the check-first kernel runs), the same
    planted values in each, at indices that cross vector, wave and batch
    boundaries; every other logit is -1.0 and not allowed."""
    bits, allowed, expect = OPP_BF16[case]
    V = len(bits) * spread + 3
    B = 256
    x = np.full((B, V), 0xBF80, np.uint16)
    x[:, np.arange(len(bits)) * spread] = np.array(bits, np.uint16)
    ns, al = _one_row_table(V, [a * spread for a in allowed])
    xt = _dev(x.view(np.int16)).view(torch.bfloat16)
    zeros = _dev(np.zeros(B, np.int32))
    tok, new = dv.masked_step(_dev(ns), _dev(al.view(np.int32)), zeros, xt, opportunistic=True)
    tok_o, new_o, _ = oracle.masked_step_opportunistic(ns, al, np.zeros(B, np.int32), x)
    np.testing.assert_array_equal(tok.cpu().numpy(), tok_o)
    np.testing.assert_array_equal(new.cpu().numpy(), new_o)
    assert int(tok_o[0]) == expect * spread


@pytest.mark.parametrize("allowed_last", [True, False])
def test_opportunistic_tail_maximum(dv, allowed_last):
    """The overall maximum in the scalar tail (V not a multiple of 8)."""
    B, V = 300, 1003
    rng = np.random.default_rng(7)
    x = rng.standard_normal((B, V)).astype(np.float32)
    x[:, V - 1] = 9.0
    allowed = [3, 500, 1000] + ([V - 1] if allowed_last else [])
    ns, al = _one_row_table(V, allowed)
    xt = _dev(x).to(torch.bfloat16)
    zeros = _dev(np.zeros(B, np.int32))
    tok, _ = dv.masked_step(_dev(ns), _dev(al.view(np.int32)), zeros, xt, opportunistic=True)
    tok_o, _, ok = oracle.masked_step_opportunistic(ns, al, np.zeros(B, np.int32), to_oracle(xt))
    np.testing.assert_array_equal(tok.cpu().numpy(), tok_o)
    assert bool(ok.all()) == allowed_last


@pytest.mark.parametrize("wid", [3])
@pytest.mark.parametrize("adherent", [0.0, 0.9])
def test_opportunistic_workload(dv, wid, adherent):
    """The benchmark's shapes: sampled rows against the oracle, every row
    against dv_masked_step.  ``adherent``: the fraction of rows whose logits
    favour an allowed token (chosen from the oracle's table row)."""
    w = W.WORKLOADS[wid]
    _say(f"opportunistic step workload {w.describe()} adherent={adherent}")
    trans, offsets, data, ns, al = _workload_table(dv, wid)
    cache = oracle.RowCache(trans, offsets, data)
    init = W.init_states(wid)
    x = W.logits(wid, 0, device=DEV)
    rng = np.random.default_rng(400 + wid)
    if adherent:
        pick = np.nonzero(rng.random(w.B) < adherent)[0]
        cols = []
        for b in pick:
            ns_row, _ = cache.get(int(init[b]))
            ok = np.nonzero(ns_row != -1)[0]
            cols.append(int(ok[rng.integers(0, ok.size)]) if ok.size else 0)
        x[torch.from_numpy(pick).to(DEV), torch.from_numpy(np.array(cols, np.int64)).to(DEV)] = 30.0
    states = _dev(init)
    tok, new = dv.masked_step(ns, al, states, x, opportunistic=True)
    t2, n2 = dv.masked_step(ns, al, states, x)
    torch.cuda.synchronize()
    assert torch.equal(tok, t2) and torch.equal(new, n2)
    rows = np.unique(np.concatenate([[0, w.B - 1], rng.integers(0, w.B, 14)]))
    xr = to_oracle(x[torch.from_numpy(rows.astype(np.int64)).to(DEV)])
    for i, b in enumerate(rows):
        t_o, _ = oracle.masked_chain(cache, init[b], xr[i][None])
        assert int(tok[b]) == int(t_o[0]), f"workload {wid} row {b}"


# ----------------------------------------------- masked sampling (Sec. 4: T = 1.0)

SEED = 0x5EED_0000_0000_2403


def _sample_chain(dv, ns, al, init_states, x, seed, inv_t, ws):
    """Sampled decoding on the device: step k draws with offset k."""
    steps, B = x.shape[0], x.shape[1]
    sts = torch.empty((steps + 1, B), dtype=torch.int32, device=DEV)
    tks = torch.empty((steps, B), dtype=torch.int32, device=DEV)
    sts[0].copy_(init_states)
    for k in range(steps):
        dv.masked_sample(ns, al, sts[k], x[k], seed, k, inv_temperature=inv_t, token=tks[k],
                         new_state=sts[k + 1], workspace=ws)
    return tks, sts


@pytest.mark.parametrize("wid,steps,inv_t", [(1, 64, 1.0), (2, 64, 1.0), (2, 16, 0.5), (3, 16, 1.0),
                                             (6, 32, 1.0), (7, 32, 2.0), (8, 32, 1.0), (9, 32, 1.0),
                                             (10, 32, 0.5)])
def test_sample_chain_workload_full(dv, wid, steps, inv_t):
    """Every row and step against the oracle's own sampled chain (its own
    table, its own previous states)."""
    w = W.WORKLOADS[wid]
    _say(f"sampled chain workload {w.describe()} steps={steps} 1/T={inv_t}")
    trans, offsets, data, ns, al = _workload_table(dv, wid)
    ns_o, al_o = oracle.align(trans, offsets, data)
    init = W.init_states(wid)
    x = W.logits_all(wid, device=DEV, steps=steps)
    ws = dv.sample_workspace(w.B, w.V, DEV)
    tks, sts = _sample_chain(dv, ns, al, _dev(init), x, SEED + wid, inv_t, ws)
    torch.cuda.synchronize()
    xs = to_oracle(x)
    cur = init
    for k in range(steps):
        t_o, n_o = oracle.masked_sample(ns_o, al_o, cur, xs[k], inv_t, SEED + wid, k)
        np.testing.assert_array_equal(tks[k].cpu().numpy(), t_o, err_msg=f"workload {wid} step {k}")
        np.testing.assert_array_equal(sts[k + 1].cpu().numpy(), n_o, err_msg=f"workload {wid} step {k}")
        cur = n_o
    # a sampled chain differs from the greedy one (it is a draw, not the argmax)
    g_t, _ = oracle.masked_step(ns_o, al_o, init, xs[0])
    assert (tks[0].cpu().numpy() != g_t).any() or w.B == 1


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("inv_t", [1.0, 0.25, 3.0, 1e4])
@pytest.mark.parametrize("B,layout", [(1030, "misaligned"), (1030, "aligned"), (100, "misaligned"),
                                      (100, "aligned")])
def test_sample_planted_and_random_rows(dv, dtype, inv_t, B, layout):
    """Random tables (dead and out-of-range states), NaN, +-inf and tied
    logits, V = 4099 (a last group of 3 tokens), rows of stride V + 1 that
    start aligned to a 4-token group or one element off it; B = 1030 takes one
    block per row, B = 100 splits rows over blocks."""
    rng = np.random.default_rng(int(inv_t * 100) + (dtype == torch.float32) + B)
    S, V = 11, 4099
    off = 1 if layout == "misaligned" else 0
    alive = rng.random((S, V)) < rng.choice([0.0, 0.003, 0.1, 0.6, 1.0], size=(S, 1))
    ns = np.where(alive, rng.integers(0, S, (S, V)), -1).astype(np.int32)
    Wd = (V + 31) // 32
    pad = np.zeros((S, Wd * 32), bool)
    pad[:, :V] = alive
    al = np.packbits(pad, axis=1, bitorder="little").view("<u4").reshape(S, Wd)
    states = rng.integers(-2, S + 2, B).astype(np.int32)
    buf = torch.from_numpy((rng.standard_normal(B * (V + 1) + 8) * 3).astype(np.float32)).to(dtype)
    buf[torch.from_numpy(rng.integers(0, buf.numel(), 200))] = float("nan")
    buf[torch.from_numpy(rng.integers(0, buf.numel(), 20))] = float("inf")
    buf[torch.from_numpy(rng.integers(0, buf.numel(), 20))] = -float("inf")
    buf[: 5 * (V + 1)] = 1.5                                  # rows 0-4: every logit tied
    x_h = buf[off:off + B * (V + 1)].view(B, V + 1)[:, :V]    # row stride V + 1
    x = buf.to(DEV)[off:off + B * (V + 1)].view(B, V + 1)[:, :V]
    tok, new = dv.masked_sample(_dev(ns), _dev(al.view(np.int32)), _dev(states), x, 77, 5, inv_temperature=inv_t)
    t_o, n_o = oracle.masked_sample(ns, al, states, to_oracle(x_h.contiguous()), inv_t, 77, 5)
    np.testing.assert_array_equal(tok.cpu().numpy(), t_o)
    np.testing.assert_array_equal(new.cpu().numpy(), n_o)


def _queue_mode_masks(rng, S, V):
    """Allow sets built per aligned 2,048-token window (the tokens one wave
    compacts per pass), cycling through the patterns on both sides of the
    sampler's choice between queuing single tokens and 4-token groups:
    sparse random (about 1.1 tokens per group), runs of whole groups (4 per
    group), exactly 512 tokens at 2 per group (the queue full, ratio 2),
    513 tokens (one past the queue), ratio just above 2, empty and full."""
    alive = np.zeros((S, V), bool)
    nwin = (V + 2047) // 2048
    for st in range(S):
        for w in range(nwin):
            lo, hi = w * 2048, min(V, (w + 1) * 2048)
            n = hi - lo
            kind = (st * nwin + w) % 7
            m = np.zeros(n, bool)
            if kind == 0:
                m = rng.random(n) < 0.05
            elif kind == 1:  # runs of whole groups
                for g0 in rng.choice(n // 4, size=min(n // 4, 75), replace=False):
                    m[4 * g0:4 * g0 + 4] = True
            elif kind in (2, 3) and n >= 2048:  # 256 groups of 2 (+ one more token for 513)
                groups = rng.choice(512, size=257, replace=False)
                for g0 in groups[:256]:
                    m[4 * g0 + rng.choice(4, size=2, replace=False)] = True
                if kind == 3:
                    m[4 * groups[256] + rng.integers(0, 4)] = True
            elif kind == 4 and n >= 2048:  # 100 groups of 2 and 20 of 3: 4 T = 1,040 > 8 G = 960
                groups = rng.choice(n // 4, size=120, replace=False)
                for i, g0 in enumerate(groups):
                    m[4 * g0 + rng.choice(4, size=2 if i < 100 else 3, replace=False)] = True
            elif kind == 5:
                m[:] = True
            alive[st, lo:hi] = m
    return alive


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B", [40, 200, 1030])
def test_sample_token_and_group_queues(dv, dtype, B):
    """Masks on both sides of every bound of the token-or-group queue choice
    (see `_queue_mode_masks`), V = 20,517 (a ragged last window), rows split
    over blocks with half an allow word per lane (B = 40) and a whole word
    (B = 200), and one block per row (B = 1,030)."""
    rng = np.random.default_rng(9000 + B + (dtype == torch.float32))
    S, V = 9, 2048 * 10 + 37
    alive = _queue_mode_masks(rng, S, V)
    ns = np.where(alive, rng.integers(0, S, (S, V)), -1).astype(np.int32)
    Wd = (V + 31) // 32
    pad = np.zeros((S, Wd * 32), bool)
    pad[:, :V] = alive
    al = np.packbits(pad, axis=1, bitorder="little").view("<u4").reshape(S, Wd)
    states = np.concatenate([np.arange(S), rng.integers(-1, S, B - S)]).astype(np.int32)
    x_h = torch.from_numpy((rng.standard_normal((B, V)) * 3).astype(np.float32)).to(dtype)
    x = x_h.to(DEV)
    for seed, off in ((3, 0), (4, 17)):
        tok, new = dv.masked_sample(_dev(ns), _dev(al.view(np.int32)), _dev(states), x, seed, off)
        t_o, n_o = oracle.masked_sample(ns, al, states, to_oracle(x_h), 1.0, seed, off)
        np.testing.assert_array_equal(tok.cpu().numpy(), t_o)
        np.testing.assert_array_equal(new.cpu().numpy(), n_o)


def test_sample_is_reproducible_and_graph_safe(dv):
    w = W.WORKLOADS[3]
    trans, offsets, data, ns, al = _workload_table(dv, 3)
    x = W.logits(3, 0, device=DEV)
    st = _dev(W.init_states(3))
    ws = dv.sample_workspace(w.B, w.V, DEV)
    t1, n1 = dv.masked_sample(ns, al, st, x, 123, 0, workspace=ws)
    t2, _ = dv.masked_sample(ns, al, st, x, 123, 0, workspace=ws)
    t3, _ = dv.masked_sample(ns, al, st, x, 123, 1, workspace=ws)
    t4, _ = dv.masked_sample(ns, al, st, x, 124, 0, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(t1, t2)
    assert (t1 != t3).sum() > w.B // 4 and (t1 != t4).sum() > w.B // 4
    tk = torch.empty_like(t1)
    nw = torch.empty_like(n1)
    side = torch.cuda.Stream(DEV)
    side.wait_stream(torch.cuda.current_stream(DEV))
    with torch.cuda.stream(side):
        dv.masked_sample(ns, al, st, x, 123, 0, token=tk, new_state=nw, workspace=ws)
    torch.cuda.current_stream(DEV).wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        dv.masked_sample(ns, al, st, x, 123, 0, token=tk, new_state=nw, workspace=ws)
    for rep in range(3):
        tk.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(tk, t1) and torch.equal(nw, n1), f"replay {rep}"


@pytest.mark.parametrize("B,V,head,extra_ld", [
    (256, 128_256, 0, 0), (300, 70_001, 3, 5), (256, 4099, 7, 1), (260, 9, 1, 0), (256, 5, 0, 3),
    (1030, 20_517, 5, 0), (512, 65_536, 0, 0),
])
def test_sample_large_batches_every_alignment(dv, B, V, head, extra_ld):
    """bf16 batches of 256 rows or more: every row-start alignment (`head`
    elements before the first 16-byte boundary), rows shorter than a vector,
    random masks from empty to full, planted NaN, +-inf and ties, dead and
    out-of-range states; two draws against the oracle."""
    _say(f"sample large batches B={B} V={V} head={head} ld=V+{extra_ld}")
    rng = np.random.default_rng(B * 31 + V + head)
    S = 9
    alive = rng.random((S, V)) < rng.choice([0.0, 0.002, 0.05, 0.3, 0.97, 1.0], size=(S, 1))
    alive[S - 1, : V // 2] = True                 # a dense half, then an empty half
    alive[S - 1, V // 2:] = False
    ns = np.where(alive, rng.integers(0, S, (S, V)), -1).astype(np.int32)
    Wd = (V + 31) // 32
    pad = np.zeros((S, Wd * 32), bool)
    pad[:, :V] = alive
    al = np.packbits(pad, axis=1, bitorder="little").view("<u4").reshape(S, Wd)
    states = rng.integers(-2, S + 2, B).astype(np.int32)
    ld = V + extra_ld
    offset = (8 - head) % 8
    vals = (rng.standard_normal(B * ld + offset + 8) * 3).astype(np.float32)
    buf = torch.from_numpy(vals).to(torch.bfloat16)
    special = torch.tensor([float("nan"), float("inf"), -float("inf"), 1.5], dtype=torch.bfloat16)
    pos = torch.from_numpy(rng.integers(0, buf.numel(), max(8, buf.numel() // 500)))
    buf[pos] = special[torch.from_numpy(rng.integers(0, 4, pos.numel()))]
    base = torch.empty(buf.numel() + 64, dtype=torch.bfloat16, device=DEV)
    shift = (-(base.data_ptr() // 2)) % 8               # first 16-byte boundary of base
    buf_d = base[shift:shift + buf.numel()]
    buf_d.copy_(buf.to(DEV))
    x = buf_d[offset:offset + B * ld].view(B, ld)[:, :V]
    assert (x.data_ptr() // 2 + head) % 8 == 0
    xo = to_oracle(buf[offset:offset + B * ld].view(B, ld))
    for seed, off in ((5, 0), (6, 123)):
        tok, new = dv.masked_sample(_dev(ns), _dev(al.view(np.int32)), _dev(states), x, seed, off)
        t_o, n_o = oracle.masked_sample(ns, al, states, xo, 1.0, seed, off)
        np.testing.assert_array_equal(tok.cpu().numpy(), t_o)
        np.testing.assert_array_equal(new.cpu().numpy(), n_o)


def test_split_rows_every_meeting_form_one_workspace(dv):
    """Rows split in two, three and four chunks (which meet in pairs) and in
    more (which meet through a maximum and a count), greedy in both dtypes and
    sampled, all through one workspace: every call against the oracle, with
    chunks and whole rows that hold no allowed token, and the workspace all
    zero after every call."""
    rng = np.random.default_rng(4242)
    S = 6
    calls = [("step", torch.bfloat16, 64, 128256), ("step", torch.bfloat16, 100, 128256),
             ("step", torch.bfloat16, 128, 128256), ("step", torch.bfloat16, 33, 128256),
             ("step", torch.float32, 64, 70001), ("step", torch.float32, 100, 70001),
             ("step", torch.float32, 150, 40000), ("step", torch.float32, 20, 70001),
             ("sample", torch.bfloat16, 512, 32000), ("sample", torch.bfloat16, 700, 32000),
             ("sample", torch.float32, 1000, 32000), ("sample", torch.bfloat16, 256, 32000)]
    need = max(dv.masked_step_workspace_bytes(B, V) if k == "step" else dv.masked_sample_workspace_bytes(B, V)
               for k, _, B, V in calls)
    ws = torch.zeros(need, dtype=torch.uint8, device=DEV)
    for i, (kind, dtype, B, V) in enumerate(calls):
        _say(f"meeting forms: {kind} {dtype} B={B} V={V}")
        alive = rng.random((S, V)) < np.array([[0.0], [0.0005], [0.05], [0.6], [1.0], [0.0]])
        alive[5, V // 3: V // 3 + 40] = True          # allowed tokens in one chunk only
        ns = np.where(alive, rng.integers(0, S, (S, V)), -1).astype(np.int32)
        Wd = (V + 31) // 32
        pad = np.zeros((S, Wd * 32), bool)
        pad[:, :V] = alive
        al = np.packbits(pad, axis=1, bitorder="little").view("<u4").reshape(S, Wd)
        states = rng.integers(-1, S, B).astype(np.int32)
        x = torch.from_numpy((rng.standard_normal((B, V)) * 3).astype(np.float32)).to(dtype)
        xo = to_oracle(x)
        if kind == "step":
            tok, new = dv.masked_step(_dev(ns), _dev(al.view(np.int32)), _dev(states), x.to(DEV), workspace=ws)
            t_o, n_o = oracle.masked_step(ns, al, states, xo)
        else:
            tok, new = dv.masked_sample(_dev(ns), _dev(al.view(np.int32)), _dev(states), x.to(DEV), 9, i,
                                        workspace=ws)
            t_o, n_o = oracle.masked_sample(ns, al, states, xo, 1.0, 9, i)
        np.testing.assert_array_equal(tok.cpu().numpy(), t_o, err_msg=f"{kind} {dtype} B={B} V={V}")
        np.testing.assert_array_equal(new.cpu().numpy(), n_o, err_msg=f"{kind} {dtype} B={B} V={V}")
        assert int(torch.count_nonzero(ws)) == 0, f"workspace left non-zero after {kind} {dtype} B={B} V={V}"


def _random_step_case(i):
    rng = np.random.default_rng(0xC0FFEE + i)
    B = int(rng.choice([1, 2, 7, 33, 64, 100, 255, 256, 257, 300, 513, 1024, 1100]))
    V = int(rng.choice([1, 8, 9, 31, 4099, 32000, 50257, 65536, 70001, 128256, 140000, 262147]))
    if B * V > 60_000_000:
        V = max(1, 60_000_000 // B)
    dtype = torch.bfloat16 if rng.random() < 0.75 else torch.float32
    extra_ld = int(rng.choice([0, 0, 1, 3, 8, 13]))
    offset = int(rng.integers(0, 8))
    return rng, B, V, dtype, extra_ld, offset


@pytest.mark.parametrize("case", range(40))
def test_step_random_shapes(dv, case):
    """Seeded random shapes across every launch form of the greedy step (one
    block per row or split rows, mask bytes staged, two ahead or streamed,
    aligned or shifted rows, bf16 and fp32): batch, vocabulary, row stride
    and start offset, mask densities per state, dead and out-of-range
    states, planted NaN, +-inf and signed zeros; greedy and opportunistic
    steps against the oracle."""
    rng, B, V, dtype, extra_ld, offset = _random_step_case(case)
    _say(f"random step case {case}: B={B} V={V} {dtype} ld=V+{extra_ld} offset={offset}")
    S = 7
    alive = rng.random((S, V)) < rng.choice([0.0, 0.001, 0.05, 0.4, 0.95, 1.0], size=(S, 1))
    ns = np.where(alive, rng.integers(0, S, (S, V)), -1).astype(np.int32)
    Wd = (V + 31) // 32
    pad = np.zeros((S, Wd * 32), bool)
    pad[:, :V] = alive
    al = np.packbits(pad, axis=1, bitorder="little").view("<u4").reshape(S, Wd)
    states = rng.integers(-2, S + 1, B).astype(np.int32)
    ld = V + extra_ld
    n = B * ld + offset + 8
    vals = rng.integers(-4, 5, n).astype(np.float32) if rng.random() < 0.5 else \
        (rng.standard_normal(n) * 3).astype(np.float32)
    buf = torch.from_numpy(vals).to(dtype)
    special = torch.tensor([float("nan"), float("inf"), -float("inf"), -0.0, 0.0], dtype=dtype)
    pos = torch.from_numpy(rng.integers(0, n, max(4, n // 2000)))
    buf[pos] = special[torch.from_numpy(rng.integers(0, 5, pos.numel()))]
    buf_d = buf.to(DEV)
    x = buf_d[offset:offset + B * ld].view(B, ld)[:, :V]
    xo = to_oracle(buf[offset:offset + B * ld].view(B, ld))
    tok_o, new_o = oracle.masked_step(ns, al, states, xo)
    for opp in (False, True):
        tok, new = dv.masked_step(_dev(ns), _dev(al.view(np.int32)), _dev(states), x, opportunistic=opp)
        np.testing.assert_array_equal(tok.cpu().numpy(), tok_o, err_msg=f"case {case} opportunistic={opp}")
        np.testing.assert_array_equal(new.cpu().numpy(), new_o, err_msg=f"case {case} opportunistic={opp}")
