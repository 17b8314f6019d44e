"""Host-side arithmetic of bench.py, on the CPU: the algorithmic byte count of
the masked step (the 128-byte logit lines that hold an allowed token) against
a brute-force count over every line of every row."""
import numpy as np
import pytest
import torch

import bench


def brute(al, states, base, ld, V, elt):
    total = 0
    for r, s in enumerate(states.tolist()):
        if s < 0:
            continue
        start = base + r * ld * elt
        lines = set()
        for i in range(V):
            if (int(al[s, i >> 5]) >> (i & 31)) & 1:
                lines.add((start + i * elt) // 128)
        total += 128 * len(lines)
    return total


@pytest.mark.parametrize("V,elt,ld,base", [
    (1000, 4, 1000, 0), (1000, 4, 1003, 4), (4099, 2, 4099, 2), (4099, 2, 4107, 126), (64, 2, 64, 0),
    (65, 2, 70, 64), (1, 4, 1, 124), (300, 2, 300, 0),
])
def test_touched_line_bytes_matches_brute_force(V, elt, ld, base):
    rng = np.random.default_rng(V + ld + base)
    S, B = 5, 7
    W = (V + 31) // 32
    dens = np.array([0.0, 0.003, 0.05, 0.5, 1.0])[:, None]
    alive = rng.random((S, W * 32)) < dens
    alive[:, V:] = False
    al = np.packbits(alive, axis=1, bitorder="little").view("<u4").reshape(S, W).view(np.int32)
    states = rng.integers(-2, S, B).astype(np.int32)
    got = bench.touched_line_bytes(torch.from_numpy(al), torch.from_numpy(states), base, ld, V, elt)
    assert got == brute(al.view(np.uint32), states, base, ld, V, elt)


def test_touched_line_bytes_whole_rows_when_all_allowed():
    V, B = 128256, 3
    al = torch.full((1, (V + 31) // 32), -1, dtype=torch.int32)
    states = torch.zeros(B, dtype=torch.int32)
    assert bench.touched_line_bytes(al, states, 0, V, V, 2) == B * V * 2  # rows are whole lines
    assert bench.touched_line_bytes(al, torch.full((B,), -1, dtype=torch.int32), 0, V, V, 2) == 0


def test_inputs_record_names_the_inputs():
    """The bench line's input record: hashes that change with any input
    byte, and the realised token lengths."""
    trans = np.full((3, 256), -1, np.int32)
    trans[0, 97] = 1
    offsets = np.array([0, 1, 3, 3, 7], np.int32)
    data = np.frombuffer(b"abcdefg", np.uint8)
    init = np.zeros(2, np.int32)
    r = bench.inputs_record(trans, offsets, data, init)
    assert r["token_len_mean"] == 7 / 4 and r["token_len_max"] == 4 and r["token_bytes"] == 7
    assert r == bench.inputs_record(trans.copy(), offsets.copy(), data.copy(), init.copy())
    t2 = trans.copy()
    t2[2, 5] = 0
    d2 = data.copy()
    d2[6] = ord("h")
    assert bench.inputs_record(t2, offsets, data, init)["dfa_sha256"] != r["dfa_sha256"]
    assert bench.inputs_record(trans, offsets, d2, init)["vocab_sha256"] != r["vocab_sha256"]
    assert bench.inputs_record(trans, offsets, data, init + 1)["init_states_sha256"] != r["init_states_sha256"]


def test_kernel_source_hash_ignores_comments_only(tmp_path, monkeypatch):
    """A recorded measurement stays attached to its kernel through edits of
    the comments alone, and detaches on any change of code."""
    import bench

    src = tmp_path / "k.hip"
    monkeypatch.setattr(bench, "CSRC", str(tmp_path))
    monkeypatch.setattr(bench, "KERNEL_SOURCES", {"k": ("k.hip",)})
    src.write_text("// header\nint f(int x) { return x + 1; }  // add one\n\n")
    h0 = bench.kernel_source_hash("k")
    src.write_text("// a longer header\n\n// more words\nint f(int x) { return x + 1; }  // adds one\n")
    assert bench.kernel_source_hash("k") == h0
    src.write_text("// header\nint f(int x) { return x + 2; }  // add one\n")
    assert bench.kernel_source_hash("k") != h0
