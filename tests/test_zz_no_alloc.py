"""dv_masked_step_noalloc (the step whose split rows meet in the library's
own scratch array instead of a caller's workspace) against dv_masked_step
with a workspace, bit for bit, and against the oracle.

Two calls in a row per dtype, the second with a smaller batch and
vocabulary: the first call's rows carry much larger logits than the
second's, so a meeting entry the first call failed to put back to zero
would win the second call's row and show up as a wrong token."""
import numpy as np
import pytest
import torch

import oracle
from tests.gpu_common import to_oracle

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


@pytest.fixture(scope="module")
def dv():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2403_06988_amd as dv_mod
    return dv_mod


def _table(rng, S, V):
    alive = rng.random((S, V)) < np.linspace(0.0, 1.0, S)[:, None] ** 2
    ns = np.where(alive, rng.integers(0, S, (S, V)), -1).astype(np.int32)
    Wd = (V + 31) // 32
    pad = np.zeros((S, Wd * 32), bool)
    pad[:, :V] = alive
    al = np.packbits(pad, axis=1, bitorder="little").view("<u4").reshape(S, Wd)
    return ns, al


def _case(dv, rng, dtype, B, V, extra_ld, scale):
    S = 9
    ns, al = _table(rng, S, V)
    states = rng.integers(-1, S, B).astype(np.int32)
    states[0] = S - 1                      # a row with every token allowed
    full = torch.from_numpy((rng.integers(-4, 5, (B, V + extra_ld)) * scale).astype(np.float32)).to(dtype)
    x = full[:, :V]                        # row stride V + extra_ld
    xd = full.to(DEV)[:, :V]
    nsd = torch.from_numpy(ns).to(DEV)
    ald = torch.from_numpy(al.view(np.int32)).to(DEV)
    st = torch.from_numpy(states).to(DEV)
    tok = torch.full((B,), 77, dtype=torch.int32, device=DEV)
    new = torch.full((B,), 77, dtype=torch.int32, device=DEV)
    dv.masked_step_noalloc(nsd, ald, st, xd, tok, new)
    ref_t, ref_n = dv.masked_step(nsd, ald, st, xd)
    torch.cuda.synchronize()
    assert torch.equal(tok, ref_t) and torch.equal(new, ref_n)
    t_o, n_o = oracle.masked_step(ns, al, states, to_oracle(x.contiguous()))
    np.testing.assert_array_equal(tok.cpu().numpy(), t_o)
    np.testing.assert_array_equal(new.cpu().numpy(), n_o)


@pytest.mark.parametrize("dtype,first,second", [
    # (B, V, extra row stride): rows split over several blocks at these batches
    (torch.bfloat16, (8, 128256, 0), (3, 70001, 5)),
    (torch.float32, (6, 40000, 0), (2, 5003, 3)),
])
def test_noalloc_step_matches_the_workspace_step(dv, dtype, first, second):
    rng = np.random.default_rng(1234)
    print(f"noalloc step {dtype} first B,V,extra={first}", flush=True)
    _case(dv, rng, dtype, *first, scale=25.0)
    print(f"noalloc step {dtype} second B,V,extra={second}", flush=True)
    _case(dv, rng, dtype, *second, scale=1.0)


def test_noalloc_step_rejects_a_batch_beyond_the_scratch(dv):
    n = dv.NOALLOC_MAX_BATCH + 1
    ns = torch.zeros((2, 10), dtype=torch.int32, device=DEV)
    al = torch.zeros((2, 1), dtype=torch.int32, device=DEV)
    st = torch.zeros(n, dtype=torch.int32, device=DEV)
    x = torch.zeros((n, 10), dtype=torch.bfloat16, device=DEV)
    tok = torch.empty(n, dtype=torch.int32, device=DEV)
    new = torch.empty(n, dtype=torch.int32, device=DEV)
    with pytest.raises(dv.DvError) as e:
        dv.masked_step_noalloc(ns, al, st, x, tok, new)
    assert "DV_NOALLOC_MAX_BATCH" in str(e.value)
