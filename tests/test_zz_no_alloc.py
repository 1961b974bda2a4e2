"""ress_select_noalloc, the selection entry point for callers that cannot
allocate (its workspace is the library's fixed per-GPU scratch array), against
ress_select with a caller workspace on the same inputs: every output identical,
on calls in a row over layers that shrink (32 views, 8 views, a 301-token layer on
the 64-token grid) and then grow again (32 views on the 128/64 grid), so that
nothing left in the scratch array from a previous call can matter. Also the host-side checks
(no GPU work): a shape whose workspace exceeds the scratch array, and a pooled
state the caller cannot have written there."""
import ctypes as C

import numpy as np
import pytest

import synth
from gpu_helpers import device_inputs, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ress():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_35593_amd as r

    return r


def _outputs(L, dev):
    import torch

    return dict(kept_count=torch.full((L.H, L.n_qb), -7, dtype=torch.int32, device=dev),
                kept_idx=torch.full((L.H, L.n_qb, L.n_kb), -7, dtype=torch.int32, device=dev),
                drift=torch.full((L.H, L.n_qb, 2), -7.0, dtype=torch.float64, device=dev),
                key_out=torch.full((L.H, L.n_qb, L.n_kb), -7.0, dtype=torch.float64, device=dev),
                prob_out=torch.full((L.H, L.n_qb, L.n_kb), -7.0, dtype=torch.float64, device=dev))


def test_noalloc_matches_select_in_a_row(ress):
    import torch

    dev = "cuda:0"
    layers = (synth.make_config("32v"), synth.make_config("8v", sparsity=0.5),
              synth.make_layer(1, 300, 1, H=3, block=64, sparsity=0.5, seed=77, name="n301"),
              synth.make_config("32v", bk=64))
    for L in layers:
        say(f"[noalloc] {L.name} H={L.H} N={L.N} n_kb={L.n_kb}")
        q, k, v, gram = device_inputs(L, dev)
        kw = dict(bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail, rounds=5)
        out = _outputs(L, dev)
        got = ress.ress_select_noalloc(q, k, v, gram, L.budgets, **kw, **out)
        ref = ress.ress_select(q, k, v, gram, L.budgets, want_debug=True, **kw)
        torch.cuda.synchronize()
        for name in ("kept_count", "kept_idx", "drift", "key", "prob"):
            assert torch.equal(got[name], ref[name]), (L.name, name)
        assert int((got["kept_count"] < 0).sum()) == 0


def test_noalloc_host_checks(ress):
    """Rejected on the host before any device work: a workspace beyond the scratch
    array (100 views, 256 heads) and pooled_in_workspace."""
    shape = ress.make_shape(64, 137400, bq=128, bk=128, n_special_tail=500)
    assert ress.ress_select_workspace_size(shape) > ress.NOALLOC_SCRATCH_BYTES
    params = ress.ress_select_params(5, 0.5, 1e-4, 1, 1, 0, 0.0, 0)
    budget = np.full(64, 100, np.int32)
    p = C.c_void_p(1 << 41)
    st = ress.lib.ress_select_noalloc(C.byref(shape), C.byref(params), p, p, p, p, budget.ctypes.data, p, p, None,
                                      None, None, None)
    assert st == ress.RESS_E_UNSUPPORTED
    small = ress.make_shape(2, 1230, bq=64, bk=64)
    params.pooled_in_workspace = 1
    st = ress.lib.ress_select_noalloc(C.byref(small), C.byref(params), p, p, p, p, budget.ctypes.data, p, p, None,
                                      None, None, None)
    assert st == ress.RESS_E_INVALID_ARG
