"""Selection and block-sparse attention recorded in a HIP graph (torch.cuda.CUDAGraph
captured on the caller's stream). With every output and the selection workspace
passed in, the entry points only launch kernels on that stream (no allocation,
memset or synchronisation), so one layer's selection + attention can be captured
once and replayed. Every replay, with eager work and a synchronisation between
replays and the outputs overwritten before each, must reproduce the eager results
exactly (the kernels are deterministic). Also two layers enqueued on two streams
at once (default priority) against their runs alone."""
import pytest

import synth
from gpu_helpers import device_inputs, say

pytestmark = pytest.mark.gpu


def test_select_and_sparse_attention_graph_replay():
    import torch

    import paper_2609_35593_amd as ress

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    dev = torch.device("cuda:0")
    L = synth.make_config("8v", sparsity=0.5)
    say(f"[graph] {L.name} H={L.H} N={L.N} n_kb={L.n_kb}")
    q, k, v, gram = device_inputs(L, dev)
    shape = ress.make_shape(L.H, L.N, bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail)
    ws = torch.empty(ress.ress_select_workspace_size(shape), dtype=torch.uint8, device=dev)
    kc = torch.empty((L.H, L.n_qb), dtype=torch.int32, device=dev)
    ki = torch.empty((L.H, L.n_qb, L.n_kb), dtype=torch.int32, device=dev)
    drift = torch.empty((L.H, L.n_qb, 2), dtype=torch.float64, device=dev)
    o = torch.empty_like(q)
    stream = torch.cuda.Stream(device=dev)

    def layer():
        ress.ress_select(q, k, v, gram, L.budgets, bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail, rounds=5,
                         kept_count=kc, kept_idx=ki, drift=drift, workspace=ws, stream=stream)
        ress.ress_sparse_attn(q, k, v, kc, ki, bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail, out=o,
                              stream=stream)

    stream.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(stream):
        layer()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (kc, ki, drift, o)]
    assert int((ref[0] < 0).sum()) == 0

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        layer()
    torch.cuda.synchronize()
    for rep in range(3):
        # Eager work between replays: overwrite every output.
        kc.fill_(-3)
        ki.fill_(-3)
        drift.fill_(-3.0)
        o.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, t, r in zip(("kept_count", "kept_idx", "drift", "out"), (kc, ki, drift, o), ref):
            assert torch.equal(t, r), (rep, name)
        say(f"[graph] replay {rep}: identical to the eager layer")


def test_two_streams_at_once():
    """Two layers' selection + attention enqueued on two streams at once (each with
    its own outputs and workspace): the calls share no state, so each stream's
    results equal those of the same calls run alone."""
    import torch

    import paper_2609_35593_amd as ress

    dev = torch.device("cuda:0")
    layers = [synth.make_config("8v", sparsity=0.5), synth.make_layer(3, 700, 5, H=4, bq=128, bk=64, seed=9)]
    runs = []
    for L in layers:
        q, k, v, gram = device_inputs(L, dev)
        shape = ress.make_shape(L.H, L.N, bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail)
        runs.append(dict(L=L, q=q, k=k, v=v, gram=gram,
                         ws=torch.empty(ress.ress_select_workspace_size(shape), dtype=torch.uint8, device=dev),
                         kc=torch.empty((L.H, L.n_qb), dtype=torch.int32, device=dev),
                         ki=torch.empty((L.H, L.n_qb, L.n_kb), dtype=torch.int32, device=dev),
                         o=torch.empty_like(q)))

    def layer(r, stream):
        L = r["L"]
        ress.ress_select(r["q"], r["k"], r["v"], r["gram"], L.budgets, bq=L.bq, bk=L.bk,
                         n_special_tail=L.n_special_tail, kept_count=r["kc"], kept_idx=r["ki"], workspace=r["ws"],
                         want_drift=False, stream=stream)
        ress.ress_sparse_attn(r["q"], r["k"], r["v"], r["kc"], r["ki"], bq=L.bq, bk=L.bk,
                              n_special_tail=L.n_special_tail, out=r["o"], stream=stream)

    alone = torch.cuda.current_stream(dev)
    ref = []
    for r in runs:
        layer(r, alone)
        torch.cuda.synchronize()
        ref.append([r[n].clone() for n in ("kc", "ki", "o")])
    streams = [torch.cuda.Stream(device=dev) for _ in runs]
    for rep in range(3):
        for r in runs:
            r["kc"].fill_(-3)
            r["ki"].fill_(-3)
            r["o"].zero_()
        torch.cuda.synchronize()
        for r, s in zip(runs, streams):
            layer(r, s)
        torch.cuda.synchronize()
        for i, r in enumerate(runs):
            for n, t0 in zip(("kc", "ki", "o"), ref[i]):
                assert torch.equal(r[n], t0), (rep, i, n)
        say(f"[two streams] repetition {rep}: both layers identical to their runs alone")
