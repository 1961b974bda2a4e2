"""Benchmark of one global-attention layer of the ReSS hot path on one MI355X.

One step = ress_select (pooling, drift scores, top-c, R restoration rounds,
kept lists) + ress_sparse_attn (block-sparse attention over the kept blocks) on
one synthetic layer whose inputs are already resident in HBM; L2 and the
infinity cache are flushed before every step (outside its timing). The default
workload is 32 views x 1374 tokens (43,968 tokens), 16 heads x 64, blocks of 128,
75% block sparsity, 5 rounds. --config 16v_stack runs the 24-layer stack end to
end with its float32 residual stream; --rounds-sweep adds config 3's sweep of
the restoration rounds.

Prints one JSON line (rank 0). Also reports: the dense attention baseline of the
same library, per-kernel times from HIP events recorded on the launch stream,
the roofline object of the dominant kernel (block-sparse attention, bf16 MFMA),
and the CPU oracle timed on a bounded sample of the same layer.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "ms/layer (selection + block-sparse attn) and % bf16 MFMA peak at 32 views"
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "sparse_attn_32v_traffic.txt")
ATTN_SRC = os.path.join(ROOT, "paper_2609_35593_amd", "csrc", "attn.hip")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="32v", help="workload: tiny, 8v, 32v, 100v, 16v_stack")
    ap.add_argument("--sparsity", type=float, default=None,
                    help="uniform target sparsity (default: the workload's own; 100v draws per-head sparsities)")
    ap.add_argument("--bq", type=int, default=None, help="query block size (default: the workload's)")
    ap.add_argument("--bk", type=int, default=None, help="key block size (default: the workload's)")
    ap.add_argument("--no-flush", action="store_true", help="time back-to-back steps without flushing the caches before each")
    ap.add_argument("--no-criteria", action="store_true", help="skip the per-criterion drift report")
    ap.add_argument("--no-masking", action="store_true", help="skip the single-block masking report")
    ap.add_argument("--no-neighbours", action="store_true", help="skip the fused-projection report")
    ap.add_argument("--rounds", type=int, default=5)
    ap.add_argument("--dense-steps", type=int, default=5)
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the CPU oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of known size (for HBM counter scaling)")
    ap.add_argument("--rounds-sweep", default=None,
                    help="comma-separated restoration rounds: selection time and J_best/J_init per R")
    return ap.parse_args()


def kept_flops(L, kc, ki):
    """4 D flops per (query token, kept key token) pair, summed over the layer."""
    q_len = np.minimum(L.bq, L.N - np.arange(L.n_qb) * L.bq)
    k_len = np.minimum(L.bk, L.N - np.arange(L.n_kb) * L.bk)
    kc = kc.reshape(L.H, L.n_qb)
    ki = ki.reshape(L.H, L.n_qb, L.n_kb)
    keys = np.where(ki >= 0, k_len[np.clip(ki, 0, None)], 0).sum(axis=2)  # [H][n_qb]
    return 4.0 * L.D * float((keys * q_len[None, :]).sum()), int(kc.sum())


def select_bytes(L):
    """Algorithmic HBM bytes of one ress_select: Q, K, V read once (bf16); the
    float64 pooled tensors (qbar, and kbar^T, vbar, vbar^T, M vbar) written once
    and read once; kept lists (padded to n_kb), counts and drift written once."""
    qkv = 3.0 * L.H * L.N * L.D * 2
    pooled = 2.0 * L.H * (L.n_qb + 4 * L.n_kb) * L.D * 8
    lists = 4.0 * L.H * L.n_qb * (L.n_kb + 1) + 16.0 * L.H * L.n_qb
    return qkv + pooled + lists


def traffic_from_profile():
    """HBM bytes per sparse-attention launch measured with rocprofv3 counters, if
    they were taken on the current kernel source (else None)."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    vals = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    sha = hashlib.sha256(open(ATTN_SRC, "rb").read()).hexdigest()[:16]
    if vals.get("attn_source_sha256_16") != sha or "hbm_bytes_per_launch" not in vals:
        return None
    return float(vals["hbm_bytes_per_launch"])


def cpu_baseline(L, rounds, kc_gpu, ki_gpu, budget_s):
    """The oracle on the host cores: selection of a sample of rows and sparse
    attention of a sample of query tokens, each scaled to the whole layer."""
    import oracle

    threads = oracle.max_threads()
    rng = np.random.default_rng(0)
    R = L.H * L.n_qb
    n_rows = min(R, 512)
    rows = np.sort(rng.choice(R, size=n_rows, replace=False)).astype(np.int32)
    t0 = time.perf_counter()
    oracle.select(L.q, L.k, L.v, L.gram, L.budgets, N=L.N, bq=L.bq, bk=L.bk, n_special=L.n_special_tail,
                  rounds=rounds, rows=rows, want_key=False)
    t_sel = time.perf_counter() - t0
    n_tok = 256
    toks = 0
    t_attn = 0.0
    while t_attn < budget_s and toks < L.H * L.N:
        hs = rng.integers(0, L.H, n_tok).astype(np.int32)
        ts = rng.integers(0, L.N, n_tok).astype(np.int32)
        t0 = time.perf_counter()
        oracle.attn_tokens(L.q, L.k, L.v, N=L.N, bq=L.bq, bk=L.bk, scale=1 / math.sqrt(L.D), sel_h=hs, sel_t=ts,
                           kept_count=kc_gpu, kept_idx=ki_gpu)
        t_attn += time.perf_counter() - t0
        toks += n_tok
        n_tok *= 2
    ms = 1e3 * (t_sel * R / n_rows + t_attn * (L.H * L.N) / toks)
    return {"value": round(ms, 3), "unit": "ms/layer", "cores": threads, "kind": "oracle",
            "sample": f"selection of {n_rows} of {R} (head, query block) rows and sparse attention of "
                      f"{toks} of {L.H * L.N} (head, query token) rows, each timed and scaled linearly "
                      f"to the whole layer (float64, {threads} OpenMP threads)",
            "measured_seconds": round(t_sel + t_attn, 2)}


def measured_ceilings(torch, dev):
    """What the box delivers on plain library work, as context for the published
    peaks used in the roofline: a large bf16 GEMM (hipBLASLt through torch.mm)
    and a 1 GiB device-to-device copy."""
    n = 8192
    a = torch.randn((n, n), device=dev).to(torch.bfloat16).contiguous()
    b = torch.randn((n, n), device=dev).to(torch.bfloat16).contiguous()
    for _ in range(3):
        torch.mm(a, b)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        torch.mm(a, b)
    e1.record()
    torch.cuda.synchronize()
    gemm_tflops = 2.0 * n ** 3 * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e12
    del a, b
    x = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
    y = torch.empty_like(x)
    y.copy_(x)
    e0.record()
    for _ in range(5):
        y.copy_(x)
    e1.record()
    torch.cuda.synchronize()
    copy_gbs = 2.0 * (1 << 30) * 5 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del x, y
    return {"bf16_gemm_8192_tflops": round(gemm_tflops, 1), "copy_1gib_read_plus_write_gbs": round(copy_gbs, 1)}


def criteria_report(ress, L, q, k, v, gram, o_dense, stream):
    """The paper's comparison of selection criteria at one budget (Table 2 rows and
    the sign-flipped objective of Fig. 8, Sec. 6.1), on this synthetic layer: for each
    criterion the median pooled drift J of the returned selection (over rows that
    drop blocks) and the token-level residual drift it leaves,
    sum ||W_O (O_sparse - O_dense)||^2 / sum ||W_O O_dense||^2 over every token and
    head, with ||W_O x||^2 = x^T M x. Everything runs in this library's kernels
    (the norms per query block in ress_block_drift_sq); torch only adds up the
    per-block sums."""
    import torch

    cases = [("drift, R=5 (ReSS)", 0, 0.0, 5), ("drift, R=0", 0, 0.0, 0), ("probability top-k", 1, 0.0, 0),
             ("probability top-k + CDF 0.9", 1, 0.9, 0), ("drift maximised, swaps only", 2, 0.0, 5),
             ("drift maximised, full", 3, 0.0, 5)]
    gram32 = gram.float()
    od = o_dense.float()
    zero = torch.zeros_like(od)
    base = ress.ress_block_drift_sq(od, zero, gram32, bq=L.bq, stream=stream).sum().item()
    rep = []
    for label, crit, tau, rounds in cases:
        sel = ress.ress_select(q, k, v, gram, L.budgets, bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail,
                               rounds=rounds, criterion=crit, cdf_tau=tau, stream=stream)
        o = ress.ress_sparse_attn(q, k, v, sel["kept_count"], sel["kept_idx"], bq=L.bq, bk=L.bk, stream=stream)
        resid = ress.ress_block_drift_sq(o.float(), od, gram32, bq=L.bq, stream=stream).sum().item()
        dr = sel["drift"].reshape(-1, 2)
        live = dr[:, 0] > 0
        kept = sel["kept_count"].sum().item()
        rep.append({"criterion": label, "J_median": float(dr[live, 1].median().item()) if live.any() else 0.0,
                    "residual_drift_rel": resid / base, "kept_tiles": int(kept)})
    return rep


def input_stats(ress, L, q, k, v, gram, o_dense, stream):
    """Sanity statistics of the synthetic layer (not targets): the mean over (head,
    query block) rows of the pooled map's largest probability max_j P_ij and of its
    normalised entropy -sum_j P_ij log P_ij / log n_kb (Eq. 1's P, as the selection
    computes it), and the mean |O| of the dense attention output (small values keep
    the bf16 output rounding well inside the parity bounds)."""
    import torch

    sel = ress.ress_select(q, k, v, gram, L.budgets, bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail,
                           want_debug=True, stream=stream)
    P = sel["prob"].double()
    ent = -torch.where(P > 0, P * torch.log(P), torch.zeros_like(P)).sum(-1) / math.log(L.n_kb)
    mean_abs_o = o_dense.float().abs().mean()
    torch.cuda.synchronize()
    return {"pooled_row_max_p_mean": round(float(P.max(-1).values.mean()), 4),
            "pooled_row_entropy_normalised_mean": round(float(ent.mean()), 4),
            "dense_output_mean_abs": round(float(mean_abs_o), 4)}


def masking_report(ress, L, q, k, v, gram, stream):
    """Sec. 3's test of the probability assumption (Fig. 2) on this synthetic layer:
    mask one candidate key block at a time (every query block attends to all other
    blocks, float32 outputs from this library's kernel) and measure the change
    ||W_O (O_masked - O_dense)|| over each query block's tokens; then, per selected
    row, the Spearman correlation of that change with the pooled probability P_ij,
    the drift score s_ij (Eq. 6) and the ranking key s_ij / (1 - P_ij) (Eq. 7) over
    the row's candidates. Dense special rows are left out."""
    import torch

    from paper_2609_35593_amd import masking
    import synth

    t0 = time.time()
    n_qb, n_kb = L.n_qb, L.n_kb
    nf = synth.forced_block_count(L.N, L.bk, L.n_special_tail)
    cand = np.arange(n_kb - nf)
    sel = ress.ress_select(q, k, v, gram, L.budgets, bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail,
                           want_debug=True, stream=stream)
    P = sel["prob"].cpu().numpy()[:, :, cand]
    key = sel["key"].cpu().numpy()[:, :, cand]
    s = key * np.maximum(1.0 - P, 1e-4)
    change = masking.block_masking_change(q, k, v, gram, bq=L.bq, bk=L.bk, blocks=cand, stream=stream)
    torch.cuda.synchronize()
    first_special = (L.N - L.n_special_tail) // L.bq if L.n_special_tail > 0 else n_qb
    rows = (slice(None), slice(0, first_special))
    out = {"rows": int(L.H * first_special), "candidates": int(len(cand))}
    for name, x in (("probability", P), ("drift_score", s), ("ranking_key", key)):
        r = masking.spearman_rows(change[rows], x[rows])
        r = r[np.isfinite(r)]
        out[name] = {"mean": round(float(r.mean()), 4), "median": round(float(np.median(r)), 4),
                     "p10": round(float(np.percentile(r, 10)), 4), "min": round(float(r.min()), 4)}
    rp = masking.spearman_rows(change[rows], P[rows])
    rk = masking.spearman_rows(change[rows], key[rows])
    out["key_above_probability_frac"] = round(float(np.mean(rk > rp)), 4)
    out["per_head_mean"] = {"probability": [round(float(np.nanmean(rp[h])), 3) for h in range(L.H)],
                            "ranking_key": [round(float(np.nanmean(rk[h])), 3) for h in range(L.H)]}
    out["seconds"] = round(time.time() - t0, 1)
    return out


def neighbours_report(ress, L, stream, reps=10):
    """The steps on either side of the path at this layer's shape, fused into our
    GEMMs against the vendor GEMM (hipBLASLt through torch) plus the layout copies
    and the separate pooling pass the unfused chain needs. Inputs are random
    (x ~ N(0, 1), weights ~ N(0, 1/width)); every time is the mean of `reps`
    back-to-back launches between HIP events on the library's stream."""
    import torch

    dev = torch.device("cuda:0")
    H, N = L.H, L.N
    dm = 64 * H
    g = torch.Generator(device=dev).manual_seed(7)
    x = torch.randn(N, dm, device=dev, generator=g).bfloat16()
    w_qkv = (torch.randn(3 * dm, dm, device=dev, generator=g) / dm ** 0.5).bfloat16()
    w_o = (torch.randn(dm, dm, device=dev, generator=g) / dm ** 0.5).bfloat16()
    resid = torch.randn(N, dm, device=dev, generator=g).bfloat16()
    o = torch.randn(H, N, 64, device=dev, generator=g).bfloat16()
    gram = torch.from_numpy(L.gram).to(dev)
    fused = ress.ress_qkv_proj_pool(x, w_qkv, gram, bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail, stream=stream)
    q, k, v, ws = fused["q"], fused["k"], fused["v"], fused["workspace"]
    y = torch.empty(N, 3 * dm, device=dev, dtype=torch.bfloat16)
    r_out = torch.empty_like(resid)
    sel_kw = dict(bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail, stream=stream)

    def timed(fn):
        with torch.cuda.stream(stream):
            fn()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for _ in range(reps):
                fn()
            b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    def vendor_qkv():
        torch.mm(x, w_qkv.t(), out=y)
        yy = y.view(N, 3, H, 64).permute(1, 2, 0, 3)
        q.copy_(yy[0])
        k.copy_(yy[1])
        v.copy_(yy[2])

    def vendor_out():
        torch.addmm(resid, o.permute(1, 0, 2).reshape(N, dm), w_o.t(), out=r_out)

    t_qkv = timed(lambda: ress.ress_qkv_proj_pool(x, w_qkv, gram, bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail,
                                                  q=q, k=k, v=v, workspace=ws, stream=stream))
    t_sel_pooled = timed(lambda: ress.ress_select(q, k, v, gram, L.budgets, workspace=ws, pooled_in_workspace=True,
                                                  **sel_kw))
    t_sel_plain = timed(lambda: ress.ress_select(q, k, v, gram, L.budgets, **sel_kw))
    t_mm = timed(lambda: torch.mm(x, w_qkv.t(), out=y))
    t_vqkv = timed(vendor_qkv)
    t_out = timed(lambda: ress.ress_out_proj_residual(o, w_o, resid, resid_out=r_out, stream=stream))
    t_vout = timed(vendor_out)
    fl_qkv, fl_out = 2.0 * N * dm * 3 * dm, 2.0 * N * dm * dm
    tf = lambda fl, ms: round(fl / (ms * 1e-3) / 1e12, 1)
    return {
        "qkv_proj_pool_ms": round(t_qkv, 4), "qkv_proj_pool_tflops": tf(fl_qkv, t_qkv),
        "vendor_qkv_mm_ms": round(t_mm, 4), "vendor_qkv_mm_tflops": tf(fl_qkv, t_mm),
        "vendor_qkv_mm_plus_head_major_ms": round(t_vqkv, 4),
        "select_from_fused_pooling_ms": round(t_sel_pooled, 4), "select_with_own_pooling_ms": round(t_sel_plain, 4),
        "before_path_fused_ms": round(t_qkv + t_sel_pooled, 4),
        "before_path_unfused_ms": round(t_vqkv + t_sel_plain, 4),
        "out_proj_residual_ms": round(t_out, 4), "out_proj_residual_tflops": tf(fl_out, t_out),
        "vendor_permute_addmm_ms": round(t_vout, 4), "vendor_permute_addmm_tflops": tf(fl_out, t_vout),
    }


def copy_calibration():
    import torch

    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": n, "copy_calibration_bytes_written": n, "launches": 5}))


def timed_steps(step, n, stream, flush=None):
    """n steps, each bracketed by HIP events on the launch stream (per-kernel
    boundaries as recorded by `step`); with `flush`, L2 and the infinity cache are
    overwritten before every step, outside the events. Returns [n][kernels] ms."""
    import torch

    evs = []
    for _ in range(n):
        if flush is not None:
            flush()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(step.n_events)]
        step(e)
        evs.append(e)
    torch.cuda.synchronize()
    return np.array([[e[i].elapsed_time(e[i + 1]) for i in range(len(e) - 1)] for e in evs])


def stack_run(ress, args, torch, dev, stream, flush):
    """The 24-layer stack end to end: per layer selection + block-sparse attention
    (timed, caches flushed before each layer), the dense attention, and the
    change sparse attention makes to what the layer adds to the residual stream,
    accumulated in a float32 stream of width 1024: r = sum_l W_O^l (O_sparse -
    O_dense) against base = sum_l W_O^l O_dense (Sec. 3, "The Right Objective").
    Layers are drawn on the host one at a time (outside the timed events)."""
    import synth

    out_layers = []
    r = base = None
    t_gen = 0.0
    for layer in range(24):
        t0 = time.time()
        L = synth.make_config("16v_stack", layer=layer, sparsity=args.sparsity)
        w, _ = synth.draw_w_o(L.H, L.D, L.seed)
        w_bits = synth.f32_to_bf16_bits(w.transpose(1, 0, 2).reshape(w.shape[1], L.H * L.D).astype(np.float32))
        q, k, v = (ress.bf16_from_bits(x, dev) for x in (L.q, L.k, L.v))
        gram = torch.from_numpy(L.gram).to(dev)
        w_d, w_neg = ress.bf16_from_bits(w_bits, dev), ress.bf16_from_bits(w_bits ^ np.uint16(0x8000), dev)
        t_gen += time.time() - t0
        if r is None:
            r = torch.zeros((L.N, L.H * L.D), dtype=torch.float32, device=dev)
            base = torch.zeros_like(r)
        kc = torch.empty((L.H, L.n_qb), dtype=torch.int32, device=dev)
        ki = torch.empty((L.H, L.n_qb, L.n_kb), dtype=torch.int32, device=dev)
        drift = torch.empty((L.H, L.n_qb, 2), dtype=torch.float64, device=dev)
        o_s, o_d = torch.empty_like(q), torch.empty_like(q)
        ws = torch.empty(ress.ress_select_workspace_size(
            ress.make_shape(L.H, L.N, bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail)), dtype=torch.uint8,
            device=dev)

        def step(e=None):
            if e is not None:
                e[0].record(stream)
            ress.ress_select(q, k, v, gram, L.budgets, bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail,
                             rounds=args.rounds, kept_count=kc, kept_idx=ki, drift=drift, workspace=ws, stream=stream)
            if e is not None:
                e[1].record(stream)
            ress.ress_sparse_attn(q, k, v, kc, ki, bq=L.bq, bk=L.bk, out=o_s, stream=stream)
            if e is not None:
                e[2].record(stream)
        step.n_events = 3
        for _ in range(2):
            step()
        t = timed_steps(step, 5, stream, flush)
        ress.ress_dense_attn(q, k, v, bq=L.bq, bk=L.bk, out=o_d, stream=stream)
        ress.ress_out_proj_residual_f32(o_s, w_d, r, resid_out=r, stream=stream)
        ress.ress_out_proj_residual_f32(o_d, w_neg, r, resid_out=r, stream=stream)
        ress.ress_out_proj_residual_f32(o_d, w_d, base, resid_out=base, stream=stream)
        torch.cuda.synchronize()
        dr = drift.cpu().numpy().reshape(-1, 2)
        live = dr[:, 0] > 0
        out_layers.append({"layer": layer, "noise_sigma": round(synth.stack_sigma(layer), 4),
                           "select_ms": round(float(t[:, 0].mean()), 4), "sparse_attn_ms": round(float(t[:, 1].mean()), 4),
                           "J_best_median": float(np.median(dr[live, 1])),
                           "J_best_over_J_init_median": round(float(np.median(dr[live, 1] / dr[live, 0])), 4),
                           "stream_drift_rel_so_far": round((torch.linalg.vector_norm(r) /
                                                             torch.linalg.vector_norm(base)).item(), 5)})
        del q, k, v, gram, kc, ki, drift, o_s, o_d, ws, w_d, w_neg
    layer_ms = [x["select_ms"] + x["sparse_attn_ms"] for x in out_layers]
    return {"layers": out_layers, "ms_per_layer_mean": round(float(np.mean(layer_ms)), 4),
            "stack_ms": round(float(np.sum(layer_ms)), 3),
            "stream_drift_rel": out_layers[-1]["stream_drift_rel_so_far"],
            "host_generation_s": round(t_gen, 1)}


def rounds_sweep(ress, L, q, k, v, gram, stream, flush, rounds_list, n=10):
    """Config 3's sweep of the restoration rounds (the synthetic analogue of
    Fig. 7): selection time (caches flushed before each call) and the median
    J_best / J_init over rows that drop blocks, per R."""
    import torch

    out = []
    for R in rounds_list:
        drift = torch.empty((L.H, L.n_qb, 2), dtype=torch.float64, device=q.device)
        kc = torch.empty((L.H, L.n_qb), dtype=torch.int32, device=q.device)
        ki = torch.empty((L.H, L.n_qb, L.n_kb), dtype=torch.int32, device=q.device)

        def step(e=None):
            if e is not None:
                e[0].record(stream)
            ress.ress_select(q, k, v, gram, L.budgets, bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail,
                             rounds=R, kept_count=kc, kept_idx=ki, drift=drift, stream=stream)
            if e is not None:
                e[1].record(stream)
        step.n_events = 2
        step()
        t = timed_steps(step, n, stream, flush)[:, 0]
        dr = drift.cpu().numpy().reshape(-1, 2)
        live = dr[:, 0] > 0
        out.append({"rounds": R, "select_ms_mean": round(float(t.mean()), 4),
                    "select_ms_median": round(float(np.median(t)), 4),
                    "J_best_over_J_init_median": round(float(np.median(dr[live, 1] / dr[live, 0])), 4),
                    "J_best_over_J_init_mean": round(float(np.mean(dr[live, 1] / dr[live, 0])), 4)})
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: this build has no multi-GPU path "
              f"(--gpus {args.gpus} requested). Run with --gpus 1.", file=sys.stderr)
        return 2
    import torch

    import paper_2609_35593_amd as ress
    import synth

    if args.copy_calibration:
        copy_calibration()
        return 0

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    # Caches are flushed before every timed step by overwriting a 512 MB buffer
    # (larger than L2 and the 256 MB infinity cache), outside the timed events.
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    flush = None if args.no_flush else (lambda: scratch.fill_(1))

    if args.config == "16v_stack":
        t0 = time.perf_counter()
        res = stack_run(ress, args, torch, dev, stream, flush)
        wall = time.perf_counter() - t0
        out = {"metric": METRIC, "value": res["ms_per_layer_mean"], "unit": "ms/layer", "n_gpus": 1,
               "steps": 5, "warmup": 2, "ms_per_step": res["ms_per_layer_mean"], "higher_is_better": False,
               "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
               "config": {"workload": "16v_stack: 24 global-attention layers of 21,984 tokens (16 heads x 64), "
                                      "blocks 128, noise 0.3 -> 1.0, float32 residual stream of width 1024",
                          "sparsity_target": 0.75 if args.sparsity is None else args.sparsity,
                          "rounds": args.rounds},
               "stack": res, "wall_s": round(wall, 1)}
        print(json.dumps(out), flush=True)
        return 0

    t_gen = time.time()
    L = synth.make_config(args.config, sparsity=args.sparsity, bq=args.bq, bk=args.bk)
    q, k, v = (ress.bf16_from_bits(x, dev) for x in (L.q, L.k, L.v))
    gram = torch.from_numpy(L.gram).to(dev)
    gen_s = time.time() - t_gen
    n_qb, n_kb = L.n_qb, L.n_kb
    kc = torch.empty((L.H, n_qb), dtype=torch.int32, device=dev)
    ki = torch.empty((L.H, n_qb, n_kb), dtype=torch.int32, device=dev)
    drift = torch.empty((L.H, n_qb, 2), dtype=torch.float64, device=dev)
    o = torch.empty_like(q)
    ws = torch.empty(ress.ress_select_workspace_size(
        ress.make_shape(L.H, L.N, bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail)), dtype=torch.uint8, device=dev)

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        ress.ress_select(q, k, v, gram, L.budgets, bq=L.bq, bk=L.bk, n_special_tail=L.n_special_tail,
                         rounds=args.rounds, kept_count=kc, kept_idx=ki, drift=drift, workspace=ws, stream=stream)
        if ev is not None:
            ev[1].record(stream)
        ress.ress_sparse_attn(q, k, v, kc, ki, bq=L.bq, bk=L.bk, out=o, stream=stream)
        if ev is not None:
            ev[2].record(stream)
    step.n_events = 3

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # Timed region: exactly `steps` steps, synchronised on both sides; each step is
    # bracketed by HIP events on the launch stream, with the caches flushed before
    # it (outside the events). value = mean event time of a step.
    t0 = time.perf_counter()
    t_flush = timed_steps(step, args.steps, stream, flush)
    wall_incl_flush_ms = 1e3 * (time.perf_counter() - t0) / args.steps
    sel_ms, sp_ms = t_flush[:, 0], t_flush[:, 1]
    step_ms = sel_ms + sp_ms
    t_sel, t_sp = float(np.mean(sel_ms)), float(np.mean(sp_ms))
    value_ms = float(np.mean(step_ms))

    # Secondary: back-to-back steps without flushing (warm L2 / infinity cache).
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    warm_wall_ms = 1e3 * (time.perf_counter() - t0) / args.steps
    t_warm = timed_steps(step, args.steps, stream)
    warm = {"ms_per_step_wall": round(warm_wall_ms, 4), "select_ms_mean": round(float(t_warm[:, 0].mean()), 4),
            "sparse_attn_ms_mean": round(float(t_warm[:, 1].mean()), 4),
            "layer_ms_median": round(float(np.median(t_warm.sum(axis=1))), 4)}

    # Dense baseline of the same library, timed the same way (flushed).
    od = torch.empty_like(q)

    def dense_step(e=None):
        if e is not None:
            e[0].record(stream)
        ress.ress_dense_attn(q, k, v, bq=L.bq, bk=L.bk, out=od, stream=stream)
        if e is not None:
            e[1].record(stream)
    dense_step.n_events = 2
    dense_step()
    t_dense = float(timed_steps(dense_step, args.dense_steps, stream, flush)[:, 0].mean())
    t_dense_warm = float(timed_steps(dense_step, args.dense_steps, stream)[:, 0].mean())

    sweep = None
    if args.rounds_sweep:
        sweep = rounds_sweep(ress, L, q, k, v, gram, stream, flush, [int(x) for x in args.rounds_sweep.split(",")])
    ceilings = measured_ceilings(torch, dev)
    stats = input_stats(ress, L, q, k, v, gram, od, stream)
    criteria = None if args.no_criteria else criteria_report(ress, L, q, k, v, gram, od, stream)
    mask_rep = None if args.no_masking else masking_report(ress, L, q, k, v, gram, stream)
    neigh = None if args.no_neighbours else neighbours_report(ress, L, stream)

    kc_h, ki_h, dr = kc.cpu().numpy(), ki.cpu().numpy(), drift.cpu().numpy().reshape(-1, 2)
    sparsity_desc = (float(L.sparsity[0]) if np.all(L.sparsity == L.sparsity[0])
                     else f"per head in [{L.sparsity.min():.3f}, {L.sparsity.max():.3f}]")
    flops_kept, kept_tiles = kept_flops(L, kc_h, ki_h)
    flops_dense = 4.0 * L.D * L.H * float(L.N) * float(L.N)
    tf_kept = flops_kept / (t_sp * 1e-3) / 1e12
    tf_dense_eq = flops_dense / (value_ms * 1e-3) / 1e12
    sel_bytes = select_bytes(L)
    measured_sparsity = 1.0 - kept_tiles / float(L.H * n_qb * n_kb)
    ok = dr[:, 0] > 0
    # The committed counters cover the default workload only.
    default_workload = (args.config == "32v" and L.bq == 128 and L.bk == 128 and np.all(L.sparsity == 0.75)
                        and args.rounds == 5)
    traffic = traffic_from_profile() if default_workload else None

    out = {
        "metric": METRIC,
        "value": round(value_ms, 4),
        "unit": "ms/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(value_ms, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"{args.config}: one global-attention layer, {L.N} tokens "
                        f"({L.H} heads x {L.D}), blocks {L.bq}/{L.bk}, {n_qb}x{n_kb} blocks per head, "
                        f"target sparsity {sparsity_desc}, {args.rounds} restoration rounds",
            "tokens": L.N, "heads": L.H, "head_dim": L.D, "block_q": L.bq, "block_k": L.bk,
            "sparsity_target": sparsity_desc,
            "rounds": args.rounds, "select_dtype": "f64", "attention_dtype": "bf16 MFMA, f32 accumulate",
            "timing": "mean of per-step HIP events, L2 and infinity cache flushed before every step"
                      if flush is not None else "mean of per-step HIP events, back to back",
        },
        "roofline": {
            "kernel": f"attn_kernel<{L.bq},{L.bk},sparse> (ress_sparse_attn)",
            "bound": "mfma",
            "achieved": round(tf_kept, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(tf_kept / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic,
            "algorithmic_flops_per_launch": flops_kept,
            "launch_ms_mean": round(t_sp, 4),
        },
        "breakdown": {
            "select_ms": round(t_sel, 4),
            "sparse_attn_ms": round(t_sp, 4),
            "selection_overhead_frac": round(t_sel / (t_sel + t_sp), 4),
            "dense_attn_ms": round(t_dense, 4),
            "speedup_vs_dense": round(t_dense / value_ms, 3),
            "dense_tflops": round(flops_dense / (t_dense * 1e-3) / 1e12, 2),
            "dense_frac_peak": round(flops_dense / (t_dense * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "dense_equivalent_tflops": round(tf_dense_eq, 2),
            "kept_only_tflops": round(tf_kept, 2),
            "select_gbs": round(sel_bytes / (t_sel * 1e-3) / 1e9, 1),
            "select_frac_hbm": round(sel_bytes / (t_sel * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "measured_sparsity": round(measured_sparsity, 4),
            "J_best_over_J_init_median": round(float(np.median(dr[ok, 1] / dr[ok, 0])), 4) if ok.any() else None,
            "select_ms_median": round(float(np.median(sel_ms)), 4),
            "select_ms_p90": round(float(np.percentile(sel_ms, 90)), 4),
            "sparse_attn_ms_median": round(float(np.median(sp_ms)), 4),
            "sparse_attn_ms_p90": round(float(np.percentile(sp_ms, 90)), 4),
            "layer_ms_median": round(float(np.median(step_ms)), 4),
            "layer_ms_p90": round(float(np.percentile(step_ms, 90)), 4),
            "timed_region_wall_ms_per_step_incl_flush": round(wall_incl_flush_ms, 4),
            "warm_cache": warm,
            "dense_attn_ms_warm": round(t_dense_warm, 4),
            "speedup_vs_dense_warm": round(t_dense_warm / warm["layer_ms_median"], 3),
            "kept_only_frac_of_measured_gemm": round(tf_kept / ceilings["bf16_gemm_8192_tflops"], 4),
            "select_frac_of_measured_copy": round(sel_bytes / (t_sel * 1e-3) / 1e9 /
                                                  ceilings["copy_1gib_read_plus_write_gbs"], 4),
            "measured_ceilings": ceilings,
            "rounds_sweep": sweep,
            "criteria_same_budget": criteria,
            "single_block_masking": mask_rep,
            "fused_neighbours": neigh,
            "input_generation_s": round(gen_s, 1),
            "input_statistics": stats,
        },
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(L, args.rounds, kc_h, ki_h, args.cpu_seconds)
        out["cpu_baseline"]["gpu_speedup"] = round(out["cpu_baseline"]["value"] / value_ms, 1)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
