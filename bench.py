#!/usr/bin/env python3
"""Benchmark of the Ember step on one MI355X.

Workload (one "step"): the Ember update of the two untied token tables of a
model with a 128256-token vocabulary and width 4096, both bf16 with fp32
state: the LM head takes a dense step (gradient with Zipf(1.1) per-row
scales), the input embedding a sparse-row step (8 x 2048 Zipf(1.1) token ids
per step, ~4650 distinct rows).  All inputs are synthetic, made before the
timed region and resident in HBM.

By default both tables take their step in one ember_step_multi call (the
sparse table's one-launch step, then statistics, finalize and apply launches
of the dense table; the same bits as one call per table); --schedule
sequential times one call per table instead, and the line reports both.

Prints one JSON line: whole-step throughput in algorithmic GB/s (the bytes
the method must move, see paper_2607_01455_amd.workloads.algorithmic_bytes),
ms per step, the dense LM-head step and the sparse embedding step each with
its own ms, % of peak and kernel roofline, the roofline of the dominant
kernel (the dense apply pass, timed with HIP events around each launch),
torch's device copy and the library's streaming probe as reference rates,
the other table shapes, and the CPU oracle on every host thread and on one.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "Ember step ms + achieved HBM GB/s (% of peak) at V=128256, D=4096"
PEAK_GBPS = 8000.0
V, D = 128256, 4096
CSRC = os.path.join(ROOT, "paper_2607_01455_amd", "csrc")
# a traffic record holds for the kernel source and the launch header (tuning constants) it was taken on
KERNEL_SRC = (os.path.join(CSRC, "ember_kernels.hip"), os.path.join(CSRC, "ember_launch.h"))
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "ember_apply_lmhead128k_traffic.txt")
MULTI_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "ember_apply_multi_lmhead128k_embed128k_traffic.txt")
ROWONLY_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "ember_rowonly_lmhead128k_traffic.txt")
LMHEAD_SRC = (os.path.join(CSRC, "ember_lmhead.hip"), os.path.join(CSRC, "ember_launch.h"))
LMHEAD_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "ember_lmhead_grad_lmhead128k_wgrad_traffic.txt")
SPARSE_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "ember_sparse_onchip_embed128k_traffic.txt")
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-configs", action="store_true",
                   help="only time the oracle on every configuration (one thread and all threads) and print that")
    p.add_argument("--cpu-rows", type=int, default=32768, help="rows of the single-thread oracle sample")
    p.add_argument("--no-other-configs", action="store_true")
    p.add_argument("--no-row-only", action="store_true")
    p.add_argument("--no-coalesce", action="store_true")
    p.add_argument("--no-lmhead-wgrad", action="store_true")
    p.add_argument("--schedule", choices=("multi", "sequential"), default="multi",
                   help="multi: both tables in one ember_step_multi call; "
                        "sequential: ember_step_dense, then ember_step_sparse_rows")
    return p.parse_args()


def kernel_source_hash(src=KERNEL_SRC) -> str:
    """First 16 hex digits of the sha256 of the source files, concatenated."""
    h = hashlib.sha256()
    for path in ((src,) if isinstance(src, str) else src):
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_for_current_kernel(path=TRAFFIC_FILE, src=KERNEL_SRC):
    """HBM bytes per launch of the kernel a committed PMC summary covers, if
    it was taken on the current source of that kernel (else None)."""
    rec = {}
    try:
        with open(path) as f:
            for line in f:
                if "=" in line and not line.lstrip().startswith("#"):
                    k, v = line.split("=", 1)
                    rec[k.strip()] = v.strip()
    except OSError:
        return None
    if rec.get("kernel_source_sha256_16") != kernel_source_hash(src):
        return None
    try:
        return int(rec["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def stats_kept_bytes(V: int, D: int, g_size: int) -> int:
    """Bytes of G rows the statistics pass loads through the caches for the
    apply pass to find in the last-level cache (its kStatsKeepMB tail, read
    from the launch header), at most the whole of G."""
    import re
    with open(os.path.join(CSRC, "ember_launch.h")) as f:
        mb = int(re.search(r"constexpr int kStatsKeepMB = (\d+);", f.read()).group(1))
    row = D * g_size
    return min(V, int(mb * 1048576 // row)) * row


def traffic_rate(traffic, ms):
    """HBM GB/s from the PMC bytes per launch and the launch's average duration."""
    return None if traffic is None or not ms else round(traffic / (ms * 1e-3) / 1e9, 1)


def cpu_baseline(dev, rows_1t: int, steps: int = 2):
    """The oracle (float64 C, OpenMP over rows and column ranges) on the dense
    LM-head step: on every thread it is given (the whole 128256-row table) and
    on one thread (the first rows_1t rows), each for `steps` steps.  Inputs are
    made on the device (the same generators as the GPU timing) and copied to
    host memory before the oracle's timed calls."""
    import numpy as np
    import torch

    import oracle
    from paper_2607_01455_amd import workloads as wl

    def run(rows, threads):
        used = oracle.set_threads(threads)
        cfg = wl.Config("cpu_sample", rows, D, torch.bfloat16, torch.bfloat16, steps, "zipf_rows")
        W = wl.make_weights(cfg, seed=21, device=dev).contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        scales = (wl.zipf_probs(V, device=dev) * V).float()[:rows]
        r = np.zeros(rows, np.float32)
        c = np.zeros(D, np.float32)
        times = []
        for t in range(1, steps + 1):
            G = wl.make_dense_grad(cfg, t, seed=21, device=dev, scales=scales)
            G = G.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
            t0 = time.perf_counter()
            assert oracle.step(W, G, r, c, t) == 0
            times.append(time.perf_counter() - t0)
        sec = sum(times) / len(times)
        return used, sec, wl.algorithmic_bytes(rows, D, 2, 2) / sec / 1e9

    all_threads = oracle.set_threads(0)
    used, sec, gbps = run(V, all_threads)
    _, sec1, gbps1 = run(rows_1t, 1)
    oracle.set_threads(all_threads)
    return {"value": round(gbps, 4), "unit": "GB/s", "cores": used, "kind": "oracle",
            "sample": f"dense bf16 LM-head step, all {V} rows x {D}, {steps} steps, float64 C oracle on "
                      f"{used} threads: {sec * 1e3:.0f} ms/step",
            "single_thread": {"value": round(gbps1, 4), "unit": "GB/s", "cores": 1,
                              "sample": f"the first {rows_1t} of the {V} rows, {steps} steps: "
                                        f"{sec1 * 1e3:.0f} ms/step"}}


def cpu_configs(dev, budget_s: float = 10.0):
    """The oracle on every configuration (C1-C5 of the benchmark table): ms per
    step on every host thread it is given and on one thread, the first step
    from zero state.  On one thread a table whose step would take longer than
    about budget_s is timed on its first rows (stated in the output).  Inputs
    are the benchmark's generators, made on the device and copied to host
    memory before the timed calls."""
    import numpy as np
    import torch

    import oracle
    from paper_2607_01455_amd import workloads as wl

    def host(t):
        t = t.contiguous()
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).cpu().numpy().view(np.uint16)
        return t.cpu().numpy()

    def timed(fn, min_s=0.2):
        n, t0 = 0, time.perf_counter()
        while True:
            fn()
            n += 1
            el = time.perf_counter() - t0
            if el >= min_s or n >= 50:
                return el / n * 1e3

    all_threads = oracle.set_threads(0)
    out = {"threads": all_threads}
    for key, name in (("C1", "tiny"), ("C2", "lmhead32k"), ("C3", "lmhead128k"), ("C4", "embed128k"),
                      ("C5a", "tied152k"), ("C5b", "wide262k")):
        cfg = wl.CONFIGS[name]
        W = host(wl.make_weights(cfg, seed=51, device=dev))
        V_, D_ = W.shape
        if key == "C4":
            idx_d, G_d = wl.make_sparse_batch(cfg, 1, seed=51, device=dev)
            idx, G = idx_d.cpu().numpy(), host(G_d)
            n = int(idx.shape[0])
            nbytes = wl.algorithmic_bytes(V_, D_, W.itemsize, G.itemsize, rows=n)
        else:
            G = host(wl.make_dense_grad(cfg, 1, seed=51, device=dev, scales=wl.row_scales(cfg, 51, dev)))
            idx, n = None, V_
            nbytes = wl.algorithmic_bytes(V_, D_, W.itemsize, G.itemsize)

        def run(rows=None):
            Wc = W if rows is None else W[:rows]
            Gc = G if rows is None or idx is not None else G[:rows]
            r = np.zeros(Wc.shape[0], np.float32)
            c = np.zeros(D_, np.float32)
            return lambda: oracle.step(Wc.copy() if Wc.size < (1 << 22) else Wc, Gc, r, c, 1, idx=idx)

        oracle.set_threads(all_threads)
        ms_all = timed(run())
        oracle.set_threads(1)
        t0 = time.perf_counter()
        run(min(V_, 4096) if idx is None else None)()
        probe_ms = (time.perf_counter() - t0) * 1e3
        est_full = probe_ms * (V_ / min(V_, 4096) if idx is None else 1.0)
        rows_1t = V_ if est_full <= budget_s * 1e3 or idx is not None else max(4096, int(V_ * budget_s * 1e3 / est_full))
        ms_1t = timed(run(None if rows_1t == V_ else rows_1t), min_s=0.0)
        out[key] = {"config": name, "V": V_, "D": D_, "rows_with_gradient": n,
                    "ms_all_threads": round(ms_all, 3), "GBps_all_threads": round(nbytes / (ms_all * 1e-3) / 1e9, 4),
                    "ms_one_thread": round(ms_1t, 3), "one_thread_rows": rows_1t,
                    "ms_one_thread_whole_table": round(ms_1t * V_ / rows_1t, 1)}
        print(f"cpu oracle {key} {name}: {out[key]}", file=sys.stderr, flush=True)
        del W, G
    oracle.set_threads(all_threads)
    return out


def other_configs(ember, wl, torch, dev, K):
    """ms/step and algorithmic GB/s of the dense configurations other than the
    headline one, each timed over K steps after 2 warm-up steps."""
    out = {}
    for name in ("tiny", "lmhead32k", "tied152k", "wide262k"):
        cfg = wl.CONFIGS[name]
        W = wl.make_weights(cfg, seed=41, device=dev)
        sc = wl.row_scales(cfg, 41, dev)
        grads = [wl.make_dense_grad(cfg, t + 1, seed=41, device=dev, scales=sc) for t in range(2)]
        tab = ember.EmberTable(cfg.V, cfg.D, device=dev)
        for k in range(2):
            tab.step(W, grads[k % 2])
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for k in range(K):
            tab.step(W, grads[k % 2])
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / K
        ws, gs = W.element_size(), grads[0].element_size()
        nbytes = wl.algorithmic_bytes(cfg.V, cfg.D, ws, gs)
        out[name] = {"V": cfg.V, "D": cfg.D, "dtype_w": str(cfg.w_dtype).replace("torch.", ""),
                     "ms": round(ms, 4), "GBps": round(nbytes / (ms * 1e-3) / 1e9, 1),
                     "pct_of_peak": round(100.0 * nbytes / (ms * 1e-3) / 1e9 / PEAK_GBPS, 2)}
        del W, grads, tab
        torch.cuda.empty_cache()
    return out


def row_only_section(ember, wl, torch, dev, K, Wm, W_head, W_emb, grads, batches):
    """The same two-table workload with row-only Ember (Section 2.1; state V,
    one fused pass per table): whole-step time (both tables in one multi-table
    call, and one call per table), per-table medians and kernel averages, in
    row-only algorithmic bytes."""
    stream = torch.cuda.current_stream()
    head = ember.EmberTable(V, D, device=dev, row_only=True)
    emb = ember.EmberTable(V, D, device=dev, row_only=True)
    n_grads = len(grads)

    def step_sequential(k):
        head.step(W_head, grads[k % n_grads])
        idx, Gr = batches[k]
        emb.step_sparse_rows(W_emb, Gr, idx)

    def step_multi(k):
        idx, Gr = batches[k]
        ember.step_tables([(head, W_head, grads[k % n_grads]), (emb, W_emb, Gr, idx)])

    def whole_steps(fn):
        for k in range(Wm):
            fn(k)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for k in range(K):
            fn(Wm + k)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / K

    seq_ms = whole_steps(step_sequential)
    ms_step = whole_steps(step_multi)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]
    for k in range(K):
        ev[k][0].record(stream)
        head.step(W_head, grads[(Wm + k) % n_grads])
        ev[k][1].record(stream)
        idx, Gr = batches[Wm + k]
        emb.step_sparse_rows(W_emb, Gr, idx)
        ev[k][2].record(stream)
    torch.cuda.synchronize()
    dense_ms = sorted(e[0].elapsed_time(e[1]) for e in ev)[K // 2]
    sparse_ms = sorted(e[1].elapsed_time(e[2]) for e in ev)[K // 2]
    def profiled(fn):
        ember.ember_profile_enable(True)
        for k in range(K):
            fn(k)
        torch.cuda.synchronize()
        ember.ember_profile_enable(False)
        return ember.ember_profile_collect()

    dstats = profiled(lambda k: head.step(W_head, grads[(Wm + k) % n_grads]))
    sstats = profiled(lambda k: emb.step_sparse_rows(W_emb, batches[Wm + k][1], batches[Wm + k][0]))
    if ember.ember_get_error(emb.ws) != ember.EMBER_OK:
        raise RuntimeError("row-only sparse step reported an index error")
    fused_launches, fused_ms = dstats["ember_rowonly"]
    fused_avg_ms = fused_ms / fused_launches
    dense_bytes = wl.rowonly_algorithmic_bytes(V, D, 2, 2)
    n_rows = [int(b[0].numel()) for b in batches[Wm:Wm + K]]
    sparse_bytes = sum(wl.rowonly_algorithmic_bytes(V, D, 2, 2, rows=n) for n in n_rows) / K
    gbps = (dense_bytes + sparse_bytes) / (ms_step * 1e-3) / 1e9
    fused_gbps = dense_bytes / (fused_avg_ms * 1e-3) / 1e9
    return {
        "ms_per_step": round(ms_step, 4),
        "GBps": round(gbps, 1),
        "pct_of_peak": round(100.0 * gbps / PEAK_GBPS, 2),
        "schedules_ms_per_step": {"multi": round(ms_step, 4), "sequential": round(seq_ms, 4)},
        "algorithmic_bytes_per_step": int(dense_bytes + sparse_bytes),
        "dense_lmhead": {"ms": round(dense_ms, 4), "bytes": dense_bytes,
                         "GBps": round(dense_bytes / (dense_ms * 1e-3) / 1e9, 1),
                         "pct_of_peak": round(100.0 * dense_bytes / (dense_ms * 1e-3) / 1e9 / PEAK_GBPS, 2)},
        "sparse_embedding": {"ms": round(sparse_ms, 4), "bytes": int(sparse_bytes)},
        "kernels_ms_avg": {
            "dense": {k: round(v[1] / v[0], 5) for k, v in dstats.items()},
            "sparse": {k: round(v[1] / v[0], 5) for k, v in sstats.items()},
        },
        "roofline": {"kernel": "ember_rowonly (dense LM-head step)", "bound": "hbm",
                     "achieved": round(fused_gbps, 1), "peak": PEAK_GBPS, "unit": "GB/s",
                     "frac": round(fused_gbps / PEAK_GBPS, 4),
                     "traffic": traffic_for_current_kernel(ROWONLY_TRAFFIC_FILE),
                     "traffic_GBps": traffic_rate(traffic_for_current_kernel(ROWONLY_TRAFFIC_FILE),
                                                  fused_avg_ms),
                     "avg_launch_ms": round(fused_avg_ms, 5),
                     "algorithmic_bytes_per_launch": dense_bytes},
    }


def coalesce_section(ember, wl, torch, dev, K, Wm):
    """Coalescing of the embedding batch (8 x 2048 token ids, one 4096-wide bf16
    signal row per position) into distinct ids and summed rows: time per call
    with inputs resident (no host read of n inside the timed region), and the
    whole tokens -> sparse step path, with n read on the host each step or left
    on the device (the step then takes its form from n on the device)."""
    cfg = wl.CONFIGS["embed128k"]
    P, V_, D_ = cfg.batch_tokens, cfg.V, cfg.D
    nb = 4
    batches = [wl.make_token_batch(cfg, t + 1, seed=33, device=dev) for t in range(nb)]
    co = ember.Coalescer(P, V_, D_, device=dev)
    ns = []
    for tok, U in batches:
        idx, G = co(tok, U)
        ns.append(int(idx.numel()))
    stream = torch.cuda.current_stream()
    for k in range(Wm):
        tok, U = batches[k % nb]
        ember.ember_coalesce_rows(tok, U, V_, co.idx, co.G_rows, co.n_out, co.ws)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for k in range(K):
        tok, U = batches[k % nb]
        ember.ember_coalesce_rows(tok, U, V_, co.idx, co.G_rows, co.n_out, co.ws)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / K
    if ember.ember_get_error(co.ws) != ember.EMBER_OK:
        raise RuntimeError("coalescing reported an index error")
    n_avg = sum(ns[k % nb] for k in range(K)) / K
    nbytes = sum(wl.coalesce_bytes(P, ns[k % nb], D_, 2, 2) for k in range(K)) / K
    # tokens -> coalesce -> sparse step, n read on the host every step
    W_emb = wl.make_weights(cfg, seed=34, device=dev)
    emb = ember.EmberTable(V_, D_, device=dev)
    for k in range(Wm):
        tok, U = batches[k % nb]
        idx, G = co(tok, U)
        emb.step_sparse_rows(W_emb, G, idx)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(K):
        tok, U = batches[k % nb]
        idx, G = co(tok, U)
        emb.step_sparse_rows(W_emb, G, idx)
    torch.cuda.synchronize()
    e2e_ms = (time.perf_counter() - t0) * 1e3 / K
    # the same path with the count left on the device: nothing read back
    for k in range(Wm):
        tok, U = batches[k % nb]
        emb.step_tokens(W_emb, tok, U, co)
    torch.cuda.synchronize()
    e0.record(stream)
    for k in range(K):
        tok, U = batches[k % nb]
        emb.step_tokens(W_emb, tok, U, co)
    e1.record(stream)
    torch.cuda.synchronize()
    devn_ms = e0.elapsed_time(e1) / K
    if ember.ember_get_error(emb.ws) != ember.EMBER_OK or ember.ember_get_error(co.ws) != ember.EMBER_OK:
        raise RuntimeError("tokens -> step with a device count reported an error")
    gbps = nbytes / (ms * 1e-3) / 1e9
    return {"workload": f"embed128k batch: {P} token ids over V={V_}, D={D_} bf16 signal rows, "
                        f"{n_avg:.0f} distinct ids on average",
            "ms": round(ms, 4), "bytes": int(nbytes), "GBps": round(gbps, 1),
            "pct_of_peak": round(100.0 * gbps / PEAK_GBPS, 2),
            "tokens_to_sparse_step_ms": round(e2e_ms, 4),
            "tokens_to_sparse_step_device_count_ms": round(devn_ms, 4)}


def lmhead_wgrad_section(ember, wl, torch, dev, K, Wm):
    """The LM-head step with the statistics fused into the weight-gradient GEMM
    (ember_lmhead_step): G = dY^T H for 8 x 2048 tokens (logits gradient
    16384 x 128256 and hidden states 16384 x 4096, bf16) and the Ember step on
    the 128256 x 4096 bf16 head, against the same work done as a library GEMM
    (torch.matmul) followed by the two-pass dense step.  The GEMM kernel is
    timed with HIP events around each launch: MFMA roofline at the bf16 peak."""
    cfg = wl.CONFIGS["lmhead128k_wgrad"]
    V_, D_, T = cfg.V, cfg.D, cfg.batch_tokens
    batches = [wl.make_lmhead_batch(cfg, t + 1, seed=35, device=dev) for t in range(2)]
    W = wl.make_weights(cfg, seed=35, device=dev)
    G = torch.empty(V_, D_, dtype=torch.bfloat16, device=dev)
    tab = ember.EmberTable(V_, D_, device=dev)
    stream = torch.cuda.current_stream(dev)

    def fused(k):
        dY, H = batches[k % 2]
        tab.step_lmhead(W, dY, H, G)

    def unfused(k):
        dY, H = batches[k % 2]
        torch.matmul(dY.t(), H, out=G)
        tab.step(W, G)

    def timed(fn, n):
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for k in range(n):
            fn(k)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    for k in range(Wm):
        fused(k)
        unfused(k)
    fused_ms = timed(fused, K)
    unfused_ms = timed(unfused, K)
    gemm_ms = timed(lambda k: torch.matmul(batches[k % 2][0].t(), batches[k % 2][1], out=G), K)
    ember.ember_profile_enable(True)
    timed(fused, K)
    ember.ember_profile_enable(False)
    st = ember.ember_profile_collect()
    n, tot = st["ember_lmhead_grad"]
    k_ms = tot / n
    flops = wl.lmhead_flops(T, V_, D_)
    tflops = flops / (k_ms * 1e-3) / 1e12
    del batches, W, G, tab
    torch.cuda.empty_cache()
    return {"workload": f"lmhead128k_wgrad: G = dY^T H for T={T} tokens, V={V_}, D={D_} bf16, then the "
                        "Ember step on the bf16 head",
            "fused_step_ms": round(fused_ms, 4),
            "library_gemm_plus_two_pass_step_ms": round(unfused_ms, 4),
            "library_gemm_ms": round(gemm_ms, 4),
            "speedup_vs_library_path": round(unfused_ms / fused_ms, 4),
            "kernels_ms_avg": {k: round(v[1] / v[0], 4) for k, v in st.items()},
            "roofline": {"kernel": "ember_lmhead_grad (GEMM + statistics epilogue)", "bound": "mfma",
                         "achieved": round(tflops, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(tflops / PEAK_BF16_TFLOPS, 4),
                         "traffic": traffic_for_current_kernel(LMHEAD_TRAFFIC_FILE, LMHEAD_SRC),
                         "traffic_GBps": traffic_rate(
                             traffic_for_current_kernel(LMHEAD_TRAFFIC_FILE, LMHEAD_SRC), k_ms),
                         "avg_launch_ms": round(k_ms, 4), "flops_per_launch": flops}}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the Ember step here runs on a single MI355X "
              "(no sharding or collectives are built); run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2607_01455_amd import ember
    from paper_2607_01455_amd import workloads as wl

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.cpu_configs:
        print(json.dumps({"cpu_oracle_configs": cpu_configs(dev)}), flush=True)
        return
    K, Wm = args.steps, args.warmup
    head_cfg = wl.CONFIGS["lmhead128k"]
    emb_cfg = wl.CONFIGS["embed128k"]

    # --- inputs, resident before timing -----------------------------------
    W_head = wl.make_weights(head_cfg, seed=31, device=dev)
    W_emb = wl.make_weights(emb_cfg, seed=32, device=dev)
    scales = wl.row_scales(head_cfg, 31, dev)
    n_grads = 4  # distinct dense gradients, reused round-robin (1 GiB each)
    grads = [wl.make_dense_grad(head_cfg, t + 1, seed=31, device=dev, scales=scales) for t in range(n_grads)]
    batches = [wl.make_sparse_batch(emb_cfg, t + 1, seed=32, device=dev) for t in range(K + Wm)]
    head = ember.EmberTable(V, D, device=dev)
    emb = ember.EmberTable(V, D, device=dev)
    torch.cuda.synchronize()

    def step_sequential(k):
        head.step(W_head, grads[k % n_grads])
        idx, Gr = batches[k]
        emb.step_sparse_rows(W_emb, Gr, idx)

    def step_multi(k):
        idx, Gr = batches[k]
        ember.step_tables([(head, W_head, grads[k % n_grads]), (emb, W_emb, Gr, idx)])

    schedules = {"multi": step_multi, "sequential": step_sequential}
    step = schedules[args.schedule]
    other = "sequential" if args.schedule == "multi" else "multi"
    # warm-up of both schedules (the clocks settle over the first milliseconds)
    for fn in (step, schedules[other]):
        for k in range(Wm):
            fn(k)
    torch.cuda.synchronize()
    if ember.ember_get_error(emb.ws) != ember.EMBER_OK:
        raise RuntimeError("sparse step reported an index error")

    stream = torch.cuda.current_stream()

    # --- timed region A: K whole steps, nothing else on the stream -----------
    def whole_steps(fn):
        torch.cuda.synchronize()
        t_start = torch.cuda.Event(enable_timing=True)
        t_end = torch.cuda.Event(enable_timing=True)
        t_start.record(stream)
        for k in range(K):
            fn(Wm + k)
        t_end.record(stream)
        torch.cuda.synchronize()
        return t_start.elapsed_time(t_end) / K

    # the other schedule on the same inputs, for comparison (not the value); then
    # the timed schedule, right after warm-up steps of its own
    other_ms = whole_steps(schedules[other])
    for k in range(Wm):
        step(k)
    ms_step = whole_steps(step)
    schedule_ms = {args.schedule: round(ms_step, 4), other: round(other_ms, 4)}

    # --- timed region A1: the same steps with a marker between the two tables
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]
    torch.cuda.synchronize()
    for k in range(K):
        ev[k][0].record(stream)
        head.step(W_head, grads[(Wm + k) % n_grads])
        ev[k][1].record(stream)
        idx, Gr = batches[Wm + k]
        emb.step_sparse_rows(W_emb, Gr, idx)
        ev[k][2].record(stream)
    torch.cuda.synchronize()
    dense_ms = sorted(e[0].elapsed_time(e[1]) for e in ev)[K // 2]
    sparse_ms = sorted(e[1].elapsed_time(e[2]) for e in ev)[K // 2]
    if ember.ember_get_error(emb.ws) != ember.EMBER_OK:
        raise RuntimeError("sparse step reported an index error")

    # --- timed region A2: each table's step alone, K steps back to back -------
    # (no marker between steps; the sparse table's hot rows may still sit in
    # the last-level cache from the step before, which region A1 rules out)
    dense_alone_ms = whole_steps(lambda k: head.step(W_head, grads[k % n_grads]))
    sparse_alone_ms = whole_steps(lambda k: emb.step_sparse_rows(W_emb, batches[k][1], batches[k][0]))
    if ember.ember_get_error(emb.ws) != ember.EMBER_OK:
        raise RuntimeError("sparse step reported an index error")

    dense_bytes = wl.algorithmic_bytes(V, D, 2, 2)
    n_rows = [int(b[0].numel()) for b in batches[Wm:Wm + K]]
    sparse_bytes = [wl.algorithmic_bytes(V, D, 2, 2, rows=n) for n in n_rows]
    step_bytes = dense_bytes + sum(sparse_bytes) / K
    value = step_bytes / (ms_step * 1e-3) / 1e9

    # --- timed region B: dense steps with HIP events around every kernel ------
    def kernel_region(fn):
        ember.ember_profile_enable(True)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for k in range(K):
            fn(k)
        e1.record(stream)
        torch.cuda.synchronize()
        ember.ember_profile_enable(False)
        return ember.ember_profile_collect(), e0.elapsed_time(e1) / K

    dstats, dense_ms_events = kernel_region(lambda k: head.step(W_head, grads[(Wm + K + k) % n_grads]))
    sstats, sparse_ms_events = kernel_region(lambda k: emb.step_sparse_rows(W_emb, batches[Wm + k][1], batches[Wm + k][0]))
    mstats, multi_ms_events = kernel_region(lambda k: step_multi(Wm + k))
    if ember.ember_get_error(emb.ws) != ember.EMBER_OK:
        raise RuntimeError("sparse step reported an index error")
    apply_launches, apply_ms = dstats["ember_apply"]
    apply_avg_ms = apply_ms / apply_launches
    # apply pass: G read, W read and written, r and the column factors read
    apply_bytes = V * D * (2 + 2 * 2) + 4 * (V + D)
    apply_gbps = apply_bytes / (apply_avg_ms * 1e-3) / 1e9
    # the dense table's apply launch of the multi-table call (the sparse table
    # takes its one-launch step in the same call)
    mapply_launches, mapply_ms = mstats["ember_apply_multi"]
    mapply_avg_ms = mapply_ms / mapply_launches
    mapply_gbps = apply_bytes / (mapply_avg_ms * 1e-3) / 1e9
    kept_bytes = stats_kept_bytes(V, D, 2)
    dense_roofline = {
        "kernel": "ember_apply (dense LM-head step, apply pass)",
        "bound": "hbm",
        "achieved": round(apply_gbps, 1),
        "peak": PEAK_GBPS,
        "unit": "GB/s",
        "frac": round(apply_gbps / PEAK_GBPS, 4),
        "traffic": traffic_for_current_kernel(),
        "traffic_GBps": traffic_rate(traffic_for_current_kernel(), apply_avg_ms),
        "avg_launch_ms": round(apply_avg_ms, 5),
        "algorithmic_bytes_per_launch": apply_bytes,
        # achieved/frac count every algorithmic byte as HBM traffic; the G rows
        # the statistics pass leaves in the last-level cache are read from it
        # (no counter separates them), so the HBM-only estimate subtracts them
        "llc_kept_bytes": kept_bytes,
        "hbm_bytes_est": apply_bytes - kept_bytes,
        "hbm_GBps_est": round((apply_bytes - kept_bytes) / (apply_avg_ms * 1e-3) / 1e9, 1),
        "hbm_frac_est": round((apply_bytes - kept_bytes) / (apply_avg_ms * 1e-3) / 1e9 / PEAK_GBPS, 4),
    }
    multi_roofline = {
        "kernel": "ember_apply_multi (dense LM-head table's apply pass inside the two-table call)",
        "bound": "hbm",
        "achieved": round(mapply_gbps, 1),
        "peak": PEAK_GBPS,
        "unit": "GB/s",
        "frac": round(mapply_gbps / PEAK_GBPS, 4),
        "traffic": traffic_for_current_kernel(MULTI_TRAFFIC_FILE),
        "traffic_GBps": traffic_rate(traffic_for_current_kernel(MULTI_TRAFFIC_FILE), mapply_avg_ms),
        "avg_launch_ms": round(mapply_avg_ms, 5),
        "algorithmic_bytes_per_launch": apply_bytes,
        "llc_kept_bytes": kept_bytes,
        "hbm_bytes_est": apply_bytes - kept_bytes,
        "hbm_GBps_est": round((apply_bytes - kept_bytes) / (mapply_avg_ms * 1e-3) / 1e9, 1),
        "hbm_frac_est": round((apply_bytes - kept_bytes) / (mapply_avg_ms * 1e-3) / 1e9 / PEAK_GBPS, 4),
    }
    # the sparse step's one launch: algorithmic bytes as the method counts them
    # (G read twice, W rows read and written, r read and written, ids); the
    # launch keeps its gradient rows in registers and reads them once, so it
    # moves one G read less (bytes_moved_min)
    sparse_launches, sparse_k_ms = sstats["ember_sparse_onchip"]
    sparse_avg_ms = sparse_k_ms / sparse_launches
    sparse_step_bytes = sum(sparse_bytes) / K
    sparse_min_bytes = sum(wl.algorithmic_bytes(V, D, 2, 2, rows=n) - n * D * 2 for n in n_rows) / K
    sparse_gbps = sparse_step_bytes / (sparse_avg_ms * 1e-3) / 1e9
    sparse_roofline = {
        "kernel": "ember_sparse_onchip (whole sparse step, one launch)",
        "bound": "hbm",
        "achieved": round(sparse_gbps, 1),
        "peak": PEAK_GBPS,
        "unit": "GB/s",
        "frac": round(sparse_gbps / PEAK_GBPS, 4),
        "traffic": traffic_for_current_kernel(SPARSE_TRAFFIC_FILE),
        "traffic_GBps": traffic_rate(traffic_for_current_kernel(SPARSE_TRAFFIC_FILE), sparse_avg_ms),
        "avg_launch_ms": round(sparse_avg_ms, 5),
        "algorithmic_bytes_per_launch": int(sparse_step_bytes),
        "bytes_moved_min": int(sparse_min_bytes),
        "bytes_moved_min_GBps": round(sparse_min_bytes / (sparse_avg_ms * 1e-3) / 1e9, 1),
    }

    # --- plain device copy over a W-sized buffer: practical ceiling ----------
    src = torch.empty(V * D, dtype=torch.bfloat16, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    c0 = torch.cuda.Event(enable_timing=True)
    c1 = torch.cuda.Event(enable_timing=True)
    c0.record(stream)
    for _ in range(10):
        dst.copy_(src)
    c1.record(stream)
    torch.cuda.synchronize()
    copy_gbps = 2 * src.numel() * 2 / (c0.elapsed_time(c1) / 10 * 1e-3) / 1e9
    # the library's streaming probe over the same bytes: rates of a plain
    # grid-stride read, copy and two reads + one write (reference points, not
    # ceilings: the apply pass, with several rows in flight per wavefront and
    # part of G in the last-level cache, runs faster than the third)
    src2 = torch.empty_like(src).fill_(2.0)
    ceilings = {}
    for mode, name, ops in ((0, "read", 1), (1, "copy", 2), (2, "two_reads_one_write", 3)):
        for _ in range(2):
            ember.ember_stream_probe(mode, dst, src, src2)
        c0.record(stream)
        for _ in range(10):
            ember.ember_stream_probe(mode, dst, src, src2)
        c1.record(stream)
        torch.cuda.synchronize()
        ceilings[name] = round(ops * src.numel() * 2 / (c0.elapsed_time(c1) / 10 * 1e-3) / 1e9, 1)
    del src, src2, dst

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wm,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "storage": "bf16 W and G, fp32 r and c",
        "data": "synthetic",
        "config": {
            "workload": "Ember step of both untied token tables, V=128256 x D=4096: "
                        "LM head dense (Zipf(1.1) row-scaled gradient) + input embedding "
                        "sparse rows (8x2048 Zipf(1.1) ids per step)",
            "V": V, "D": D, "storage": "bf16 W and G, fp32 r and c",
            "sparse_rows_per_step": round(sum(n_rows) / K, 1),
            "algorithmic_bytes_per_step": int(step_bytes),
            "schedule": ("both tables in one ember_step_multi call: statistics, finalize and apply "
                         "launches shared by the two tables, one stream" if args.schedule == "multi"
                         else "dense step then sparse step, one stream"),
        },
        "schedules_ms_per_step": schedule_ms,
        "pct_of_peak": round(100.0 * value / PEAK_GBPS, 2),
        "parts": {
            "dense_lmhead": {"workload": "LM head 128256 x 4096 bf16, dense step (three launches)",
                             "ms": round(dense_ms, 4), "bytes": dense_bytes,
                             "ms_back_to_back": round(dense_alone_ms, 4),
                             "GBps": round(dense_bytes / (dense_ms * 1e-3) / 1e9, 1),
                             "pct_of_peak": round(100.0 * dense_bytes / (dense_ms * 1e-3) / 1e9 / PEAK_GBPS, 2),
                             "roofline": dense_roofline},
            "sparse_embedding": {"workload": "input embedding 128256 x 4096 bf16, sparse-row step of an "
                                             "8 x 2048-token Zipf(1.1) batch (one launch)",
                                 "ms": round(sparse_ms, 4), "bytes": int(sparse_step_bytes),
                                 "ms_back_to_back": round(sparse_alone_ms, 4),
                                 "pct_of_peak_back_to_back": round(100.0 * sparse_step_bytes / (sparse_alone_ms * 1e-3)
                                                                   / 1e9 / PEAK_GBPS, 2),
                                 "GBps": round(sparse_step_bytes / (sparse_ms * 1e-3) / 1e9, 1),
                                 "pct_of_peak": round(100.0 * sparse_step_bytes / (sparse_ms * 1e-3) / 1e9
                                                      / PEAK_GBPS, 2),
                                 "rows_per_step": round(sum(n_rows) / K, 1),
                                 "roofline": sparse_roofline},
        },
        "kernels_ms_avg": {
            "dense": {k: round(v[1] / v[0], 5) for k, v in dstats.items()},
            "sparse": {k: round(v[1] / v[0], 5) for k, v in sstats.items()},
            "multi": {k: round(v[1] / v[0], 5) for k, v in mstats.items()},
        },
        "ms_with_kernel_events": {"dense": round(dense_ms_events, 4), "sparse": round(sparse_ms_events, 4),
                                  "multi": round(multi_ms_events, 4)},
        "roofline": multi_roofline if args.schedule == "multi" else dense_roofline,
        "torch_device_copy_GBps": round(copy_gbps, 1),
        "stream_probe_GBps": ceilings,
        "row_only": None,
        "coalesce": None,
        "lmhead_wgrad": None,
        "other_configs": None,
        "cpu_baseline": None,
    }
    del head, emb
    if not args.no_row_only:
        out["row_only"] = row_only_section(ember, wl, torch, dev, K, Wm, W_head, W_emb, grads, batches)
    if not args.no_coalesce:
        out["coalesce"] = coalesce_section(ember, wl, torch, dev, K, Wm)
    if not args.no_other_configs or not args.no_lmhead_wgrad:
        del W_head, W_emb, grads, batches
        torch.cuda.empty_cache()
    if not args.no_lmhead_wgrad:
        out["lmhead_wgrad"] = lmhead_wgrad_section(ember, wl, torch, dev, K, Wm)
    if not args.no_other_configs:
        out["other_configs"] = other_configs(ember, wl, torch, dev, K)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(dev, args.cpu_rows)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
