#!/usr/bin/env python3
"""Benchmark of the CLSA decode step on one MI355X.

One step = one clsa_decode_step call: the indexer over every cached token, one
top-k, then L sparse-attention layers that share the index set.  Workload (by
default): batch 4, 131072-token contexts, top-k 2048, 32 query / 8 KV heads of
128, 16 layers, 64 planted aligned index keys per sequence; synthetic seeded
bf16 inputs.

Prints ONE JSON line: metric, value (us per decode step), the roofline of the
kernel with the largest share of the step (the sparse-attention kernel, one
launch per layer) and of the indexer, each timed with HIP events recorded by
the library on its own stream, and the CPU oracle timed on a bounded sample of
the same workload.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "CLSA decode-step µs + HBM GB/s (index+top-k+L sparse attn), 128K ctx"
KD_METRIC = ("CLSA distillation step ms (Eq. 5 multi-layer target + Eq. 6 KL loss and indexer "
             "gradient), 32K-token sequence")
HBM_PEAK_GBPS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0   # dense bf16 matrix-core peak
# exp2 on the vector units: 256 CUs x 4 SIMDs x 8 lanes per clock (v_exp_f32 at
# half the FMA rate) x 2.4 GHz
EXP_PEAK_TPS = 256 * 4 * 8 * 2.4e9 / 1e12
PREFILL_MIN_ROWS = 32            # query rows per sequence from which the indexer uses MFMA


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def valid_keys_per_row(w, x):
    """Valid keys of every query row (causal rows stop at their position)."""
    lens = np.asarray(w.lens, dtype=np.int64)[:, None].repeat(w.n_q, axis=1)
    if x.get("q_pos") is not None:
        lens = np.minimum(lens, np.maximum(x["q_pos"].astype(np.int64) + 1, 0))
    return lens


def algorithmic_bytes(w, x):
    """Bytes the step must move at least once: index keys read + scores written,
    the selected K/V rows (for decode each row's once; for many query rows the
    logical gather of every row), per-layer queries and outputs, the index set."""
    n = valid_keys_per_row(w, x)
    toks = sum(w.lens)
    index_keys = toks * w.idx_heads * w.idx_dim * 2
    scores = int(n.sum()) * 4
    sel = int(np.minimum(n, w.top_k).sum())
    kv_rows = sel * w.kv_heads * w.head_dim * 2 * 2
    qo = w.n_layers * w.batch * w.n_q * w.q_heads * w.head_dim * 2 * 2
    idx = w.batch * w.n_q * w.top_k * 4
    # one sparse-attention launch: the selected K/V rows of every row, its query
    # and its index list (the output leaves through the split merge)
    attn = kv_rows + w.batch * w.n_q * (w.q_heads * w.head_dim * 2 + w.top_k * 4)
    # matrix FLOPs of one attention launch: q.k and the weighted V, 2 x 2 x head_dim
    # per (row, query head, selected token)
    attn_flops = sel * w.q_heads * w.head_dim * 4
    return dict(index=index_keys + scores, step=index_keys + scores + kv_rows + qo + idx,
                kv_rows=kv_rows, attn=attn, attn_flops=attn_flops,
                index_flops=2 * w.idx_heads * w.idx_dim * int(n.sum()))


KERNEL_SOURCES = {
    "kd_lse_kernel": ["kd.hip", "device_common.h", "clsa_internal.h"],
    "kd_target_kernel": ["kd.hip", "device_common.h", "clsa_internal.h"],
    "sparse_attn_kernel": ["sparse_attn.hip", "device_common.h", "clsa_internal.h"],
    "index_decode_kernel": ["index_decode.hip", "device_common.h", "clsa_internal.h"],
    "index_prefill_kernel": ["index_prefill.hip", "device_common.h", "clsa_internal.h"],
    "index_emit_kernel": ["index_prefill.hip", "device_common.h", "clsa_internal.h"],
}


def source_digest(kernel: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2606_06467_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_bytes(kernel: str, workload: str):
    """HBM bytes per launch from the recorded FETCH_SIZE / WRITE_SIZE counters,
    or None when there is no record for this kernel and workload or the
    kernel's sources have changed since the counters were taken."""
    import glob
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        with open(path) as fh:
            for line in fh:
                if not line.startswith("traffic_record "):
                    continue
                rec = json.loads(line[len("traffic_record "):])
                if rec["kernel"] == kernel and rec["workload"] == workload:
                    if rec["source_digest"] != source_digest(kernel):
                        return None
                    return int(rec["bytes_per_launch"])
    return None


def roofline_mfma(kernel: str, w, flops: int, ms: float):
    achieved = flops / (ms * 1e-3) / 1e12
    return {"bound": "mfma", "kernel": kernel, "achieved": round(achieved, 1),
            "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4),
            "traffic": traffic_bytes(kernel, w.name), "algorithmic_flops_per_launch": flops,
            "avg_launch_us": round(ms * 1e3, 2)}


def roofline(kernel: str, w, alg_bytes: int, ms: float):
    achieved = alg_bytes / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "kernel": kernel, "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": traffic_bytes(kernel, w.name), "algorithmic_bytes_per_launch": alg_bytes,
            "avg_launch_us": round(ms * 1e3, 2)}


def host_cpu():
    """(threads for the oracle, CPUs this process may run on, CPU model name).

    The oracle uses one thread per CPU available to the process, or
    OMP_NUM_THREADS when that is set lower (the GPU machines set it to the
    host-core share of one GPU)."""
    try:
        avail = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        avail = os.cpu_count() or 1
    threads = avail
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        threads = min(threads, int(env))
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return threads, avail, model


def cpu_baseline(w, x, budget_s: float):
    """Time the CPU oracle on the same workload, repeating whole steps until
    ``budget_s`` seconds have passed (at least one).  With many query rows per
    sequence (chunked prefill) a whole step would take the oracle far longer;
    it then runs the step for the first 16 query rows of each sequence (same
    caches, same layers) and the time is scaled to all rows, and labelled so."""
    import dataclasses
    import oracle as orc
    ws, xs, scale = w, x, 1.0
    if w.n_q > 16:
        ws = dataclasses.replace(w, n_q=16)
        xs = dict(x, q_idx=np.ascontiguousarray(x["q_idx"][:, :16]),
                  q_layers=np.ascontiguousarray(x["q_layers"][:, :, :16]),
                  q_pos=None if x["q_pos"] is None else np.ascontiguousarray(x["q_pos"][:, :16]))
        scale = w.n_q / 16
    sh = orc.shape_of(ws)
    threads, avail, model = host_cpu()
    orc.set_threads(threads)
    try:
        reps, t0 = 0, time.perf_counter()
        while True:
            orc.decode_step(sh, xs["q_idx"], xs["k_idx"], xs["k_cache"], xs["v_cache"],
                            xs["seq_lens"], xs["q_layers"], xs["q_pos"], xs["page_table"])
            reps += 1
            el = time.perf_counter() - t0
            if el >= budget_s or el / reps * (reps + 1) > 3 * budget_s:
                break
    finally:
        orc.set_threads(1)
    us = el / reps * 1e6 * scale
    how = f"C oracle on {threads} host thread(s)"
    if scale == 1.0:
        sample = f"{reps} full step(s) of {w.name} (B={w.batch}, L={w.n_layers}), {how}, {el:.1f} s"
    else:
        sample = (f"{reps} step(s) over the first 16 of {w.n_q} query rows of {w.name} "
                  f"(L={w.n_layers}), {how}, {el:.1f} s; scaled x{scale:g} "
                  f"to all rows (extrapolated)")
    return {"value": round(us, 1), "unit": "us/step", "cores": threads, "kind": "oracle",
            "sample": sample, "host_cpus_available": avail, "cpu_model": model}


def cold_read_reference(dev, stream, n_bytes: int, reps: int = 7):
    """What one launch reading ``n_bytes`` from HBM cold achieves on this GPU:
    the library's decode indexer (a coalesced 16-byte streaming read of index
    keys, 1 FLOP per byte) over a key set of ``n_bytes``, timed with events
    around the launch exactly as the attention layers are, each time after a
    2 GiB read that evicts the 256 MB Infinity Cache.  Median of ``reps``."""
    import torch
    from paper_2606_06467_amd import binding as B
    batch = 4
    n = max(64, n_bytes // (batch * 512))
    sh = B.make_shape(batch=batch, n_q=1, max_len=n, top_k=64)
    q = torch.zeros((batch, 1, 4, 64), dtype=torch.bfloat16, device=dev)
    k = torch.ones((batch, n, 4, 64), dtype=torch.bfloat16, device=dev)
    lens = torch.full((batch,), n, dtype=torch.int32, device=dev)
    scores = torch.empty((batch, 1, n), dtype=torch.float32, device=dev)
    flush = torch.ones(2 << 30, dtype=torch.uint8, device=dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t = []
    for r in range(reps + 1):
        flush.sum(dtype=torch.int32)
        e0.record(stream)
        B.clsa_index_scores(sh, q, k, None, lens, None, scores, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        if r:
            t.append(e0.elapsed_time(e1))
    us = float(np.median(t)) * 1e3
    read = batch * n * 512
    del q, k, lens, scores, flush
    return {"kernel": "index_decode_kernel", "bytes": read, "us": round(us, 2),
            "achieved_GBps": round(read / (us * 1e-6) / 1e9, 1),
            "frac_of_hbm_peak": round(read / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
            "note": "one launch streaming this many bytes cold (Infinity Cache evicted), "
                    "timed between events like the attention layers"}


def copy_reference(mib: int, dev) -> None:
    """Three plain device-to-device copies of ``mib`` MiB: a known-size
    reference for the hardware byte counters."""
    import torch
    n = mib << 20
    src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def kd_counts(w, x):
    """Work of one distillation step: (row, key) pairs, the logit flops of one
    pass over every (layer, query head, pair) (the statistics and the target
    pass each make one), the exponentials of one such pass, and the index
    scores and gradient products of the loss."""
    n = valid_keys_per_row(w, x)
    pairs = int(n.sum())
    lh = w.n_layers * w.q_heads
    d_idx = w.idx_heads * w.idx_dim
    return dict(pairs=pairs, logit_flops=2 * w.head_dim * pairs * lh, exps=pairs * lh,
                index_flops=2 * d_idx * pairs, grad_flops=2 * 2 * d_idx * pairs)


def kd_cpu_baseline(w, x, budget_s: float):
    """The oracle's Eq. 5 target and Eq. 6 loss on the last rows of the sequence
    (the longest causal rows; same caches and layers), as many rows as fit the
    budget, scaled to the whole sequence by the ratio of (row, key) pairs."""
    import dataclasses
    import oracle as orc

    def run(rows):
        t0 = w.n_q - rows
        ws = dataclasses.replace(w, n_q=rows, q_pos0=[int(x["q_pos"][b, t0]) for b in range(w.batch)])
        sh = orc.shape_of(ws)
        ql = np.ascontiguousarray(x["q_layers"][:, :, t0:])
        qi = np.ascontiguousarray(x["q_idx"][:, t0:])
        qp = np.ascontiguousarray(x["q_pos"][:, t0:])
        t = time.perf_counter()
        abar = orc.kd_target(sh, ql, x["k_cache"], x["seq_lens"], qp, x["page_table"], fill=0.0)
        orc.kd_loss(sh, abar, qi, x["k_idx"], x["seq_lens"], qp, x["page_table"])
        el = time.perf_counter() - t
        pairs = int(valid_keys_per_row(ws, {"q_pos": qp}).sum())
        return el, pairs

    threads, avail, model = host_cpu()
    orc.set_threads(threads)
    try:
        el, pairs = run(threads)
        rows = threads
        more = int(budget_s / max(el, 1e-6)) * threads
        if more >= 2 * threads:
            rows = min(more, w.n_q)
            el, pairs = run(rows)
    finally:
        orc.set_threads(1)
    scale = kd_counts(w, x)["pairs"] / pairs
    return {"value": round(el * scale * 1e3, 1), "unit": "ms/step", "cores": threads,
            "kind": "oracle", "host_cpus_available": avail, "cpu_model": model,
            "sample": (f"Eq. 5 target + Eq. 6 loss and gradient of the oracle over the last "
                       f"{rows} of {w.n_q} rows of {w.name} (L={w.n_layers}, {pairs} row-key "
                       f"pairs), C oracle with the target on {threads} host thread(s) (the "
                       f"loss's sums across rows on one), {el:.1f} s; scaled x{scale:.4g} by "
                       f"row-key pairs to the whole sequence (extrapolated)")}


def run_kd(args, w) -> int:
    """The training-side distillation step on one sequence: clsa_kd_target (the
    Eq. 5 target averaged over every layer and query head) and clsa_kd_loss (the
    indexer scores, the Eq. 6 KL loss and the gradients of the index queries and
    keys), timed over K steps after W warm-up steps, then once more with the
    library's phase events for the per-kernel times."""
    import torch
    from paper_2606_06467_amd import binding as B
    from paper_2606_06467_amd import inputs
    log(f"[kd] generating {w.name} ...")
    t = time.time()
    x = inputs.make_inputs(w)
    log(f"[kd] inputs ready in {time.time() - t:.1f} s")
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    bf = lambda a: B.bf16_from_bits(a, dev)
    ql, kc = bf(x["q_layers"]), bf(x["k_cache"])
    qi, ki = bf(x["q_idx"]), bf(x["k_idx"])
    seq_lens = torch.from_numpy(x["seq_lens"]).to(dev)
    q_pos = torch.from_numpy(x["q_pos"]).to(dev)
    pt = None if x["page_table"] is None else torch.from_numpy(x["page_table"]).to(dev)
    sh = B.make_shape(batch=w.batch, n_q=w.n_q, max_len=w.max_len, top_k=w.top_k,
                      q_heads=w.q_heads, kv_heads=w.kv_heads, page_size=w.page_size,
                      max_pages=w.max_pages, causal=w.causal)
    L = w.n_layers
    abar = torch.empty((w.batch, w.n_q, w.max_len), dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    dq = torch.empty(x["q_idx"].shape, dtype=torch.float32, device=dev)
    dk = torch.empty(x["k_idx"].shape, dtype=torch.float32, device=dev)
    ws_t = B.workspace(sh, B.CLSA_OP_KD_TARGET, L, dev)
    ws_l = B.workspace(sh, B.CLSA_OP_KD_LOSS, 0, dev)
    stream = torch.cuda.current_stream(dev)

    def target():
        B.clsa_kd_target(sh, L, ql, kc, pt, seq_lens, q_pos, abar, ws_t, stream)

    def kd_loss():
        B.clsa_kd_loss(sh, abar, qi, ki, pt, seq_lens, q_pos, loss, dq, dk, ws_l, stream)

    log(f"[kd] warmup {args.warmup} ...")
    for _ in range(args.warmup):
        target()
        kd_loss()
    torch.cuda.synchronize()
    # ---- timed region: exactly K steps ----
    log(f"[kd] timing {args.steps} steps ...")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        target()
        kd_loss()
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) * 1e3 / args.steps
    # ---- per-kernel times from the library's phase events (a separate pass) ----
    ev = B.HipEvents(8 * args.steps, timing_only=True)
    for i in range(args.steps):
        B.clsa_set_phase_events(ev.handles[8 * i: 8 * i + 4])
        target()
        B.clsa_set_phase_events(ev.handles[8 * i + 4: 8 * i + 8])
        kd_loss()
    B.clsa_set_phase_events(None)
    torch.cuda.synchronize()
    ph = np.array([[ev.elapsed_ms(8 * i, 8 * i + 1), ev.elapsed_ms(8 * i + 1, 8 * i + 2),
                    ev.elapsed_ms(8 * i + 4, 8 * i + 5), ev.elapsed_ms(8 * i + 5, 8 * i + 6),
                    ev.elapsed_ms(8 * i + 6, 8 * i + 7)] for i in range(args.steps)])
    ev.close()
    lse_ms, tgt_ms, scores_ms, rows_ms, grad_ms = (float(v) for v in ph.mean(axis=0))
    # ---- the same step when the caller passes the dense forward pass's
    # log-sum-exps (a training step has them): the statistics pass is skipped.
    # Timed with stand-in values of the right size, ln(t + 1) + 1/2 (the target
    # pass does the same work whatever they are). ----
    lse_fwd = (torch.log(torch.arange(1, w.n_q + 1, device=dev, dtype=torch.float32)) + 0.5)
    lse_fwd = lse_fwd.view(1, 1, w.n_q, 1).expand(L, w.batch, w.n_q, w.q_heads).contiguous()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        B.clsa_kd_target(sh, L, ql, kc, pt, seq_lens, q_pos, abar, ws_t, stream,
                         lse_layers=lse_fwd)
        kd_loss()
    torch.cuda.synchronize()
    ms_fwd_lse = (time.perf_counter() - t0) * 1e3 / args.steps
    del lse_fwd
    if args.copy_mib > 0:
        copy_reference(args.copy_mib, dev)
    cnt = kd_counts(w, x)
    kern = {"kd_lse_kernel": lse_ms, "kd_target_kernel": tgt_ms}
    main_k = max(kern, key=kern.get)
    other_k = min(kern, key=kern.get)
    exp_rate = cnt["exps"] / (lse_ms * 1e-3) / 1e12
    res = {
        "metric": KD_METRIC,
        "value": round(ms_per_step, 3),
        "unit": "ms/step",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "tokens": w.n_q, "context": max(w.lens),
                   "causal": w.causal, "layers": L, "q_heads": w.q_heads,
                   "kv_heads": w.kv_heads, "head_dim": w.head_dim,
                   "index_dim": w.idx_heads * w.idx_dim, "row_key_pairs": cnt["pairs"]},
        "tokens_per_s": round(w.batch * w.n_q / (ms_per_step * 1e-3), 1),
        "ms_per_step_with_forward_lse": round(ms_fwd_lse, 3),
        "phases_ms": {"statistics_kernel": round(lse_ms, 3), "target_kernel": round(tgt_ms, 3),
                      "index_scores": round(scores_ms, 3), "loss_rows": round(rows_ms, 3),
                      "gradients": round(grad_ms, 3)},
        # the kernel with the largest share: both target-pass kernels make one
        # logit product over every (layer, head, row, key)
        "roofline": roofline_mfma(main_k, w, cnt["logit_flops"], kern[main_k]),
        "roofline_other": roofline_mfma(other_k, w, cnt["logit_flops"], kern[other_k]),
        "exp_rate": {"kernel": "kd_lse_kernel", "achieved": round(exp_rate, 2),
                     "peak": round(EXP_PEAK_TPS, 2), "unit": "Texp/s",
                     "frac": round(exp_rate / EXP_PEAK_TPS, 4),
                     "note": "one exp2 per (layer, head, row, key) at least"},
    }
    if args.cpu_budget > 0:
        log("[kd] CPU oracle baseline ...")
        res["cpu_baseline"] = kd_cpu_baseline(w, x, args.cpu_budget)
    print(json.dumps(res), flush=True)
    return 0


def run_schedules(args, w) -> int:
    """Per-layer decode cost of routing schedules on one workload.

    * shared: one index pass + one top-k, every layer reuses the set (the
      method's schedule, clsa_decode_step);
    * every 4 / every layer: the set is recomputed every 4 layers / before
      every layer (clsa_decode_step_grouped), each set from its own copy of the
      index keys (so that every index pass reads HBM like a distinct indexer);
    * dense: every layer attends over all valid keys (clsa_dense_attn).
    Each is timed over K steps after W warm-up steps."""
    import torch
    from paper_2606_06467_amd import binding as B
    from paper_2606_06467_amd import inputs
    log(f"[schedules] generating {w.name} ...")
    x = inputs.make_inputs(w)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    bf = lambda a: B.bf16_from_bits(a, dev)
    q_idx, k_idx = bf(x["q_idx"]), bf(x["k_idx"])
    kc, vc, ql = bf(x["k_cache"]), bf(x["v_cache"]), bf(x["q_layers"])
    seq_lens = torch.from_numpy(x["seq_lens"]).to(dev)
    q_pos = None if x["q_pos"] is None else torch.from_numpy(x["q_pos"]).to(dev)
    pt = None if x["page_table"] is None else torch.from_numpy(x["page_table"]).to(dev)
    sh = B.make_shape(batch=w.batch, n_q=w.n_q, max_len=w.max_len, top_k=w.top_k,
                      q_heads=w.q_heads, kv_heads=w.kv_heads, page_size=w.page_size,
                      max_pages=w.max_pages, causal=w.causal)
    L = w.n_layers
    out = torch.empty((L, w.batch, w.n_q, w.q_heads, w.head_dim), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((L, w.batch, w.n_q, w.q_heads), dtype=torch.float32, device=dev)
    ws = B.workspace(sh, B.CLSA_OP_DECODE, L, dev)
    wsd = B.workspace(sh, B.CLSA_OP_DENSE, 0, dev)

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        t = time.perf_counter()
        for _ in range(args.steps):
            fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t) * 1e6 / args.steps

    res = {}
    for name, group in (("shared", L), ("every 4 layers", 4), ("every layer", 1)):
        n_sets = max(1, -(-L // group))
        qi = q_idx.unsqueeze(0).repeat(n_sets, *([1] * q_idx.dim())).contiguous()
        ki = k_idx.unsqueeze(0).repeat(n_sets, *([1] * k_idx.dim())).contiguous()
        idx = torch.empty((n_sets, w.batch, w.n_q, w.top_k), dtype=torch.int32, device=dev)
        ns = torch.empty((n_sets, w.batch, w.n_q), dtype=torch.int32, device=dev)
        fn = lambda: B.clsa_decode_step_grouped(sh, qi, q_idx.numel(), ki, k_idx.numel(), kc, vc,
                                                pt, seq_lens, q_pos, group, ql, out, lse, idx, ns,
                                                ws)
        log(f"[schedules] {name} ...")
        us = timed(fn)
        res[name] = {"index_sets": n_sets, "step_us": round(us, 2),
                     "per_layer_us": round(us / L, 2)}
        del qi, ki
    log("[schedules] dense ...")

    def dense_step():
        for l in range(L):
            B.clsa_dense_attn(sh, ql[l], kc, vc, pt, seq_lens, q_pos, out[l], lse[l], wsd)
    us = timed(dense_step)
    res["dense"] = {"step_us": round(us, 2), "per_layer_us": round(us / L, 2)}
    print(json.dumps({"metric": "per-layer decode cost by routing schedule", "unit": "us",
                      "workload": w.name, "layers": L, "steps": args.steps,
                      "warmup": args.warmup, "schedules": res}), flush=True)
    return 0


def run_project(args) -> int:
    """Eq. 2 for a chunk of new tokens (the projections of the index query and key
    and the shared K / V, written into the caches): 8192 rows of d_model 2560 on a
    131072-token cache, 32 query / 8 KV heads (2560 output features), synthetic
    bf16 activations and weights."""
    import torch
    from paper_2606_06467_amd import binding as B
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    rows, d_model, max_len, kv_heads = 8192, 2560, 131072, 8
    n_feat = 512 + 2 * kv_heads * 128
    g = torch.Generator(device=dev)
    g.manual_seed(2606)
    h = torch.randn((rows, d_model), generator=g, device=dev).to(torch.bfloat16)
    wt = (torch.randn((n_feat, d_model), generator=g, device=dev) * 0.02).to(torch.bfloat16)
    pos = (max_len - rows + torch.arange(rows, device=dev)).to(torch.int32)
    q_idx = torch.empty((rows, 256), dtype=torch.bfloat16, device=dev)
    k_idx = torch.zeros((1, max_len, 256), dtype=torch.bfloat16, device=dev)
    kc = torch.zeros((1, max_len, kv_heads * 128), dtype=torch.bfloat16, device=dev)
    vc = torch.zeros_like(kc)
    sh = B.make_shape(batch=1, n_q=rows, max_len=max_len, top_k=2048, q_heads=32,
                      kv_heads=kv_heads, causal=True)

    def call():
        B.clsa_project_append(sh, d_model, h, wt, pos, None, q_idx, k_idx, kc, vc)
    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        call()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    flops = 2 * rows * n_feat * d_model
    tf = flops / (ms * 1e-3) / 1e12
    print(json.dumps({"metric": "Eq. 2 projection + cache append, 8192 new tokens", "value": round(ms * 1e3, 2),
                      "unit": "us/call", "steps": args.steps, "warmup": args.warmup,
                      "higher_is_better": False, "dtype": "bf16", "data": "synthetic",
                      "config": {"rows": rows, "d_model": d_model, "features": n_feat, "context": max_len},
                      "roofline": {"bound": "mfma", "kernel": "project_gemm_kernel", "achieved": round(tf, 1),
                                   "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                                   "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4),
                                   "algorithmic_flops_per_launch": flops}}), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="decode_b4_n128k_planted")
    ap.add_argument("--cpu-budget", type=float, default=12.0,
                    help="seconds of oracle time for the CPU baseline (0 = skip)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after the timed steps, run plain device-to-device copies of this "
                         "many MiB (a known-size reference for hardware byte counters)")
    ap.add_argument("--graph", action="store_true",
                    help="also time the step captured in a HIP graph and replayed "
                         "(graph_us_per_step; one cache copy)")
    ap.add_argument("--kd", action="store_true",
                    help="instead of the decode step, time the training-side distillation step "
                         "(Eq. 5 target, Eq. 6 loss and indexer gradient) on the 32K-token "
                         "sequence workload (one JSON line)")
    ap.add_argument("--project", action="store_true",
                    help="instead of the decode step, time the Eq. 2 projection with its cache "
                         "writes (clsa_project_append) for a chunk of 8192 new tokens at "
                         "d_model 2560 (one JSON line)")
    ap.add_argument("--top-k", type=int, default=0,
                    help="run the workload with this top_k instead of its own (the workload "
                         "name gets a _k<K> suffix); e.g. index sets whose rows fit the L2")
    ap.add_argument("--schedules", action="store_true",
                    help="instead of the step benchmark, compare routing schedules on the "
                         "workload: one shared index set, a fresh set every 4 layers, a fresh "
                         "set every layer, and dense attention (one JSON line)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU; the decode path "
                                   "shards by sequence with no communication, so --gpus N>1 "
                                   "is not measured here"}))
        return 2

    import torch
    from paper_2606_06467_amd import binding as B
    from paper_2606_06467_amd import inputs

    if args.kd:
        wl = args.workload if args.workload in inputs.KD_WORKLOADS else inputs.KD_WORKLOADS[0]
        return run_kd(args, inputs.workload(wl))
    if args.project:
        return run_project(args)
    w = inputs.workload(args.workload)
    if args.top_k > 0:
        w = dataclasses.replace(w, name=f"{w.name}_k{args.top_k}", top_k=args.top_k)
    if args.schedules:
        return run_schedules(args, w)
    if w.n_q != 1:
        log("note: chunked-prefill workload timed through the decode-step entry point")
    log(f"[bench] generating {w.name} ...")
    t = time.time()
    x = inputs.make_inputs(w)
    log(f"[bench] inputs ready in {time.time() - t:.1f} s")
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    def bf(a):
        return B.bf16_from_bits(a, dev)

    # Several copies of the caches so that consecutive steps read different HBM
    # (no cache reuse across steps: each step starts cold like a new batch).
    per_copy = x["k_idx"].nbytes + x["k_cache"].nbytes + x["v_cache"].nbytes
    copies = int(min(16, max(2, math.ceil(768e6 / per_copy))))
    caches = []
    for c in range(copies):
        caches.append((bf(x["k_idx"]), bf(x["k_cache"]), bf(x["v_cache"])))
    q_idx = bf(x["q_idx"])
    q_layers = bf(x["q_layers"])
    seq_lens = torch.from_numpy(x["seq_lens"]).to(dev)
    q_pos = None if x["q_pos"] is None else torch.from_numpy(x["q_pos"]).to(dev)
    pt = None if x["page_table"] is None else torch.from_numpy(x["page_table"]).to(dev)
    sh = B.make_shape(batch=w.batch, n_q=w.n_q, max_len=w.max_len, top_k=w.top_k,
                      q_heads=w.q_heads, kv_heads=w.kv_heads, page_size=w.page_size,
                      max_pages=w.max_pages, causal=w.causal)
    L = w.n_layers
    out = torch.empty((L, w.batch, w.n_q, w.q_heads, w.head_dim), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((L, w.batch, w.n_q, w.q_heads), dtype=torch.float32, device=dev)
    idx = torch.empty((w.batch, w.n_q, w.top_k), dtype=torch.int32, device=dev)
    ns = torch.empty((w.batch, w.n_q), dtype=torch.int32, device=dev)
    ws = B.workspace(sh, B.CLSA_OP_DECODE, L, dev)
    stream = torch.cuda.current_stream(dev)

    def step(i):
        ki, kc, vc = caches[i % copies]
        B.clsa_decode_step(sh, q_idx, ki, kc, vc, pt, seq_lens, q_pos, q_layers, out, lse, idx,
                           ns, ws, stream)

    log(f"[bench] {copies} cache copies, warmup {args.warmup} ...")
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # ---- timed region: exactly K steps ----
    log(f"[bench] timing {args.steps} steps ...")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps

    # ---- events recorded by the library on its own stream, in two more passes
    # of K steps (events add ~1.5 us each, so they stay out of the timed region):
    # (a) the four phase marks only; (b) the phase marks plus a pair around
    # every layer's sparse-attention kernel, for that kernel's launch time ----
    def event_pass(per_layer: bool):
        ne = 4 + (2 * L if per_layer else 0)
        ev = B.HipEvents(ne * args.steps, timing_only=True)
        torch.cuda.synchronize()
        t = time.perf_counter()
        for i in range(args.steps):
            B.clsa_set_phase_events(ev.handles[ne * i: ne * (i + 1)])
            step(i)
        B.clsa_set_phase_events(None)
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t) * 1e3 / args.steps
        ph = np.array([[ev.elapsed_ms(ne * i + a, ne * i + a + 1) for a in range(3)] +
                       [ev.elapsed_ms(ne * i, ne * i + 3)] for i in range(args.steps)])
        attn = (np.array([[ev.elapsed_ms(ne * i + 4 + 2 * l, ne * i + 5 + 2 * l)
                           for l in range(L)] for i in range(args.steps)])
                if per_layer else None)
        ev.close()
        return wall, ph, attn

    _, ph, _ = event_pass(False)
    ms_per_step_events, ph_layers, attn = event_pass(True)
    index_ms, topk_ms, layers_ms = (float(v) for v in ph[:, :3].mean(axis=0))
    step_pct = np.percentile(ph[:, 3], [10, 50, 90]) * 1e3  # per step, from the phase pass

    graph_us = None
    if args.graph:
        # the same step captured in a HIP graph (one cache copy), replayed K times
        g = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            ki, kc, vc = caches[0]
            B.clsa_decode_step(sh, q_idx, ki, kc, vc, pt, seq_lens, q_pos, q_layers, out, lse,
                               idx, ns, ws)
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        t = time.perf_counter()
        for _ in range(args.steps):
            g.replay()
        torch.cuda.synchronize()
        graph_us = (time.perf_counter() - t) * 1e6 / args.steps
        del g
    attn_ms = float(attn.mean())
    attn_first_ms = float(attn[:, 0].mean())
    attn_warm_ms = float(attn[:, 1:].mean()) if L > 1 else attn_first_ms
    prefill = w.n_q >= PREFILL_MIN_ROWS
    cold_ref = None if prefill else cold_read_reference(dev, stream, algorithmic_bytes(w, x)["attn"])

    if args.copy_mib > 0:
        copy_reference(args.copy_mib, dev)

    ab = algorithmic_bytes(w, x)
    step_us = ms_per_step * 1e3
    res = {
        "metric": METRIC,
        "value": round(step_us, 2),
        "unit": "us/step",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "ms_per_step_with_layer_events": round(ms_per_step_events, 5),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "query_rows": w.n_q, "context": max(w.lens),
                   "top_k": w.top_k, "layers": L, "q_heads": w.q_heads, "kv_heads": w.kv_heads,
                   "head_dim": w.head_dim, "index_dim": w.idx_heads * w.idx_dim,
                   "paged": bool(w.page_size), "planted": w.planted},
        "tokens_per_s": round(w.batch * w.n_q / (ms_per_step * 1e-3), 1),
        "hbm_GBps": round(ab["step"] / (ms_per_step * 1e-3) / 1e9, 1),
        "step_us_p10_p50_p90": [round(float(v), 2) for v in step_pct],
        "phases_us": {"index": round(index_ms * 1e3, 2), "topk": round(topk_ms * 1e3, 2),
                      "layers": round(layers_ms * 1e3, 2),
                      "per_layer": round(layers_ms * 1e3 / max(L, 1), 2),
                      "attn_kernel": round(attn_ms * 1e3, 2),
                      "attn_kernel_first_layer": round(attn_first_ms * 1e3, 2)},
        # the kernel with the largest share of the step: the sparse-attention
        # kernel, launched once per layer.  Decode: bound by reading its rows
        # (HBM for the first layer after the top-k, the caches after); chunked
        # prefill: most of its 68.7 GB of logical gathers per layer are served by
        # the caches, so it is priced by its matrix FLOPs
        "roofline": (roofline_mfma("sparse_attn_kernel", w, ab["attn_flops"], attn_ms)
                     if prefill else roofline("sparse_attn_kernel", w, ab["attn"], attn_ms)),
        # chunked prefill: the index phase (sampled pass, threshold, candidate
        # pass) priced by the causal block's FLOPs; its traffic record is the
        # candidate pass's, the phase's largest kernel
        "roofline_index": (roofline_mfma("index_emit_kernel", w, ab["index_flops"], index_ms)
                           if w.n_q >= PREFILL_MIN_ROWS else
                           roofline("index_decode_kernel", w, ab["index"], index_ms)),
    }
    if prefill:
        res["roofline"]["logical_gather_bytes_per_launch"] = ab["attn"]
    else:
        cold = roofline("sparse_attn_kernel", w, ab["attn"], attn_first_ms)
        cold["frac_of_cold_read_reference"] = round(cold_ref["us"] / (attn_first_ms * 1e3), 4)
        res["roofline_cold_layer"] = cold
        res["roofline_warm_layers"] = roofline("sparse_attn_kernel", w, ab["attn"], attn_warm_ms)
        res["cold_read_reference"] = cold_ref
    if graph_us is not None:
        res["graph_us_per_step"] = round(graph_us, 2)
    if args.cpu_budget > 0:
        log("[bench] CPU oracle baseline ...")
        res["cpu_baseline"] = cpu_baseline(w, x, args.cpu_budget)
    print(json.dumps(res), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
