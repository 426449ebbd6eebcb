"""Benchmark: block-sparse video self-attention on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                    [--no-cpu-baseline] [--no-dense] [--cpu-seconds S] [--all-workloads]

One step = the whole sparse path on one synthetic layer already resident in
HBM: block pooling -> block selection -> sparse attention (the dense fallback
is timed separately as the speedup denominator).  Prints one JSON line.

value        kept-block attention FLOPs / step time (pool + select + attend)
roofline     the sparse-attention kernel alone: kept FLOPs per launch / mean
             launch time (HIP events on the stream the kernel runs on),
             against the bf16 dense MFMA peak; traffic = HBM bytes per launch
             from the committed rocprofv3 counter record while the kernel
             sources still match it (else null)
cpu_baseline the float64 oracle on the host cores, timed before the GPU is
             touched: one forked worker per core (at most 16), one BLAS
             thread each, each on its own head (pooling and selection of every
             query block, then as many query blocks' attention as fit the time
             budget); kept FLOPs / wall seconds, in the same unit, with a
             labelled extrapolation to the whole layer
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "effective TFLOP/s of sparse attention (kept blocks) + % bf16 MFMA peak"
BF16_PEAK_TFLOPS = 2516.6   # 256 CU x 2.4 GHz x 4096 dense bf16 flop/clk/CU
FP8_PEAK_TFLOPS = 5033.2   # dense fp8 MFMA: twice the bf16 rate
HBM_PEAK_GBS = 8000.0


TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "attention_traffic_large_64b.json")


def measured_traffic(workload: str):
    """HBM bytes per sparse-attention launch from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE record, or None when the record is for another
    workload or the kernel sources changed since it was taken."""
    import hashlib
    try:
        with open(TRAFFIC_RECORD) as f:
            rec = json.load(f)
        if rec.get("workload") != workload:
            return None
        h = hashlib.sha256()
        for rel in rec["sources"]:
            with open(os.path.join(ROOT, rel), "rb") as f:
                h.update(f.read())
        if h.hexdigest() != rec["sources_sha256"]:
            return None
        return int(rec["hbm_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def kept_flops(idx: np.ndarray, cnt: np.ndarray, N: int, S: int, D: int):
    """(valid-token FLOPs, full-block FLOPs, kept pairs): 4*D*n_i*n_j per kept
    (query block i, key block j) pair; n = valid tokens of the block."""
    nb = cnt.shape[-1]
    ntok = np.full(nb + 1, S, dtype=np.int64)
    ntok[nb - 1] = N - (nb - 1) * S
    ntok[nb] = 0
    kmax = idx.shape[-1]
    col = np.arange(kmax)[None, None, None, :]
    live = col < cnt[..., None]
    j = np.where(live & (idx >= 0) & (idx < nb), idx, nb)
    kept_tok = ntok[j].sum(axis=-1)                  # [B, H, nB]
    flops = 4 * D * float((ntok[None, None, :nb] * kept_tok).sum())
    pairs = int(cnt.sum())
    return flops, 4.0 * D * S * S * pairs, pairs


_CPU_BITS = None     # the workload's inputs, inherited by the forked baseline workers


def _cpu_head(task):
    """One baseline worker: head (b, h) of the workload with one BLAS thread:
    float64 pooling, scores and selection over all query blocks, then
    block-sparse attention on query blocks in a seeded random order until the
    time budget is spent."""
    import oracle
    from threadpoolctl import threadpool_limits

    wl, b, h, budget_s = task
    with threadpool_limits(1):
        t0 = time.perf_counter()
        f = {n: oracle.bf16_bits_to_f64(_CPU_BITS[n][b, h]) for n in ("q", "k", "v")}
        c = 1.0 / np.sqrt(wl.head_dim)
        s = oracle.block_scores(oracle.pool_blocks(f["q"], wl.block), oracle.pool_blocks(f["k"], wl.block), c)
        nb = s.shape[-1]
        if wl.mode == "mass":
            forced = (oracle.first_frame_blocks(wl.grid_h, wl.grid_w, wl.block, nb)
                      if wl.force_first_frame else [])
            kept = oracle.select_cummass(s, wl.mass_threshold,
                                         oracle.mass_cap(nb, wl.max_keep_ratio, len(forced)), forced)
        else:
            kept = oracle.select_topk(s, oracle.topk_count(nb, wl.keep_ratio, wl.topk))
        t_select = time.perf_counter() - t0
        q4, k4, v4 = (f[n][None, None] for n in ("q", "k", "v"))
        ntok = [min(wl.block, wl.seq_len - i * wl.block) for i in range(nb)]
        flops, done = 0.0, 0
        t1 = time.perf_counter()
        for i in np.random.default_rng(1000 * b + h).permutation(nb):
            oracle.block_sparse_attention(q4, k4, v4, [[kept]], wl.block, c, rows=[(0, 0, int(i))])
            flops += 4.0 * wl.head_dim * ntok[i] * sum(ntok[j] for j in kept[i])
            done += 1
            if time.perf_counter() - t1 > budget_s:
                break
        return {"flops": flops, "select_s": t_select, "attn_s": time.perf_counter() - t1, "blocks": done,
                "n_blocks": nb}


def cpu_baseline(wl, bits, budget_s: float):
    """Time the oracle on the host cores: one forked worker per core (the
    process's CPU affinity, at most 16), one BLAS thread each, each worker on
    its own head; value = kept FLOPs of the attended query blocks / wall time.
    Runs before the GPU is first touched, so the forked workers inherit no
    device state."""
    import multiprocessing as mp

    global _CPU_BITS
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        avail = os.cpu_count() or 1
    heads = [(b, h) for b in range(wl.batch) for h in range(wl.heads)]
    workers = max(1, min(avail, 16, len(heads)))
    step = len(heads) / workers
    tasks = [(wl, *heads[int(w * step)], budget_s) for w in range(workers)]
    _CPU_BITS = bits
    t0 = time.perf_counter()
    with mp.get_context("fork").Pool(workers) as pool:
        res = pool.map(_cpu_head, tasks)
    wall = time.perf_counter() - t0
    _CPU_BITS = None
    flops = sum(r["flops"] for r in res)
    blocks = sum(r["blocks"] for r in res)
    attn_s = sum(r["attn_s"] for r in res)
    select_s = sum(r["select_s"] for r in res)
    nb = res[0]["n_blocks"]
    return {
        "value": flops / wall / 1e12,
        "unit": "TFLOP/s",
        "cores": workers,
        "blas_threads_per_worker": 1,
        "host_cores_available": avail,
        "kind": "oracle",
        "sample": (f"{workers} heads of {wl.name} in parallel, one forked worker per core with one BLAS "
                   f"thread: float64 pooling + scores + selection over all {nb} query blocks of each head, "
                   f"then block-sparse attention on {blocks} query blocks in all ({budget_s:.0f} s budget per "
                   f"worker); value = kept FLOPs of those blocks / wall seconds"),
        "wall_seconds": round(wall, 3),
        "attention_core_seconds": round(attn_s, 3),
        "selection_core_seconds_per_head": round(select_s / workers, 3),
        "attention_blocks": blocks,
        "cpu_model": _cpu_model(),
    }


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="large_64b_b1h48d128_n111600_s128")
    ap.add_argument("--keep-ratio", type=float, default=None, help="override the top-k keep ratio")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--calib-copy-mb", type=int, default=0,
                    help="first run a plain device copy of this many MiB (a known-size kernel "
                         "for scaling the FETCH_SIZE/WRITE_SIZE counters)")
    ap.add_argument("--all-workloads", action="store_true",
                    help="one JSON line per workload (and per keep ratio of the sweep), "
                         "without the CPU baseline; not the headline line")
    args = ap.parse_args(argv)

    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}); "
              "the path shards over (batch, head) with no communication, but no multi-GPU "
              "launcher is built.", file=sys.stderr)
        return 2

    from paper_2606_23743_amd import workloads

    if args.all_workloads:
        import torch
        for base in workloads.ALL:
            for r in (base.ratios or (None,)):
                wl = base.with_ratio(r) if r is not None else base
                rec = measure(args, wl, with_cpu=False)
                print(json.dumps(rec), flush=True)
                torch.cuda.empty_cache()
        return 0

    wl = workloads.find(args.workload)
    if wl is None:
        print(f"unknown workload {args.workload}; one of {list(workloads.BY_NAME)}", file=sys.stderr)
        return 2
    if args.keep_ratio is not None:
        wl = wl.with_ratio(args.keep_ratio)
    rec = measure(args, wl, with_cpu=not args.no_cpu_baseline)
    print(json.dumps(rec), flush=True)
    return 0


def measure(args, wl, with_cpu: bool):
    """Run the timed steps on one workload and return the JSON record."""
    import torch

    import paper_2606_23743_amd as sva
    from paper_2606_23743_amd import inputs

    print(f"[bench] generating {wl.name}", file=sys.stderr, flush=True)
    bits = inputs.generate(wl)
    cpu = None
    if with_cpu:
        # before the first device call: the forked workers inherit no GPU state
        print(f"[bench] cpu baseline (~{args.cpu_seconds:.0f} s per worker)", file=sys.stderr, flush=True)
        cpu = cpu_baseline(wl, bits, args.cpu_seconds)
        print(f"[bench] cpu baseline {cpu['value']:.4f} TFLOP/s on {cpu['cores']} cores", file=sys.stderr,
              flush=True)
    dev = {n: inputs.to_device(bits[n]) for n in ("q", "k", "v")}
    prob = sva.problem_for(wl)
    sel = sva.select_for(wl)
    nb = sva.num_blocks(prob)
    kmax = sva.max_keep(prob, sel)
    B, H, N, D, S = wl.batch, wl.heads, wl.seq_len, wl.head_dim, wl.block
    f32, i32 = torch.float32, torch.int32
    qp = torch.empty((B, H, nb, D), dtype=f32, device="cuda")
    kp = torch.empty_like(qp)
    idx = torch.empty((B, H, nb, kmax), dtype=i32, device="cuda")
    cnt = torch.empty((B, H, nb), dtype=i32, device="cuda")
    out = torch.empty((B, H, N, D), dtype=torch.bfloat16, device="cuda")
    stream = torch.cuda.current_stream()

    ev = lambda: torch.cuda.Event(enable_timing=True)   # noqa: E731
    pool_ev = [(ev(), ev()) for _ in range(args.steps)]
    sel_ev = [(ev(), ev()) for _ in range(args.steps)]
    att_ev = [(ev(), ev()) for _ in range(args.steps)]

    def step(k=None):
        if k is not None:
            pool_ev[k][0].record(stream)
        sva.pool_blocks(prob, dev["q"], dev["k"], qp, kp, stream=stream)
        if k is not None:
            pool_ev[k][1].record(stream)
            sel_ev[k][0].record(stream)
        sva.select_blocks(prob, sel, qp, kp, kmax, idx, cnt, stream=stream)
        if k is not None:
            sel_ev[k][1].record(stream)
            att_ev[k][0].record(stream)
        sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], idx, cnt, out=out, stream=stream)
        if k is not None:
            att_ev[k][1].record(stream)

    if args.calib_copy_mb > 0:
        n = args.calib_copy_mb * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] calibration copy of {args.calib_copy_mb} MiB done", file=sys.stderr, flush=True)
        del src, dst

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t_start, t_end = ev(), ev()
    torch.cuda.synchronize()
    t_start.record(stream)
    for k in range(args.steps):
        step(k)
    t_end.record(stream)
    torch.cuda.synchronize()
    ms_step = t_start.elapsed_time(t_end) / args.steps
    pool_t = [a.elapsed_time(b) for a, b in pool_ev]
    sel_t = [a.elapsed_time(b) for a, b in sel_ev]
    att_t = [a.elapsed_time(b) for a, b in att_ev]
    pool_ms, sel_ms, att_ms = float(np.mean(pool_t)), float(np.mean(sel_t)), float(np.mean(att_t))
    print(f"[bench] step {ms_step:.3f} ms (pool {pool_ms:.3f}, select {sel_ms:.3f}, attention {att_ms:.3f})",
          file=sys.stderr, flush=True)

    flops, flops_full, pairs = kept_flops(idx.cpu().numpy(), cnt.cpu().numpy(), N, S, D)
    att_tflops = flops / (att_ms * 1e-3) / 1e12
    value = flops / (ms_step * 1e-3) / 1e12
    pool_bytes = 2 * B * H * N * D * 2 + 2 * B * H * nb * D * 4
    # select reads both pooled tensors and writes the index lists and counts
    select_bytes = 2 * B * H * nb * D * 4 + B * H * nb * kmax * 4 + B * H * nb * 4

    extra = {}
    if not args.no_dense:
        dout = torch.empty_like(out)
        sva.dense_attention(prob, dev["q"], dev["k"], dev["v"], out=dout, stream=stream)
        a, b = ev(), ev()
        a.record(stream)
        sva.dense_attention(prob, dev["q"], dev["k"], dev["v"], out=dout, stream=stream)
        b.record(stream)
        torch.cuda.synchronize()
        dense_ms = a.elapsed_time(b)
        dense_flops = 4.0 * D * B * H * float(N) * N
        extra["dense_attention"] = {"ms": dense_ms, "tflops": dense_flops / (dense_ms * 1e-3) / 1e12,
                                    "sparse_path_speedup": dense_ms / ms_step}
    else:
        dout = None

    # first-order remainder of the dropped blocks (same lists): the kept part
    # in float32, block moments, weights, the per-head GEMM and the pooled-key
    # attention with the merge, as one call
    if nb <= 4096:
        ws = torch.empty(sva.remainder_workspace(prob), dtype=torch.uint8, device="cuda")
        orem = torch.empty_like(out)
        sva.sparse_attention_remainder(prob, dev["q"], dev["k"], dev["v"], qp, kp, idx, cnt, out=orem,
                                       workspace=ws, stream=stream)
        a, b = ev(), ev()
        a.record(stream)
        for _ in range(args.steps):
            sva.sparse_attention_remainder(prob, dev["q"], dev["k"], dev["v"], qp, kp, idx, cnt, out=orem,
                                           workspace=ws, stream=stream)
        b.record(stream)
        torch.cuda.synchronize()
        rem_ms = a.elapsed_time(b) / args.steps
        nbp = (nb + 31) // 32 * 32
        bhn = float(B * H * N)
        rem_flops = {"moments": 2.0 * D * D * bhn,                       # one outer product per token
                     "weights_gemm": 2.0 * B * H * nb * nb * D * D,      # T_i = sum_j E_ij M_j
                     "pooled_attention": 4.0 * D * nb * bhn + 2.0 * D * D * bhn}
        rec_rem = {"ms": round(rem_ms, 4), "sparse_attention_ms": round(att_ms, 4),
                   "extra_ms_over_sparse": round(rem_ms - att_ms, 4),
                   "remainder_flops": rem_flops, "padded_blocks": nbp,
                   "workspace_bytes": int(ws.numel()),
                   "mean_abs_change_vs_sparse": float((orem.float() - out.float()).abs().mean())}
        if dout is not None:
            rec_rem["mean_abs_diff_vs_dense"] = float((orem.float() - dout.float()).abs().mean())
            rec_rem["sparse_mean_abs_diff_vs_dense"] = float((out.float() - dout.float()).abs().mean())
        extra["remainder"] = rec_rem
        del ws, orem
    if dout is not None:
        del dout

    # the fused QKNorm + RoPE + pool producer on the same Q and K (unit gamma):
    # an alternative to the pool stage when Q and K arrive before their norm
    gam = torch.ones(D, dtype=torch.float32, device="cuda")
    qo, ko = torch.empty_like(dev["q"]), torch.empty_like(dev["k"])
    sva.qknorm_rope_pool(prob, dev["q"], dev["k"], gam, gam, q_out=qo, k_out=ko, q_pool=qp, k_pool=kp,
                         stream=stream)
    a, b = ev(), ev()
    a.record(stream)
    for _ in range(args.steps):
        sva.qknorm_rope_pool(prob, dev["q"], dev["k"], gam, gam, q_out=qo, k_out=ko, q_pool=qp,
                             k_pool=kp, stream=stream)
    b.record(stream)
    torch.cuda.synchronize()
    prod_ms = a.elapsed_time(b) / args.steps
    prod_bytes = 4 * B * H * N * D * 2 + 2 * B * H * nb * D * 4 + 2 * D * 4
    extra["qknorm_rope_pool"] = {
        "ms": round(prod_ms, 4), "algorithmic_bytes": prod_bytes,
        "hbm_gbs": round(prod_bytes / (prod_ms * 1e-3) / 1e9, 1),
        "frac_of_hbm_peak": round(prod_bytes / (prod_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "replaces_pool_ms": round(pool_ms, 4)}
    del qo, ko

    # 8-bit (e4m3) attention on the same layer and kept-block lists: the
    # quantiser once, then the fp8 kernel (kept FLOPs against the fp8 peak)
    if wl.head_dim in (64, 112, 128):
        quant = sva.quantize_fp8(prob, dev["q"], dev["k"], dev["v"], stream=stream)
        o8 = torch.empty_like(out)
        sva.sparse_attention_fp8(prob, quant, idx, cnt, out=o8, stream=stream)
        fp8_ms = {}
        for name, fn in (("quantize", lambda: sva.quantize_fp8(prob, dev["q"], dev["k"], dev["v"], out=quant,
                                                                 stream=stream)),
                         ("attention", lambda: sva.sparse_attention_fp8(prob, quant, idx, cnt, out=o8,
                                                                        stream=stream))):
            a, b = ev(), ev()
            a.record(stream)
            for _ in range(args.steps):
                fn()
            b.record(stream)
            torch.cuda.synchronize()
            fp8_ms[name] = a.elapsed_time(b) / args.steps
        sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], idx, cnt, out=out, stream=stream)
        torch.cuda.synchronize()
        diff = (o8.float() - out.float()).abs()
        fp8_tf = flops / (fp8_ms["attention"] * 1e-3) / 1e12
        extra["fp8_attention"] = {
            "format": "e4m3 Q, K (smoothed), V and P; power-of-two scales",
            "quantize_ms": round(fp8_ms["quantize"], 4), "attention_ms": round(fp8_ms["attention"], 4),
            "attention_tflops": round(fp8_tf, 2),
            "frac_of_fp8_peak": round(fp8_tf / FP8_PEAK_TFLOPS, 4),
            "frac_of_bf16_peak": round(fp8_tf / BF16_PEAK_TFLOPS, 4),
            "speedup_vs_bf16_attention": round(att_ms / fp8_ms["attention"], 3),
            "mean_abs_diff_vs_bf16_path": float(diff.mean()), "max_abs_diff_vs_bf16_path": float(diff.max())}
        del quant, o8, diff

    # feat_norm token pruning at keep ratio 0.5 on this workload's hidden
    # states (the video stream's Q heads laid out token-major, [B, N, H*D])
    x = dev["q"].permute(0, 2, 1, 3).reshape(B, N, H * D).contiguous()
    C = H * D
    scores, kept_idx, kept_pos = sva.token_select(x, 0.5, stream=stream)
    ws = torch.empty(sva.token_select_workspace(sva.tokens(B, N, C)), dtype=torch.uint8, device="cuda")
    kt = kept_idx.shape[1]
    xk = sva.token_gather(x, kept_idx, stream=stream)
    xo = torch.empty_like(x)
    tp_ms = {}
    for name, fn in (("select", lambda: sva.token_select(x, 0.5, scores, kept_idx, kept_pos, ws, stream)),
                     ("gather", lambda: sva.token_gather(x, kept_idx, xk, stream)),
                     ("scatter", lambda: sva.token_scatter(xk, kept_pos, x, xo, stream))):
        fn()
        a, b = ev(), ev()
        a.record(stream)
        for _ in range(args.steps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        tp_ms[name] = a.elapsed_time(b) / args.steps
    tp_bytes = {"select": B * N * C * 2 + B * N * (8 + 4) + B * kt * 4,
                "gather": 2 * B * kt * C * 2 + B * kt * 4,
                "scatter": 2 * B * N * C * 2 + B * N * 4}
    extra["token_prune"] = {
        "hidden": [B, N, C], "keep_ratio": 0.5, "kept": kt,
        "ms": {n: round(v, 4) for n, v in tp_ms.items()},
        "algorithmic_bytes": tp_bytes,
        "hbm_gbs": {n: round(tp_bytes[n] / (tp_ms[n] * 1e-3) / 1e9, 1) for n in tp_ms},
        "frac_of_hbm_peak": {n: round(tp_bytes[n] / (tp_ms[n] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
                             for n in tp_ms}}
    del x, scores, kept_idx, kept_pos, ws, xk, xo

    if cpu is not None:
        # the whole layer on the same cores at the measured rate (kept FLOPs of
        # every row plus each head's selection), an extrapolation
        cpu["full_layer_seconds_extrapolated"] = round(
            flops / (cpu["value"] * 1e12) + cpu["selection_core_seconds_per_head"] * B * H / cpu["cores"], 1)

    sel_desc = (f"cumulative mass tau={wl.mass_threshold} cap={kmax}" if wl.mode == "mass"
                else f"top-k k={kmax} (r={wl.keep_ratio})" if not wl.topk else f"top-k k={wl.topk}")
    rec = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": B, "heads": H, "seq_len": N, "head_dim": D,
                   "grid": [wl.grid_t, wl.grid_h, wl.grid_w], "block": S, "selection": sel_desc,
                   "kept_pairs": pairs, "kept_flops": flops, "kept_flops_full_blocks": flops_full},
        "pct_of_bf16_peak": round(100.0 * value / BF16_PEAK_TFLOPS, 2),
        "roofline": {"bound": "mfma", "kernel": "sparse attention", "achieved": round(att_tflops, 2),
                     "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(att_tflops / BF16_PEAK_TFLOPS, 4),
                     "traffic": measured_traffic(wl.name),
                     "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, calibrated)"},
        "stages_ms": {"pool": round(pool_ms, 4), "select": round(sel_ms, 4), "attention": round(att_ms, 4)},
        "stages_ms_median": {"pool": round(float(np.median(pool_t)), 4),
                             "select": round(float(np.median(sel_t)), 4),
                             "attention": round(float(np.median(att_t)), 4)},
        "pool_select_hbm_gbs": round((pool_bytes + select_bytes) / ((pool_ms + sel_ms) * 1e-3) / 1e9, 1),
        "pool_hbm_gbs": round(pool_bytes / (pool_ms * 1e-3) / 1e9, 1),
        "cpu_baseline": cpu,
    }
    rec.update(extra)
    del dev, qp, kp, idx, cnt, out
    return rec


if __name__ == "__main__":
    sys.exit(main())
