"""Sparse-FFN decode benchmark on one MI355X.

One step = one decode step of one token through every layer of the FFN stack:
predictor (the fp32 product P2 P1 when that is smaller than the two factors) ->
top-k block selection -> gate/up row gather + gating -> down projection +
residual, all in the HIP kernels behind the C ABI.

Workload (default): Llama-2-7B-shaped FFN stack, 32 layers, d_model 4096,
d_ff 11008, fp16 weights, ReGLU with ~10% active neurons, rank-1024 predictor,
64-neuron blocks, top 12% of blocks (k = 21 of 172), batch 1, fresh N(0,1)
token per step; synthetic seeded weights of that shape.

Prints ONE JSON line (see the "metric" contract): tokens/s, effective weight
GB/s on the algorithmic bytes, the roofline of the dominant kernel measured
with HIP events in the timed region, and the CPU oracle timed on a bounded
sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E peak, GB/s


def predictor_bytes(cfg) -> int:
    """Bytes of one layer's predictor as the library stores it: the fp32 product P2 P1
    [n_blk, d] when that is no larger than the factors P1 [r, d] and P2 [n_blk, r]."""
    folded = 4 * cfg.n_blk * cfg.d_model
    factored = cfg.elem_bytes * (cfg.rank * cfg.d_model + cfg.n_blk * cfg.rank)
    return min(folded, factored)


def algorithmic_bytes_per_layer(cfg, U: int, Z: int = 0) -> int:
    """Bytes one layer must read: the U selected blocks' gate/up/down rows (minus Z blocks whose
    down rows are skipped as all-zero), their gate bias, and the predictor."""
    s = cfg.elem_bytes
    ffn = U * cfg.block * cfg.d_model * 3 - Z * cfg.block * cfg.d_model
    bias = U * cfg.block if cfg.gate_bias is not None else 0
    return s * (ffn + bias) + predictor_bytes(cfg)


# the dominant kernel's launches are bracketed with HIP events in every this-many-th timed step
TIMING_SAMPLE_EVERY = 8


def measured_traffic(kernel: str, cfg, n_layers_default: bool):
    """HBM bytes per launch of `kernel` on this workload from the committed rocprofv3 counter
    summary (profiles/<kernel>_<workload>.md), or None when there is none, the workload differs,
    or the kernel's sources changed since the counters were taken (their sha256 differs)."""
    import hashlib
    import re
    path = os.path.join(ROOT, "profiles", f"{kernel}_{cfg.name}.md")
    if not n_layers_default or not os.path.exists(path):
        return None
    text = open(path).read()
    m_t = re.search(r"traffic_bytes_per_launch: (\d+)", text)
    m_h = re.search(r"source_sha256: ([0-9a-f]+)", text)
    m_s = re.search(r"sources: (.+)", text)
    if not (m_t and m_h and m_s):
        return None
    h = hashlib.sha256()
    for rel in m_s.group(1).split():
        full = os.path.join(ROOT, rel)
        if not os.path.exists(full):
            return None
        h.update(open(full, "rb").read())
    return int(m_t.group(1)) if h.hexdigest() == m_h.group(1) else None


def mean_union_size(f, cfg, xs, B: int, lsffn, torch) -> float:
    """Mean number of blocks per layer (the union over the B tokens) over the given steps,
    replayed through ls_predict / ls_select_blocks / ls_sparse_ffn_step."""
    dev = xs.device
    scores = torch.empty(B, cfg.n_blk, dtype=torch.float32, device=dev)
    cap = min(cfg.n_blk, B * cfg.k)
    idx = torch.empty(cap, dtype=torch.int32, device=dev)
    cnt = torch.empty(1, dtype=torch.int32, device=dev)
    xa = torch.empty(B, cfg.d_model, dtype=torch.float32, device=dev)
    xb = torch.empty_like(xa)
    total, n = 0, 0
    for t in range(xs.shape[0]):
        xa.copy_(xs[t])
        cur, nxt = xa, xb
        for l in range(cfg.n_layers):
            f.ls_predict(l, cur, B, scores)
            f.ls_select_blocks(scores, B, lsffn.LS_SEL_TOPK, cfg.k, 0.0, 1, cap, idx, cnt)
            f.ls_sparse_ffn_step(l, cur, B, idx, cnt, 0, cap, nxt)
            total += int(cnt.item())
            n += 1
            cur, nxt = nxt, cur
    return total / n


def host_cpu_info() -> dict:
    """Host CPU model string, nproc, the size of this process's affinity mask and the threads
    the oracle may use: the affinity mask, capped by OMP_NUM_THREADS when that is set (the
    machine's CPU share for this job)."""
    model = platform.processor() or platform.machine()
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    aff = len(os.sched_getaffinity(0))
    n = aff
    omp = os.environ.get("OMP_NUM_THREADS", "")
    if omp.isdigit() and int(omp) > 0:
        n = min(n, int(omp))
    return {"cpu": model, "nproc": os.cpu_count(), "affinity": aff, "threads": n}


def cpu_baseline(cfg, weights, xs, max_tokens: int, B: int = 1, budget_s: float = 12.0):
    """The CPU oracle (as it stands) on the first decode steps of the same workload, both on one
    thread and with its output loops split over every core this job may use (the same sums in
    the same order, so the same results).  Each leg decodes tokens until budget_s has passed or
    max_tokens are done.  At B = 1 the oracle's C layer step; at B > 1 its predictor, union
    selection and sparse FFN per token (single thread only)."""
    import numpy as np

    import oracle
    info = host_cpu_info()

    def leg(n_threads):
        t0 = time.perf_counter()
        done = 0
        while done < max_tokens and (done == 0 or time.perf_counter() - t0 < budget_s):
            t = done
            if B == 1:
                x = xs[t, 0].copy()
                for l in range(cfg.n_layers):
                    _, _, _, x = oracle.layer_step(weights[l], cfg, x, n_threads=n_threads)
            else:
                x = xs[t, :B].astype(np.float64)
                for l in range(cfg.n_layers):
                    w = weights[l]
                    h = np.stack([oracle.mlp_input(x[b], cfg.prenorm) for b in range(B)])
                    s = np.stack([oracle.predict(w.p1, w.p2, h[b]) for b in range(B)]).astype(np.float32)
                    idx, cnt = oracle.select(s, k=cfg.k, union_batch=True, cap=min(cfg.n_blk, B * cfg.k))
                    blocks = idx[:cnt[0]]
                    x = np.stack([x[b] + oracle.sparse_ffn(w, h[b], blocks, cfg.block, cfg.act, w.threshold)
                                  for b in range(B)]).astype(np.float32).astype(np.float64)
            done += 1
        return done, time.perf_counter() - t0

    n1, dt1 = leg(0)
    single = {"value": B * n1 / dt1, "unit": "tokens/s", "cores": 1,
              "sample": f"first {n1} decode steps x {cfg.n_layers} layers (B={B}), {dt1:.1f} s"}
    if B == 1 and info["threads"] > 1:
        nN, dtN = leg(info["threads"])
        return {"value": nN / dtN, "unit": "tokens/s", "cores": info["threads"], "kind": "oracle",
                "sample": f"first {nN} decode steps x {cfg.n_layers} layers of the same workload (B=1), "
                          f"fp64 oracle, output loops split over {info['threads']} threads, {dtN:.1f} s",
                "single_core": single, **info}
    return {"value": single["value"], "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": single["sample"] + ", fp64 oracle, single thread", **info}


def check_fused_against_kernels(f, cfg, x0, lsffn, torch, dev):
    """One decode step (B = 1) checked layer by layer: when it ran the fused kernel, its layer
    input x_l and scores (kept by the library) are fed to the per-kernel entry points (the
    selection on those scores, then the sparse FFN on x_l), and the fused kernel's layer output
    x_{l+1} - x_l must match theirs within 2e-3 (relative L2 and largest element, over the
    largest element).  Returns None when the step did not run the fused kernel."""
    import numpy as np
    x = torch.from_numpy(np.ascontiguousarray(x0)).to(dev)
    f.ls_decode_step(x, 1, cfg.k)
    f.ls_ffn_sync()
    xin = torch.empty(1, cfg.d_model, dtype=torch.float32, device=dev)
    scores = torch.empty(1, cfg.n_blk, dtype=torch.float32, device=dev)
    try:
        f.ls_debug_decode_trace(0, scores=scores)
    except lsffn.LsError:
        return None
    idx = torch.empty(cfg.k, dtype=torch.int32, device=dev)
    cnt = torch.empty(1, dtype=torch.int32, device=dev)
    out = torch.empty(1, cfg.d_model, dtype=torch.float32, device=dev)
    xf = x.cpu().numpy()[0].astype(np.float64)
    worst = 0.0
    x_l = torch.from_numpy(np.ascontiguousarray(x0)).to(dev)
    for l in range(cfg.n_layers):
        if l > 0:
            f.ls_debug_decode_trace(l, x_in=xin[0])
            x_l = xin.clone()
        f.ls_debug_decode_trace(l, scores=scores[0])
        if l + 1 < cfg.n_layers:
            f.ls_debug_decode_trace(l + 1, x_in=xin[0])
            x_next = xin[0].cpu().numpy().astype(np.float64)
        else:
            x_next = xf
        f.ls_select_blocks(scores, 1, lsffn.LS_SEL_TOPK, cfg.k, 0.0, 0, cfg.k, idx, cnt)
        f.ls_sparse_ffn_step(l, x_l, 1, idx, cnt, 0, cfg.k, out)
        xl = x_l[0].cpu().numpy().astype(np.float64)
        y_k = out[0].cpu().numpy().astype(np.float64) - xl
        y_f = x_next - xl
        err = max(np.linalg.norm(y_f - y_k) / np.linalg.norm(y_k),
                  np.max(np.abs(y_f - y_k)) / np.max(np.abs(y_k)))
        worst = max(worst, float(err))
    f.ls_ffn_sync()
    return {"layers": cfg.n_layers, "worst_y_err": worst, "ok": worst <= 2e-3,
            "what": "fused kernel vs per-kernel entry points on its own layer inputs and scores"}


def overlap_from_trace(d: str) -> dict:
    """Copy/compute overlap from a rocprofv3 csv trace: the time during which a host-to-device
    copy and a kernel are both active, over the kernels' busy time (interval unions)."""
    import csv
    import glob

    def intervals(pattern):
        out = []
        for path in glob.glob(os.path.join(d, "**", pattern), recursive=True):
            for r in csv.DictReader(open(path)):
                out.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
        out.sort()
        merged = []
        for a, b in out:
            if merged and a <= merged[-1][1]:
                merged[-1][1] = max(merged[-1][1], b)
            else:
                merged.append([a, b])
        return merged

    k = intervals("*kernel_trace.csv")
    c = intervals("*memory_copy_trace.csv")
    busy_k = sum(b - a for a, b in k)
    busy_c = sum(b - a for a, b in c)
    both, j = 0, 0
    for a, b in k:
        while j < len(c) and c[j][1] <= a:
            j += 1
        jj = j
        while jj < len(c) and c[jj][0] < b:
            both += max(0, min(b, c[jj][1]) - max(a, c[jj][0]))
            jj += 1
    return {"kernel_busy_ms": busy_k / 1e6, "copy_busy_ms": busy_c / 1e6, "both_ms": both / 1e6,
            "overlap_of_kernel_time": both / busy_k if busy_k else None}


def bench_streaming(args, cfg) -> int:
    """Host-resident stack through ls_decode_step_streamed: per layer predict -> select -> misses
    copied from pinned host memory in priority order, in stages -> staged sparse steps that wait
    per stage, with the next layer's blocks prefetched during the current layer (--prefetch:
    none, one-shot from the layer input, or refined after every stage on the partial result,
    Eq. 2).  The HBM cache holds the same fraction of all blocks as the full workload's budget."""
    import numpy as np
    import torch

    import lsgen
    import paper_2609_03079_amd as lsffn

    # the cache holds the same fraction of the blocks as the full workload's budget does
    # (16 GiB over all of its layers), whatever the number of layers run
    full_blocks = lsgen.CONFIGS[cfg.name].n_layers * cfg.n_blk
    L = args.layers or 6
    cfg = cfg.with_(n_layers=L)
    block_bytes = 3 * cfg.block * cfg.d_model * cfg.elem_bytes
    cache_frac = cfg.hbm_cache_bytes / (full_blocks * block_bytes)
    # a layer's list and the next layer's prefetched list must fit together
    slots = max(cfg.k + (args.k_spec or cfg.k), int(cache_frac * L * cfg.n_blk))
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    t_setup = time.perf_counter()
    f = lsffn.Ffn(n_layers=L, d_model=cfg.d_model, d_ff=cfg.d_ff, block=cfg.block, rank=cfg.rank,
                  max_batch=1, dtype=cfg.dtype, act=cfg.act, residency=lsffn.LS_WEIGHTS_HOST,
                  prenorm_rms=int(cfg.prenorm), hbm_cache_bytes=slots * block_bytes, stream=stream)
    f.ls_configure(lsffn.LS_CFG_STREAM_SYNC, {"events": lsffn.LS_SYNC_EVENTS, "flags": lsffn.LS_SYNC_FLAGS,
                                              "host": lsffn.LS_SYNC_HOST}[args.stream_sync])
    weights = []
    for l in range(L):
        w = lsgen.layer_weights(cfg, l)
        f.ls_ffn_set_layer(l, w)
        weights.append(w if args.cpu_tokens > 0 else None)
        print(f"set-up: {l + 1}/{L} layers", file=sys.stderr, flush=True)
    W, K, S = args.warmup, args.steps, args.stages
    xs = torch.from_numpy(lsgen.tokens(cfg, 0, W + K, 1)).to(dev)
    # pinned host -> HBM peak of one large copy, the ceiling of this path
    src = torch.empty(1 << 30, dtype=torch.uint8, pin_memory=True)
    dst = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(4):
        dst.copy_(src, non_blocking=True)
    e1.record(stream)
    torch.cuda.synchronize()
    h2d_gbs = 4 * (1 << 30) / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    setup_s = time.perf_counter() - t_setup

    modes = {"none": lsffn.LS_PREFETCH_NONE, "oneshot": lsffn.LS_PREFETCH_ONESHOT,
             "refine": lsffn.LS_PREFETCH_REFINE}
    k_spec = args.k_spec or cfg.k
    x = torch.empty(1, cfg.d_model, dtype=torch.float32, device=dev)

    def run(mode_name):
        totals = {"final": 0, "late": 0, "spec": 0, "wasted": 0}
        mode = modes[mode_name]
        for i in range(W):
            x.copy_(xs[i])
            f.ls_decode_step_streamed(x, cfg.k, S, mode, k_spec)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(K):
            x.copy_(xs[W + i])
            r = f.ls_decode_step_streamed(x, cfg.k, S, mode, k_spec)
            totals["final"] += r.final_bytes
            totals["late"] += r.late_bytes
            totals["spec"] += r.spec_bytes
            totals["wasted"] += r.wasted_bytes
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        totals["bytes"] = totals["late"] + totals["spec"]
        return wall, totals

    compare = {}
    if args.prefetch_compare:
        for name in modes:
            if args.stream_sync == "flags" and name == "refine":
                continue  # re-scoring between stage launches needs per-stage launches
            w_, t_ = run(name)
            compare[name] = {"tokens_per_s": round(K / w_, 3),
                             "copied_GB_per_token": round(t_["bytes"] / K / 1e9, 4),
                             "late_GB_per_token": round(t_["late"] / K / 1e9, 4),
                             "relative_loading_redundancy": round(t_["wasted"] / t_["final"], 4)}
            print(f"prefetch {name}: {compare[name]}", file=sys.stderr, flush=True)
    wall, totals = run(args.prefetch)
    copy_gbs = totals["bytes"] / wall / 1e9
    cpu = None
    if args.cpu_tokens > 0:
        cpu = cpu_baseline(cfg, weights, lsgen.tokens(cfg, 0, W + K, 1), min(args.cpu_tokens, W + K))
    out = {
        "metric": "sparse-FFN decode tokens/sec and effective weight GB/s (% HBM peak), 1 GPU",
        "value": round(K / wall, 3), "unit": "tokens/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": round(1e3 * wall / K, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": lsgen.DTYPE_NAMES[cfg.dtype], "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {L} of {lsgen.CONFIGS[cfg.name].n_layers} layers, d_model {cfg.d_model}, d_ff {cfg.d_ff}, "
                               f"block {cfg.block} (k={cfg.k} of {cfg.n_blk}), rank {cfg.rank}, batch 1, "
                               f"host-resident blocks, HBM cache {slots} slots ({100 * cache_frac:.1f}% of "
                               f"the blocks), {S} copy stages per layer, prefetch {args.prefetch} "
                               f"({k_spec} blocks per prediction), stage sync {args.stream_sync}",
                   "global_batch": 1, "seq_len": 1, "parallelism": "none (1 GPU)", "decode_path": "kernels"},
        "streaming": {"copied_GB_per_token": round(totals["bytes"] / K / 1e9, 4),
                      "late_GB_per_token": round(totals["late"] / K / 1e9, 4),
                      "relative_loading_redundancy": round(totals["wasted"] / totals["final"], 4),
                      "copy_GBs": round(copy_gbs, 2), "h2d_peak_GBs": round(h2d_gbs, 2),
                      "prefetch_modes": compare or None},
        "roofline": {"bound": "host_link", "kernel": "hipMemcpyAsync (pinned host -> HBM)",
                     "achieved": round(copy_gbs, 2), "peak": round(h2d_gbs, 2), "unit": "GB/s",
                     "frac": round(copy_gbs / h2d_gbs, 4), "traffic": None},
        "cpu_baseline": cpu,
        "setup_s": round(setup_s, 1),
    }
    print(json.dumps(out))
    f.close()
    return 0


def bench_refinement(args, cfg) -> int:
    """Quality of the next layer's prediction after each of K stages of a layer (Eq. 2), on a
    workload with a planted predictor: importance ratio and top-10% recall of the predicted
    next-layer set against that layer's block importance on its complete input (sum over a
    block's neurons of |a_j| * ||Wd[:, j]||).  The stages run over the priority list and, for
    comparison, over the same blocks in reverse priority order.  Staged steps, predictions,
    selections and the all-block activations run in the library; the two ratios are computed
    on the host from its outputs."""
    import numpy as np
    import torch

    import lsgen
    import paper_2609_03079_amd as lsffn

    L = args.layers or 4
    cfg = cfg.with_(n_layers=L)
    K, k, nb = args.stages, cfg.k, cfg.n_blk
    dev = torch.device("cuda:0")
    torch.cuda.set_device(0)
    f = lsffn.Ffn(n_layers=L, d_model=cfg.d_model, d_ff=cfg.d_ff, block=cfg.block, rank=cfg.rank,
                  max_batch=1, dtype=cfg.dtype, act=cfg.act, prenorm_rms=int(cfg.prenorm))
    col = []
    for l in range(L):
        w = lsgen.layer_weights(cfg, l)
        f.ls_ffn_set_layer(l, w)
        wd = lsgen.decode_bits(w.down, cfg.dtype)
        col.append(np.sqrt((wd * wd).sum(axis=0)))
        print(f"set-up: {l + 1}/{L} layers", file=sys.stderr, flush=True)
    scores = torch.empty(1, nb, dtype=torch.float32, device=dev)
    idx = torch.empty(k, dtype=torch.int32, device=dev)
    cnt = torch.empty(1, dtype=torch.int32, device=dev)
    sel = torch.empty(k, dtype=torch.int32, device=dev)
    scnt = torch.empty(1, dtype=torch.int32, device=dev)
    acc = torch.empty(1, cfg.d_model, dtype=torch.float32, device=dev)
    full = torch.empty_like(acc)
    all_blk = torch.arange(nb, dtype=torch.int32, device=dev)
    all_cnt = torch.tensor([nb], dtype=torch.int32, device=dev)
    act = torch.empty(cfg.d_ff, dtype=torch.float32, device=dev)

    def next_set(l, feat):
        f.ls_predict(l, feat, 1, scores)
        f.ls_select_blocks(scores, 1, lsffn.LS_SEL_TOPK, k, 0.0, 0, k, sel, scnt)
        return sel.cpu().numpy().copy()

    def ratios(imp, P):
        best = np.sort(imp)[::-1][:len(P)].sum()
        m = max(1, -(-nb // 10))
        top = np.lexsort((np.arange(nb), -imp))[:m]
        return imp[P].sum() / best, np.isin(top, P).sum() / m

    curves = {"priority": np.zeros((K + 1, 2)), "reverse": np.zeros((K + 1, 2))}
    n_obs = 0
    xs = torch.from_numpy(lsgen.tokens(cfg, 0, args.steps, 1)).to(dev)
    t0 = time.perf_counter()
    for t in range(args.steps):
        x = xs[t].clone()
        for n in range(L - 1):
            f.ls_predict(n, x, 1, scores)
            f.ls_select_blocks(scores, 1, lsffn.LS_SEL_TOPK, k, 0.0, 0, k, idx, cnt)
            sets = {}
            for name, lst in (("priority", idx), ("reverse", torch.flip(idx, [0]).contiguous())):
                sets[name] = [next_set(n + 1, x)]
                for j in range(K):
                    f.ls_sparse_ffn_step(n, x, 1, lst, cnt, j * k // K, (j + 1) * k // K, acc)
                    sets[name].append(next_set(n + 1, acc))
                if name == "priority":
                    nxt = acc.clone()
            # the next layer's block importance on its complete input
            f.ls_sparse_ffn_step(n + 1, nxt, 1, all_blk, all_cnt, 0, nb, full)
            f.ls_debug_last_activations(act)
            a = act.cpu().numpy().astype(np.float64)
            imp = (np.abs(a) * col[n + 1]).reshape(nb, cfg.block).sum(axis=1)
            for name in curves:
                for j, P in enumerate(sets[name]):
                    curves[name][j] += ratios(imp, P)
            n_obs += 1
            x = nxt
        print(f"token {t + 1}/{args.steps}", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    for name in curves:
        curves[name] /= n_obs
    out = {
        "metric": "next-layer importance ratio after refinement stages (Eq. 2), planted predictor",
        "value": round(float(curves["priority"][K // 2, 0]), 4), "unit": f"ratio after {K // 2}/{K} stages",
        "n_gpus": 1, "steps": args.steps, "warmup": 0, "ms_per_step": round(1e3 * wall / args.steps, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": lsgen.DTYPE_NAMES[cfg.dtype], "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {L} layers, d_model {cfg.d_model}, d_ff {cfg.d_ff}, block "
                               f"{cfg.block} (k={k} of {nb}), rank {cfg.rank}, {K} stages, "
                               f"{n_obs} (token, layer) pairs",
                   "global_batch": 1, "seq_len": 1, "parallelism": "none (1 GPU)"},
        "refinement": {name: {"importance_ratio": [round(float(v), 4) for v in c[:, 0]],
                              "top10_recall": [round(float(v), 4) for v in c[:, 1]]}
                       for name, c in curves.items()},
        "roofline": None, "cpu_baseline": None,
    }
    print(json.dumps(out))
    f.close()
    return 0


def zero_skip_bytes(cfg, acts, n_entries: int):
    """Gate/up/down bytes of one layer's n_entries list blocks, from the activations acts
    ([B, n_entries * block] in list order; a neuron counts as active when its activation is
    nonzero for some token).  Returns (block, neuron, kernel):
      block  every row of the blocks (the block path);
      neuron gate rows of all their neurons, up and down rows of the active ones;
      kernel as neuron, but down rows come in groups of V = 16 / element-size neurons (one
             16-byte vector of the down layout holds V neurons of one output column), and a
             group with an active neuron costs all V."""
    import numpy as np
    s, d, blk = cfg.elem_bytes, cfg.d_model, cfg.block
    V = 16 // s
    row = d * s
    if n_entries <= 0:
        return 0, 0, 0
    a = np.asarray(acts).reshape(-1, n_entries * blk)
    act = (a != 0).any(axis=0)
    n_act = int(act.sum())
    n_grp = int(act.reshape(n_entries, blk // V, V).any(axis=2).sum())
    gate = n_entries * blk * row
    return 3 * gate, gate + 2 * n_act * row, gate + n_act * row + n_grp * V * row


def bench_zero_skip(args, cfg) -> int:
    """Row-level zero skip within the selected blocks on the per-kernel path: the bytes the
    gate/up and down kernels must read with and without it (counted from the activations of
    the same steps), the decode rate both ways, and a check that both give equal outputs."""
    import numpy as np
    import torch

    import lsgen
    import paper_2609_03079_amd as lsffn

    L = args.layers or cfg.n_layers
    cfg = cfg.with_(n_layers=L)
    B, K, W = args.batch, args.steps, args.warmup
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    f = lsffn.Ffn(n_layers=L, d_model=cfg.d_model, d_ff=cfg.d_ff, block=cfg.block, rank=cfg.rank,
                  max_batch=B, dtype=cfg.dtype, act=cfg.act, prenorm_rms=int(cfg.prenorm), stream=stream)
    f.ls_configure(lsffn.LS_CFG_DECODE_PATH, 1)
    for l in range(L):
        f.ls_ffn_set_layer(l, lsgen.layer_weights(cfg, l))
        if (l + 1) % 8 == 0:
            print(f"set-up: {l + 1}/{L} layers", file=sys.stderr, flush=True)
    xs = torch.from_numpy(lsgen.tokens(cfg, 0, W + K, B)).to(dev)

    # bytes and equality: the first T steps through the per-call entry points, both ways
    T = min(K, args.zero_skip_tokens)
    cap = min(cfg.n_blk, B * cfg.k)
    scores = torch.empty(B, cfg.n_blk, dtype=torch.float32, device=dev)
    idx = torch.empty(cap, dtype=torch.int32, device=dev)
    cnt = torch.empty(1, dtype=torch.int32, device=dev)
    y = [torch.empty(B, cfg.d_model, dtype=torch.float32, device=dev) for _ in range(2)]
    act = torch.empty(B * cfg.d_ff, dtype=torch.float32, device=dev)
    tot = np.zeros(3)
    n_act = n_neur = 0
    equal = True
    for t in range(T):
        x = xs[t].clone()
        for l in range(L):
            f.ls_predict(l, x, B, scores)
            f.ls_select_blocks(scores, B, lsffn.LS_SEL_TOPK, cfg.k, 0.0, 1, cap, idx, cnt)
            for zs in (0, 1):
                f.ls_configure(lsffn.LS_CFG_ZERO_SKIP, zs)
                f.ls_sparse_ffn_step(l, x, B, idx, cnt, 0, cap, y[zs])
            n = f.ls_debug_last_activations(act)
            U = int(cnt.item())
            a = act[:B * n].view(B, n)[:, :U * cfg.block].cpu().numpy()
            tot += zero_skip_bytes(cfg, a, U)
            n_act += int((a != 0).any(axis=0).sum())
            n_neur += U * cfg.block
            equal &= bool(torch.equal(y[0], y[1]))
            x = y[1].clone()
        print(f"bytes: token {t + 1}/{T}", file=sys.stderr, flush=True)
    per_tok = tot / T

    res = {}
    for zs in (0, 1):
        f.ls_configure(lsffn.LS_CFG_ZERO_SKIP, zs)
        for i in range(W):
            f.ls_decode_step(xs[i].clone(), B, cfg.k)
        # the rate with no events between the launches, then the kernels' times with an event
        # pair around each launch (the pairs widen every launch gap)
        xw = [xs[W + i].clone() for i in range(K)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(K):
            f.ls_decode_step(xw[i], B, cfg.k)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        f.ls_set_kernel_timing(True)
        f.ls_kernel_timing(0, reset=True)
        for i in range(K):
            f.ls_decode_step(xs[W + i].clone(), B, cfg.k)
        torch.cuda.synchronize()
        f.ls_set_kernel_timing(False)
        r = {"tokens_per_s": round(B * K / wall, 2), "ms_per_step": round(1e3 * wall / K, 4)}
        for kid, name in ((lsffn.LS_K_GATEUP, "gateup"), (lsffn.LS_K_DOWN, "down")):
            ms, n = f.ls_kernel_timing(kid)
            r[f"{name}_avg_us"] = round(1e3 * ms / max(n, 1), 3)
        res["on" if zs else "off"] = r
        print(f"timed: zero skip {zs}", file=sys.stderr, flush=True)

    on = res["on"]
    U_mean = n_neur / (T * L * cfg.block)
    s, row = cfg.elem_bytes, cfg.d_model * cfg.elem_bytes
    gate_b = U_mean * cfg.block * row
    act_rows = n_act / (T * L)
    # the dominant kernel under zero skip and its bytes per launch (one launch per layer)
    gu_bytes = gate_b + act_rows * row
    dn_bytes = per_tok[2] / L - gu_bytes
    dom, dom_bytes = (("gateup", gu_bytes) if on["gateup_avg_us"] >= on["down_avg_us"] else ("down", dn_bytes))
    achieved = dom_bytes / (on[f"{dom}_avg_us"] * 1e-6) / 1e9
    out = {
        "metric": "row-level zero skip (per-kernel path): weight bytes per token and decode tokens/s, 1 GPU",
        "value": on["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": on["ms_per_step"], "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": lsgen.DTYPE_NAMES[cfg.dtype], "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {L} layers, d_model {cfg.d_model}, d_ff {cfg.d_ff}, block "
                               f"{cfg.block} (k={cfg.k} of {cfg.n_blk}), rank {cfg.rank}, batch {B}",
                   "global_batch": B, "seq_len": 1, "parallelism": "none (1 GPU)", "decode_path": "kernels"},
        "zero_skip": {"outputs_equal": equal, "byte_tokens": T,
                      "active_fraction_in_selected_blocks": round(n_act / max(n_neur, 1), 4),
                      "ffn_bytes_per_token": {"block": int(per_tok[0]), "neuron": int(per_tok[1]),
                                              "kernel": int(per_tok[2])},
                      "kernel_over_block": round(per_tok[2] / per_tok[0], 4),
                      "neuron_over_block": round(per_tok[1] / per_tok[0], 4),
                      "off": res["off"], "on": on},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "bytes_per_launch": int(dom_bytes), "avg_launch_us": on[f"{dom}_avg_us"]},
        "cpu_baseline": None,
    }
    print(json.dumps(out))
    f.close()
    return 0 if equal else 1


def bench_sync_overhead(args, cfg) -> int:
    """Synchronisation overhead of one MLP layer split into K stages (the paper's Table 3
    comparison), with host-resident weights whose blocks are all already in the HBM cache, so
    no copy is waited for: per-layer time of the streamed decode step for K = 1..16 with a host
    synchronisation after every stage, with per-stage events and launches, and with device
    flags and one persistent launch per layer.  The overhead is the per-layer time minus that of
    one launch pair per layer (events, K = 1); the MLP compute is the gate/up + down kernel
    time of that case."""
    import numpy as np
    import torch

    import lsgen
    import paper_2609_03079_amd as lsffn

    L = args.layers or 8
    cfg = cfg.with_(n_layers=L)
    k, nb = cfg.k, cfg.n_blk
    bb = 3 * cfg.block * cfg.d_model * cfg.elem_bytes
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    f = lsffn.Ffn(n_layers=L, d_model=cfg.d_model, d_ff=cfg.d_ff, block=cfg.block, rank=cfg.rank, max_batch=1,
                  dtype=cfg.dtype, act=cfg.act, prenorm_rms=int(cfg.prenorm), residency=lsffn.LS_WEIGHTS_HOST,
                  hbm_cache_bytes=L * nb * bb, stream=stream)
    for l in range(L):
        f.ls_ffn_set_layer(l, lsgen.layer_weights(cfg, l))
        print(f"set-up: {l + 1}/{L} layers", file=sys.stderr, flush=True)
    every = np.arange(nb, dtype=np.int32)
    for l in range(L):  # every block of every layer resident: the timed steps copy nothing
        f.ls_stream_weights(l, every, 1)
    f.ls_ffn_sync()
    xs = torch.from_numpy(lsgen.tokens(cfg, 0, args.warmup + args.steps, 1)).to(dev)
    Ks = (1, 2, 4, 8, 16)
    names = {lsffn.LS_SYNC_HOST: "host_sync", lsffn.LS_SYNC_EVENTS: "events", lsffn.LS_SYNC_FLAGS: "device_flags"}
    per_layer = {}
    compute_us = None
    stage_us = {}
    copied = 0
    for sync, name in names.items():
        f.ls_configure(lsffn.LS_CFG_STREAM_SYNC, sync)
        per_layer[name] = {}
        for K in Ks:
            for i in range(args.warmup):
                f.ls_decode_step_streamed(xs[i].clone(), k, K, lsffn.LS_PREFETCH_NONE, k)
            torch.cuda.synchronize()
            timing = (name == "events" and K == 1) or name == "device_flags"
            if timing:
                f.ls_set_kernel_timing(True)
                f.ls_kernel_timing(0, reset=True)
            xw = [xs[args.warmup + i].clone() for i in range(args.steps)]
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for i in range(args.steps):
                r = f.ls_decode_step_streamed(xw[i], k, K, lsffn.LS_PREFETCH_NONE, k)
                copied += r.copied_bytes
            f.ls_ffn_sync()
            wall = time.perf_counter() - t0
            per_layer[name][K] = 1e3 * wall / (args.steps * L)
            if timing:
                if name == "events":
                    gu, n1 = f.ls_kernel_timing(lsffn.LS_K_GATEUP)
                    dn, n2 = f.ls_kernel_timing(lsffn.LS_K_DOWN)
                    compute_us = 1e3 * (gu / max(n1, 1) + dn / max(n2, 1))
                else:
                    ms, n = f.ls_kernel_timing(lsffn.LS_K_STAGE)
                    stage_us[K] = round(1e3 * ms / max(n, 1), 2)
                f.ls_set_kernel_timing(False)
            if name == "device_flags":
                assert all(f.ls_debug_stages_done(l) == K for l in range(L))
            print(f"timed: {name} K={K}: {per_layer[name][K]:.4f} ms per layer", file=sys.stderr, flush=True)
    base = per_layer["events"][1]
    overhead = {name: {str(K): round(v[K] - base, 4) for K in Ks} for name, v in per_layer.items()}
    out = {
        "metric": "synchronisation overhead per MLP layer vs stages (Table 3 comparison), 1 GPU",
        "value": overhead["device_flags"]["16"], "unit": "ms per layer at 16 stages (device flags)",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(per_layer["device_flags"][16] * L, 4), "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None, "dtype": lsgen.DTYPE_NAMES[cfg.dtype], "data": "synthetic",
        "config": {"workload": f"{cfg.name} shape, host-resident weights, every block cached: {L} layers, d_model "
                               f"{cfg.d_model}, d_ff {cfg.d_ff}, block {cfg.block} (k={k} of {nb}), batch 1",
                   "global_batch": 1, "seq_len": 1, "parallelism": "none (1 GPU)"},
        "sync_overhead_ms": overhead,
        "per_layer_ms": {name: {str(K): round(v[K], 4) for K in Ks} for name, v in per_layer.items()},
        "mlp_compute_ms": round(compute_us / 1e3, 4) if compute_us else None,
        "stage_kernel_us": stage_us,
        "bytes_copied_in_timed_steps": copied,
        "roofline": None, "cpu_baseline": None,
    }
    print(json.dumps(out))
    f.close()
    return 0


def bench_hash(args, cfg) -> int:
    """Latency of the stacked hashing predictor (one workgroup per token) against the low-rank
    predictor (the folded GEMV) on the same shape, per call, from the library's HIP-event
    kernel timing, at B = 1 and B = args.batch."""
    import numpy as np  # noqa: F401
    import torch

    import lsgen
    import paper_2609_03079_amd as lsffn

    Bmax = max(1, args.batch)
    cfg = cfg.with_(n_layers=1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(0)
    f = lsffn.Ffn(n_layers=1, d_model=cfg.d_model, d_ff=cfg.d_ff, block=cfg.block, rank=cfg.rank,
                  max_batch=Bmax, dtype=cfg.dtype, act=cfg.act, prenorm_rms=int(cfg.prenorm))
    f.ls_ffn_set_layer(0, lsgen.layer_weights(cfg, 0))
    f.ls_set_hash_predictor(0, lsgen.hash_weights(cfg, 0))
    xs = torch.from_numpy(lsgen.tokens(cfg, 0, 1, Bmax)[0]).to(dev)
    scores = torch.empty(Bmax, cfg.n_blk, dtype=torch.float32, device=dev)
    res = {}
    for B in sorted({1, Bmax}):
        for name, call, kid in (("hash", lambda: f.ls_hash_predict(0, xs, B, scores), lsffn.LS_K_HASH),
                                ("lowrank", lambda: f.ls_predict(0, xs, B, scores), lsffn.LS_K_PRED_P1)):
            for _ in range(args.warmup):
                call()
            f.ls_set_kernel_timing(1)
            f.ls_kernel_timing(kid, reset=True)
            for _ in range(args.steps):
                call()
            ms, n = f.ls_kernel_timing(kid)
            f.ls_set_kernel_timing(0)
            res[f"{name}_B{B}_us"] = round(1e3 * ms / max(n, 1), 3)
    # bytes one hashing call must read: x, the first layer's hyperplanes, the four binary layers'
    # rows and hyperplanes, the head row, the scores written
    hash_bytes = lambda B: B * (4 * cfg.d_model + 4 * cfg.n_blk) + 32 * cfg.d_model + 4 * (32 + 256) + cfg.n_blk
    us1 = res["hash_B1_us"]
    out = {
        "metric": "stacked hashing predictor latency per call (Sec. 3.3.1), 1 GPU",
        "value": us1, "unit": "us per call (B = 1)", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(us1 / 1e3, 6), "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32 (first layer), binary", "data": "synthetic",
        "config": {"workload": f"{cfg.name} layer shape: d_model {cfg.d_model}, {cfg.n_blk} blocks; 5 hashing "
                               f"layers, 8 bits, 256-wide; random weights", "global_batch": Bmax,
                   "seq_len": 1, "parallelism": "none (1 GPU)"},
        "latency_us": res,
        "roofline": {"bound": "latency", "kernel": "hash_predict", "achieved": round(hash_bytes(1) / us1 / 1e3, 3),
                     "peak": 8000.0, "unit": "GB/s", "frac": round(hash_bytes(1) / us1 / 1e3 / 8000.0, 6),
                     "traffic": None, "bytes_per_launch": hash_bytes(1)},
        "cpu_baseline": None,
    }
    print(json.dumps(out))
    f.close()
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--config", default="llama2_7b_ffn")
    ap.add_argument("--batch", type=int, default=1)
    ap.add_argument("--cpu-tokens", type=int, default=64,
                    help="most tokens per CPU-oracle leg (each leg stops after about 12 s; 0: skip)")
    ap.add_argument("--repeats", type=int, default=5, help="timed repetitions of --steps steps (median reported)")
    ap.add_argument("--no-check", dest="check", action="store_false",
                    help="skip the per-layer check of one timed step against the per-kernel path")
    ap.add_argument("--layers", type=int, default=0, help="override the layer count (testing)")
    ap.add_argument("--path", choices=("auto", "kernels", "fused"), default="auto",
                    help="decode path: fused kernel when supported (auto), per-kernel sequence, fused only")
    ap.add_argument("--launch", choices=("cooperative", "plain"), default="plain",
                    help="fused-kernel launch: a plain launch of the one-workgroup-per-CU grid on the idle "
                         "device (default; the launch rocprofv3 can trace) or hipLaunchCooperativeKernel")
    ap.add_argument("--stages", type=int, default=8,
                    help="host-resident workloads: copy stages per layer (events the compute waits on)")
    ap.add_argument("--prefetch", choices=("none", "oneshot", "refine"), default="refine",
                    help="host-resident workloads: cross-layer prefetch policy of the streamed step")
    ap.add_argument("--stream-sync", choices=("events", "flags", "host"), default="events",
                    help="host-resident workloads: how a stage's compute waits for its copies (per-stage "
                         "events and launches, device flags with one persistent launch per layer, or a host "
                         "synchronisation after every stage)")
    ap.add_argument("--k-spec", type=int, default=0,
                    help="host-resident workloads: blocks per next-layer prediction (0: k)")
    ap.add_argument("--hash-predict", action="store_true",
                    help="instead of the benchmark: latency of the stacked hashing predictor against the "
                         "low-rank predictor (B = 1 and --batch)")
    ap.add_argument("--refinement-quality", action="store_true",
                    help="instead of the benchmark: next-layer prediction quality per refinement "
                         "stage (use with --config llama2_7b_planted)")
    ap.add_argument("--sync-overhead", action="store_true",
                    help="instead of the benchmark: per-layer synchronisation overhead vs stage count with "
                         "host synchronisation, events and device flags (use with --config mistral_7b_ffn)")
    ap.add_argument("--zero-skip", action="store_true",
                    help="instead of the benchmark: row-level zero skip on the per-kernel path (bytes "
                         "per token with and without it, decode rate both ways)")
    ap.add_argument("--zero-skip-tokens", type=int, default=8,
                    help="with --zero-skip: tokens whose activations give the byte counts")
    ap.add_argument("--prefetch-compare", action="store_true",
                    help="host-resident workloads: also time every prefetch policy")
    ap.add_argument("--overlap-from-trace", default="", metavar="DIR",
                    help="instead of the benchmark: copy/compute overlap from a rocprofv3 kernel + "
                         "memory-copy trace (csv) in DIR")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="instead of the benchmark: copy MIB MiB device-to-device 4 times (the known-size "
                         "kernel that scales the FETCH_SIZE / WRITE_SIZE counters to bytes)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              f"(the library has no multi-GPU path).", file=sys.stderr)
        return 2
    if args.stream_sync == "flags" and args.prefetch == "refine":
        print("--stream-sync flags runs one persistent launch per layer, which refined prefetch "
              "(per-stage launches) cannot use: pass --prefetch none or oneshot.", file=sys.stderr)
        return 2

    if args.overlap_from_trace:
        print(json.dumps(overlap_from_trace(args.overlap_from_trace)))
        return 0
    if args.refinement_quality:
        import lsgen
        return bench_refinement(args, lsgen.CONFIGS[args.config])
    if args.hash_predict:
        import lsgen
        return bench_hash(args, lsgen.CONFIGS[args.config])
    if args.sync_overhead:
        import lsgen
        return bench_sync_overhead(args, lsgen.CONFIGS[args.config])
    if args.zero_skip:
        import lsgen
        return bench_zero_skip(args, lsgen.CONFIGS[args.config])

    import numpy as np
    import torch

    if args.copy_calibration:
        n = args.copy_calibration << 20
        a = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        b = torch.empty_like(a)
        for _ in range(4):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_per_launch": n}))
        return 0

    import lsgen
    import paper_2609_03079_amd as lsffn

    cfg = lsgen.CONFIGS[args.config]
    if args.layers:
        cfg = cfg.with_(n_layers=args.layers)
    if cfg.host_resident:
        return bench_streaming(args, cfg)
    B, K, W = args.batch, args.steps, args.warmup
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()

    t_setup = time.perf_counter()
    f = lsffn.Ffn(n_layers=cfg.n_layers, d_model=cfg.d_model, d_ff=cfg.d_ff, block=cfg.block,
                  rank=cfg.rank, max_batch=B, dtype=cfg.dtype, act=cfg.act,
                  prenorm_rms=int(cfg.prenorm), stream=stream)
    f.ls_configure(lsffn.LS_CFG_DECODE_PATH, {"auto": 0, "kernels": 1, "fused": 2}[args.path])
    f.ls_configure(lsffn.LS_CFG_COOPERATIVE, int(args.launch == "cooperative"))
    keep_host = args.cpu_tokens > 0
    weights = []
    for l in range(cfg.n_layers):
        w = lsgen.layer_weights(cfg, l)
        f.ls_ffn_set_layer(l, w)
        weights.append(w if keep_host else None)
        if (l + 1) % 8 == 0:
            print(f"set-up: {l + 1}/{cfg.n_layers} layers", file=sys.stderr, flush=True)
    R = args.repeats
    xs = lsgen.tokens(cfg, 0, W + R * K, B)                  # [W+R*K, B, d] fp32, a fresh token per step
    x_dev = torch.from_numpy(xs).to(dev)                      # inputs resident in HBM
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t_setup

    kernel_ids = {"prenorm": lsffn.LS_K_PRENORM, "pred_p1": lsffn.LS_K_PRED_P1,
                  "pred_p2": lsffn.LS_K_PRED_P2, "select": lsffn.LS_K_SELECT,
                  "gateup": lsffn.LS_K_GATEUP, "down": lsffn.LS_K_DOWN,
                  "decode_fused": lsffn.LS_K_DECODE}

    def kernel_times():
        out = {}
        for name, kid in kernel_ids.items():
            ms, n = f.ls_kernel_timing(kid)
            if n:
                out[name] = {"total_ms": ms, "launches": n, "avg_us": 1e3 * ms / n}
        return out

    # streaming-read ceiling of this device, measured in the same run (1 GiB, 16-byte loads)
    probe = torch.ones(1 << 28, dtype=torch.int32, device=dev)
    ceil_best, ceil_med = f.ls_measure_read_bandwidth(probe, reps=10)
    del probe
    torch.cuda.synchronize()

    # warm-up; its second half (at most 16 steps; the first steps run cold) brackets every
    # launch with HIP events for the per-kernel breakdown
    n_bd = min(W // 2, 16)
    per_kernel = {}
    for i in range(W):
        if i == W - n_bd:
            torch.cuda.synchronize()
            f.ls_set_kernel_timing(True)
            f.ls_kernel_timing(0, reset=True)
        f.ls_decode_step(x_dev[i], B, cfg.k)
    torch.cuda.synchronize()
    f.ls_ffn_sync()                     # a device-side failure ends the run here
    if n_bd:
        per_kernel = kernel_times()
        f.ls_set_kernel_timing(False)

    # timed region: K decode steps; HIP event pairs bracket the launches of the dominant kernel
    # (the largest share of the warm-up's time), or of every kernel without a warm-up, in every
    # TIMING_SAMPLE_EVERY-th step: an event pair around a launch widens the gap before the next
    # one (the per-kernel path at batch 1 ran about 25% slower with a pair around every gate/up
    # launch), so the other steps run without them
    dom_name = max(per_kernel.items(), key=lambda kv: kv[1]["total_ms"])[0] if per_kernel else None
    timed_ids = [kernel_ids[dom_name]] if dom_name else None
    f.ls_kernel_timing(0, reset=True)
    # R repetitions of exactly K steps, each between synchronisations; each step decodes a
    # fresh token
    walls, gpu_mss = [], []
    for rep in range(R):
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ev0.record(stream)
        for i in range(K):
            sample = i % TIMING_SAMPLE_EVERY == 0
            if sample:
                f.ls_set_kernel_timing(True, kernels=timed_ids)
            f.ls_decode_step(x_dev[W + rep * K + i], B, cfg.k)
            if sample:
                f.ls_set_kernel_timing(False)
        ev1.record(stream)
        torch.cuda.synchronize()
        walls.append(time.perf_counter() - t0)
        gpu_mss.append(ev0.elapsed_time(ev1))
    f.ls_ffn_sync()
    order = sorted(range(R), key=lambda r: walls[r])
    med = order[R // 2]
    wall, gpu_ms = walls[med], gpu_mss[med]
    live = kernel_times()
    f.ls_set_kernel_timing(False)
    if not per_kernel:
        per_kernel = live
        dom_name = max(per_kernel.items(), key=lambda kv: kv[1]["total_ms"])[0]

    step_s = wall / K
    tok_s = B * K / wall
    if B == 1:
        U = float(cfg.k)
    else:
        # union sizes of the timed steps: an untimed replay through the per-call entry points
        # (ls_decode_step equals their composition) with the same inputs
        U = mean_union_size(f, cfg, x_dev[W:W + K], B, lsffn, torch)
    bytes_step = int(round(sum(algorithmic_bytes_per_layer(cfg, U) for _ in range(cfg.n_layers))))
    eff_gbs = bytes_step / step_s / 1e9
    # the same bytes split: FFN blocks and bias only, and with the predictor counted as the two
    # factors P1, P2 in the weight type (the specification's formula) instead of as stored
    ffn_only = int(round(cfg.n_layers * (algorithmic_bytes_per_layer(cfg, U) - predictor_bytes(cfg))))
    factors = cfg.elem_bytes * (cfg.rank * cfg.d_model + cfg.n_blk * cfg.rank)
    with_factors = ffn_only + cfg.n_layers * factors

    # dominant kernel: its algorithmic bytes per launch over its launch time in the timed region
    s = cfg.elem_bytes
    per_launch_bytes = {
        "gateup": int(s * (U * cfg.block * cfg.d_model * 2 + (U * cfg.block if cfg.gate_bias else 0))),
        "down": int(s * U * cfg.block * cfg.d_model),
        "pred_p1": predictor_bytes(cfg) if predictor_bytes(cfg) < s * (cfg.d_model * cfg.rank + cfg.rank * cfg.n_blk)
                   else s * cfg.d_model * cfg.rank,
        "pred_p2": s * cfg.rank * cfg.n_blk,
        "decode_fused": bytes_step,
    }
    dom_t = live[dom_name]
    dom_bytes = per_launch_bytes.get(dom_name)
    roofline = None
    if dom_bytes:
        achieved = dom_bytes / (dom_t["avg_us"] * 1e-6) / 1e9
        roofline = {"bound": "hbm", "kernel": dom_name, "achieved": round(achieved, 1),
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                    "measured_ceiling_GBs": round(ceil_best, 1),
                    "frac_of_measured_ceiling": round(achieved / ceil_best, 4),
                    "traffic": measured_traffic(dom_name, cfg, args.layers in (0, lsgen.CONFIGS[args.config].n_layers)),
                    "bytes_per_launch": dom_bytes,
                    "avg_launch_us": round(dom_t["avg_us"], 3)}

    check = None
    if B == 1 and args.check:
        check = check_fused_against_kernels(f, cfg, xs[W + R * K - 1], lsffn, torch, dev)
        if check is not None and not check["ok"]:
            print(f"output check failed: {check}", file=sys.stderr)
            return 1

    cpu = None
    if args.cpu_tokens > 0:
        cpu = cpu_baseline(cfg, weights, xs, min(args.cpu_tokens, W + R * K), B)

    out = {
        "metric": "sparse-FFN decode tokens/sec and effective weight GB/s (% HBM peak), 1 GPU",
        "value": round(tok_s, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(1e3 * step_s, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": lsgen.DTYPE_NAMES[cfg.dtype],
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.n_layers} layers, d_model {cfg.d_model}, "
                               f"d_ff {cfg.d_ff}, block {cfg.block} (k={cfg.k} of {cfg.n_blk}), "
                               f"rank {cfg.rank}, batch {B}",
                   "global_batch": B, "seq_len": 1, "parallelism": "none (1 GPU)",
                   "decode_path": args.path, "launch": args.launch},
        "effective_weight_GBs": round(eff_gbs, 1),
        "hbm_frac_of_peak": round(eff_gbs / HBM_PEAK_GBS, 4),
        "algorithmic_bytes_per_step": bytes_step,
        "bytes_per_step": {"ffn_only": ffn_only, "ffn_plus_predictor_as_stored": bytes_step,
                           "ffn_plus_predictor_factors": with_factors},
        "hbm_frac_of_peak_factors_counted": round(with_factors / step_s / 1e9 / HBM_PEAK_GBS, 4),
        "blocks_per_layer": round(U, 2),
        "gpu_event_ms": round(gpu_ms, 3),
        "repeats": {"n": R, "ms_per_step_median": round(1e3 * walls[med] / K, 4),
                    "ms_per_step_min": round(1e3 * min(walls) / K, 4),
                    "tokens_per_s_median": round(B * K / walls[med], 2),
                    "tokens_per_s_max": round(B * K / min(walls), 2)},
        "hbm_read_ceiling_GBs": {"best": round(ceil_best, 1), "median": round(ceil_med, 1),
                                 "how": "ls_measure_read_bandwidth: 1 GiB, 16-byte nontemporal loads, "
                                        "8 workgroups per CU, 10 launches"},
        "output_check": check,
        "kernels": {k: {kk: round(vv, 3) if isinstance(vv, float) else vv for kk, vv in v.items()}
                    for k, v in per_kernel.items()},
        "kernels_from": (f"the last {n_bd} warm-up steps, every launch bracketed by HIP events" if n_bd
                         else "the timed steps, every launch bracketed by HIP events"),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "setup_s": round(setup_s, 1),
    }
    print(json.dumps(out))
    f.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
