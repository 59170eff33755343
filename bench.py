"""Routed sparse-MLP decode throughput on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c2]

A step is one call of ``sats_mlp_forward`` on one decode batch: routing,
gate projection, SiLU + threshold + compaction, up-projection over the kept
rows and the gathered down-projection with its two-stage reduction.  The
default workload is one Llama-3.1-8B-shaped gated-MLP layer (d=4096,
d_ff=14336, bf16 weights N(0, 0.02^2)), decode batch 1, every token on the
sparse path, threshold = CATS 50th percentile over 1024 seeded calibration
tokens.  Inputs are synthetic and resident in HBM before timing starts.

To keep the 256 MB Infinity Cache from serving weights, the step rotates over
several copies of the layer's weights at different addresses (identical
bytes, so identical results).  The same steps are timed for
``sats_mlp_dense`` (base path) to give the speedup over dense.

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "routed sparse-MLP decode tok/s at 8B shape; achieved HBM GB/s; speedup vs dense"
GOLDEN = os.path.join(ROOT, "tests", "golden", "thresholds.json")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=2000)
    p.add_argument("--warmup", type=int, default=100)
    p.add_argument("--workload", default="c2")
    p.add_argument("--copies", type=int, default=8, help="weight copies rotated to defeat the MALL")
    p.add_argument("--tokens", type=int, default=64, help="distinct decode tokens cycled over")
    p.add_argument("--cpu-sample", type=int, default=1024, help="tokens the CPU oracle is timed on")
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--no-dense", action="store_true")
    p.add_argument("--batch", type=int, default=0, help="decode batch of a stack workload (default: its first)")
    p.add_argument("--cal-rows", type=int, default=1024, help="calibration rows (sats-calib workload)")
    p.add_argument("--lora-rank", type=int, default=0,
                   help="single-layer workloads: run the LoRA-aware sparse path with adapters of this rank")
    p.add_argument("--lora-scale", type=float, default=2.0)
    p.add_argument("--batch-path", default="auto", choices=["auto", "mfma", "split", "compact"],
                   help="kernels of batched calls (sats_set_options batch_path)")
    p.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                   help="only run a plain device copy of this many MiB (counter calibration)")
    return p.parse_args()


def copy_probe(mib):
    """A plain copy kernel of known size: HBM counters of it calibrate the counter scale."""
    import torch
    n = mib * 1024 * 1024 // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": n * 4, "copy_probe_bytes_written": n * 4, "launches": 5}))


def counter_traffic(kernel, workload_tag):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary (FETCH_SIZE and WRITE_SIZE, each scaled by a plain copy of known
    size), or None when there is none or the kernel source has changed since
    the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload_tag}_counters.txt")
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            k, sep, v = line.partition(":")
            if sep:
                fields[k.strip()] = v.strip()
    src = os.path.join(ROOT, "paper_2607_08991_amd", "csrc", fields.get("kernel_source", "decode.hpp"))
    if not os.path.exists(src):
        return None
    with open(src, "rb") as f:
        now = hashlib.sha256(f.read()).hexdigest()
    if fields.get("kernel_source_sha256") != now or "traffic_bytes_per_launch" not in fields:
        return None
    return int(float(fields["traffic_bytes_per_launch"]))


def thresholds_for(cfg):
    with open(GOLDEN) as f:
        return np.asarray(json.load(f)[cfg.name]["thresholds"], np.float32)


def cpu_baseline(cfg, weights_np, ts, x_np, n_sample, adapters=None, scale=0.0):
    """The CPU oracle, as it is, on the first n_sample decode tokens (the
    LoRA-aware oracle when adapters are given)."""
    from oracle import lora, mlp  # test infrastructure: only this leg of the benchmark uses it
    try:
        from threadpoolctl import threadpool_info
        blas = [(i.get("internal_api"), i.get("num_threads")) for i in threadpool_info()]
    except Exception:  # pragma: no cover
        blas = []
    cores = len(os.sched_getaffinity(0))
    threads = max([t for _, t in blas if t] or [1])
    wg, wu, wd = weights_np
    x = x_np[:n_sample]
    t0 = time.perf_counter()
    if adapters is None:
        mlp.forward(x, np.zeros(len(x), np.int32), wg[None], wu[None], wd[None], ts, None, cfg.dtype)
    else:
        lora.forward_lora(x, np.zeros(len(x), np.int32), wg[None], wu[None], wd[None],
                          tuple(m[None] for m in adapters), scale, ts, None, cfg.dtype)
    dt = time.perf_counter() - t0
    return {"value": round(len(x) / dt, 3), "unit": "tok/s", "cores": int(min(threads, cores)),
            "kind": "oracle",
            "sample": f"{len(x)} decode tokens of the same workload through the float64 numpy oracle "
                      f"(weights decoded once per call); {dt:.1f} s; host has {cores} cores; "
                      f"BLAS {blas}"}


def cpu_baseline_stack(cfg, Wnp, ts, lut, x_np, ids_np):
    """The CPU oracle, as it is, on a sample of decode tokens through every
    layer of a stack: route, then layer by layer (each layer's stored
    weights decoded once for the sample), the glue between layers."""
    from oracle import mlp, numerics  # test infrastructure: only this leg of the benchmark uses it
    cores = len(os.sched_getaffinity(0))
    n = len(x_np)
    t0 = time.perf_counter()
    r = mlp.route(ids_np, lut)
    hs = [numerics.decode(x_np[i], cfg.dtype) for i in range(n)]
    for l in range(cfg.n_layers):
        wg, wu, wd = (numerics.decode(w[l], cfg.dtype) for w in Wnp)
        for i in range(n):
            y = mlp.layer(hs[i], wg, wu, wd, float(ts[l]), bool(r[i]))[0]
            hs[i] = mlp.glue(y, cfg.dtype) if l < cfg.n_layers - 1 else numerics.rho(y, cfg.dtype)
    dt = time.perf_counter() - t0
    return {"value": round(n / dt, 4), "unit": "tok/s", "cores": cores, "kind": "oracle",
            "sample": f"{n} decode tokens of the workload ({int(r.sum())} base-routed) through all "
                      f"{cfg.n_layers} layers of the float64 numpy oracle, each layer's weights decoded once "
                      f"for the sample; {dt:.1f} s on a host with {cores} cores"}


def bench_stack(args, cfg):
    """A 32/36-layer workload: one step = one call on one decode batch through every layer."""
    import torch
    import paper_2607_08991_amd as sats
    from workloads import synth

    batch = args.batch or cfg.batches[0]
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    ts = thresholds_for(cfg)
    d, d_ff, L, esz = cfg.d, cfg.d_ff, cfg.n_layers, cfg.elem_bytes
    log(f"[bench] generating {cfg.name} weights ({L} layers)")
    W = []
    Wnp = synth.stack_weights(cfg.seed, L, d, d_ff, cfg.dtype)
    for w in Wnp:
        W.append(torch.from_numpy(w.view(np.int16)).view(torch.bfloat16).to(dev))
    W[0] = W[0].transpose(-1, -2).contiguous()  # the library takes W_gate one row per neuron
    if args.no_cpu:
        del Wnp
    slots = max(1, args.tokens // batch)
    X = torch.from_numpy(synth.decode_x(cfg, slots * batch, idx=batch).view(np.int16)).view(
        torch.bfloat16).to(dev).view(slots, batch, d)
    ids = torch.from_numpy(synth.token_ids(cfg, slots * batch, idx=batch)).to(dev).view(slots, batch)
    lut = synth.config_lut(cfg)
    dlut = torch.from_numpy(lut).to(dev)
    thr = torch.from_numpy(ts).to(dev)
    out = torch.empty((slots, batch, d), dtype=torch.bfloat16, device=dev)
    stream = torch.cuda.current_stream()
    R = args.lora_rank
    AD = None
    if R:  # rank-R adapters of every layer on the sparse path
        AD = [torch.from_numpy(m.view(np.int16)).view(torch.bfloat16).to(dev)
              for m in synth.stack_lora_adapters(cfg.seed, L, d, d_ff, R, cfg.dtype)]

    def forward(k, lora, **inspect):
        if lora:
            sats.sats_mlp_forward_lora(X[k], ids[k], *W, AD, R, args.lora_scale, thr, dlut, out[k], batch, d, d_ff,
                                       L, stream, **inspect)
        else:
            fn = sats.sats_mlp_forward_inspect if inspect else sats.sats_mlp_forward
            fn(X[k], ids[k], *W, thr, dlut, out[k], batch, d, d_ff, L, stream, **inspect)

    # per slot: routes and the union of kept columns per layer (algorithmic bytes)
    union = np.zeros((slots, L))
    kept = []
    routes = []
    idx = torch.empty((L, batch, d_ff), dtype=torch.int32, device=dev)
    cnt = torch.empty((L, batch), dtype=torch.int32, device=dev)
    route = torch.empty(batch, dtype=torch.uint8, device=dev)
    ar = torch.arange(d_ff, device=dev)
    for s in range(slots):
        forward(s, bool(R), route_out=route, active_count=cnt, active_idx=idx)
        valid = ar[None, None, :] < cnt[:, :, None].long()
        m = torch.zeros((L, d_ff), dtype=torch.bool, device=dev)
        for l in range(L):
            m[l, idx[l][valid[l]].long()] = True
        union[s] = m.sum(dim=1).cpu().numpy()
        kept.append(cnt.cpu().numpy())
        routes.append(route.cpu().numpy().copy())
    torch.cuda.synchronize()
    routes = np.array(routes)
    kept = np.array(kept, dtype=np.float64)  # [slots][L][batch]

    sel = None  # timed slots (default: all of them, in turn)

    def step(s, dense=False, lora=bool(R)):
        k = s % slots if sel is None else sel[s % len(sel)]
        if dense:
            sats.sats_mlp_dense(X[k], *W, out[k], batch, d, d_ff, L, stream)
        else:
            forward(k, lora)

    def timed(dense=False, lora=bool(R), steps=args.steps, warmup=args.warmup, kinds=()):
        for s in range(warmup):
            step(s, dense, lora)
        torch.cuda.synchronize()
        for k in kinds:
            sats.sats_timing_begin(k, steps * L * ((batch + 63) // 64))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for s in range(steps):
            step(warmup + s, dense, lora)
        e1.record(stream)
        torch.cuda.synchronize()
        sats.sats_device_status(stream)  # raises if a bounded device-side wait gave up: the timing is void
        if kinds:
            kt = {}
            for k in kinds:
                tot, c = sats.sats_timing_end(k)
                if c:
                    kt[sats.sats_kernel_name(k)] = (tot / c, c / steps)
            return e0.elapsed_time(e1) / steps, kt
        return e0.elapsed_time(e1) / steps

    ms = timed()
    # batches whose every token takes the sparse path: timed on their own, against the dense path
    all_sparse = None
    if batch > 1 and not args.no_dense:
        sparse_slots = [k for k in range(slots) if not routes[k].any()]
        if sparse_slots:
            sel = sparse_slots
            a_ms, a_dense = timed(), timed(True)
            sel = None
            all_sparse = {"slots": len(sparse_slots), "of_slots": slots, "ms_per_step": round(a_ms, 5),
                          "dense_ms_per_step": round(a_dense, 5), "speedup_vs_dense": round(a_dense / a_ms, 4),
                          "union_fraction_per_layer_mean": round(float(union[sparse_slots].mean() / d_ff), 4)}
    kinds = (sats.SATS_K_DEC_LAYER, sats.SATS_K_DEC_REDUCE, sats.SATS_K_DEC_LORA_V, sats.SATS_K_DEC_REDUCE_LORA,
             sats.SATS_K_DENSE, sats.SATS_K_DENSE_DOWN, sats.SATS_K_GATE, sats.SATS_K_UP, sats.SATS_K_DOWN,
             sats.SATS_K_LORA_V)
    ms_ev, kt = timed(kinds=kinds)
    dense_ms = None if args.no_dense else timed(True)
    lora_res = None
    if R:
        plain_ms = timed(lora=False)
        per_token_ms = None
        if batch > 1:  # the same batch token after token on the single-token path (a few steps: it is slow)
            with sats.options(lora_per_token=1):
                per_token_ms = timed(steps=min(args.steps, 3), warmup=1)
        lora_res = {"rank": R, "scale": args.lora_scale, "plain_sparse_ms_per_step": round(plain_ms, 5),
                    "overhead_vs_plain_sparse": round(ms / plain_ms, 4),
                    "token_by_token_ms_per_step": None if per_token_ms is None else round(per_token_ms, 5),
                    "speedup_vs_token_by_token": None if per_token_ms is None else round(per_token_ms / ms, 3)}
    sl = (args.warmup + np.arange(args.steps)) % slots
    alg = (L * d * d_ff * esz + 2 * d * esz * union[sl].sum(axis=1)).mean() + 2 * batch * d * esz
    if R:  # the adapters: A_gate, A_up, B_gate and B_down whole; B_up_T and A_down whole on the batched path
        alg += L * (2 * d * R + 3 * d_ff * R + R * d) * esz if batch > 1 else \
            L * (2 * d * R + R * d_ff + R * d) * esz + 2 * R * esz * union[sl].sum(axis=1).mean()
    sparse_mask = routes[sl] == 0
    sp = 1.0 - (kept[sl].transpose(0, 2, 1)[sparse_mask].mean() / d_ff) if sparse_mask.any() else None
    # each layer's realized sparsity over the sparse-routed tokens of the timed steps
    sp_layer = ([round(float(1.0 - kept[sl].transpose(0, 2, 1)[sparse_mask][:, l].mean() / d_ff), 4)
                 for l in range(L)] if sparse_mask.any() else None)
    # per-kernel algorithmic bytes of one launch, averaged over the timed launches
    rows_mean = float(kept[sl].mean())  # kept rows of a token (all d_ff for a base-routed one)
    per_launch = {"dec_layer_kernel": d * d_ff * esz + d * esz + 2 * d * esz * rows_mean,
                  "dec_reduce_kernel": d * esz, "dense_gateup_kernel": 2 * d * d_ff * esz,
                  "dense_down_kernel": d * d_ff * esz}
    kern = {}
    for name, (kms, per_step) in kt.items():
        b = per_launch.get(name)
        kern[name] = {"avg_us": round(kms * 1e3, 3), "launches_per_step": round(per_step, 3),
                      "algorithmic_bytes_per_launch": None if b is None else int(b),
                      "achieved_gbps": None if b is None else round(b / (kms * 1e-3) / 1e9, 1)}
    dom = max((k for k in kern if kern[k]["achieved_gbps"] is not None),
              key=lambda k: kern[k]["avg_us"] * kern[k]["launches_per_step"])
    cpu = None
    if not args.no_cpu:
        ns = min(8, slots * batch)
        log(f"[bench] timing the CPU oracle on {ns} tokens through {L} layers")
        cpu = cpu_baseline_stack(cfg, Wnp, ts, lut, X.view(-1, d)[:ns].view(torch.int16).cpu().numpy().view(np.uint16),
                                 ids.view(-1)[:ns].cpu().numpy())
        del Wnp
    res = {
        "metric": METRIC, "value": round(batch * 1e3 / ms, 2), "unit": "tok/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": cfg.name + (f", LoRA rank {R} on the sparse path" if R else ""),
                   "d": d, "d_ff": d_ff, "n_layers": L, "decode_batch": batch, "batch_path": args.batch_path,
                   "route": "route_lut", "base_routed_ids": cfg.n_dense_ids, "vocab": cfg.vocab},
        "algorithmic_bytes_per_step": int(alg),
        "hbm_gbps_algorithmic": round(alg / (ms * 1e-3) / 1e9, 1),
        "hbm_frac_algorithmic": round(alg / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
        "realized_sparsity_sparse_tokens": None if sp is None else round(float(sp), 4),
        "realized_base_routed_fraction": round(float(routes[sl].mean()), 4),
        "realized_sparsity_per_layer": sp_layer,
        "all_sparse_steps": all_sparse,
        "dense_ms_per_step": None if dense_ms is None else round(dense_ms, 5),
        "speedup_vs_dense": None if dense_ms is None else round(dense_ms / ms, 4),
        "ms_per_step_with_kernel_events": round(ms_ev, 5),
        "kernels": kern,
        "roofline": {"kernel": dom, "bound": "hbm", "achieved": kern[dom]["achieved_gbps"], "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(kern[dom]["achieved_gbps"] / HBM_PEAK_GBPS, 4),
                     "traffic": counter_traffic(dom, f"{cfg.name}_b{batch}")},
        "cpu_baseline": cpu,
    }
    if lora_res:
        res["lora"] = lora_res
    print(json.dumps(res), flush=True)


BF16_MFMA_PEAK_TFLOPS = 2500.0


def bench_calib(args):
    """SATS calibration of one Llama-3.1-8B-shaped layer (Eq. 6 curves at the
    coarse grid of 20 Eq. 3 levels over `--cal-rows` calibration rows): one
    step is one sats_calibration_curves call."""
    import torch
    import paper_2607_08991_amd as sats
    from workloads import get_config, synth
    from oracle import sats as osats, numerics  # test infrastructure: the cpu_baseline leg only

    cfg = get_config(1)
    d, d_ff, n = cfg.d, cfg.d_ff, args.cal_rows
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    log(f"[bench] generating {cfg.name} weights and {n} calibration rows")
    wnp = synth.layer_weights(cfg.seed, 0, d, d_ff, cfg.dtype)
    W = [torch.from_numpy(w.view(np.int16)).view(torch.bfloat16).to(dev) for w in wnp]
    W[0] = W[0].t().contiguous()  # the library takes W_gate one row per neuron
    xnp = synth.activations(cfg.seed, synth.S_CAL, n, d, cfg.dtype)
    X = torch.from_numpy(xnp.view(np.int16)).view(torch.bfloat16).to(dev)
    levels = [0.0] + [round(0.05 * i, 4) for i in range(1, 20)]
    K = len(levels)
    stream = torch.cuda.current_stream()
    for _ in range(max(1, args.warmup)):
        sats.sats_calibration_curves(X, *W, n, d, d_ff, levels)
    steps = max(1, args.steps)
    kinds = (sats.SATS_K_CAL_ERR, sats.SATS_K_CAL_GATEUP)
    for k in kinds:
        sats.sats_timing_begin(k, 64 * steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        t, err, sp = sats.sats_calibration_curves(X, *W, n, d, d_ff, levels)
    dt = (time.perf_counter() - t0) / steps
    kern = {}
    for k in kinds:
        tot, c = sats.sats_timing_end(k)
        kern[sats.sats_kernel_name(k)] = {"avg_us": round(tot / c * 1e3, 2), "launches_per_step": c // steps}
    # the library's products: candidates at or below 0 (no neuron removed)
    # take none; from the first positive one, 15 per product, the first with
    # y; a later one of at most 4 candidates packs 4 calibration rows per tile
    z = int(np.count_nonzero(np.asarray(t) <= 0))
    kcs, packs = [], []
    for k0 in range(z, K, 15):
        kc = min(15, K - k0)
        packs.append(4 if kcs and kc <= 4 else (2 if kc <= 7 else 1))
        kcs.append(kc)
    # algorithmic flops of the error products of one step: per calibration
    # row, a masked product for every positive candidate and y once, each
    # over d_ff x d; executed: hi and lo terms, 16 / pack MFMA rows per
    # calibration row and product
    alg_flops = 2.0 * n * (K - z + 1) * d_ff * d
    exe_flops = sum(2.0 * 2 * n * (16 // pk) * d_ff * d for pk in packs)
    e = kern["cal_err_kernel"]
    e_step_us = e["avg_us"] * e["launches_per_step"]
    achieved = alg_flops / (e_step_us * 1e-6) / 1e12
    e.update(candidates_per_launch=kcs, calibration_rows_per_tile=packs, algorithmic_flops_per_step=alg_flops,
             achieved_tflops=round(achieved, 1),
             executed_flops_per_step=exe_flops, executed_tflops=round(exe_flops / (e_step_us * 1e-6) / 1e12, 1))
    cpu = None
    if not args.no_cpu:
        rows = 4
        H = numerics.decode(xnp[:rows], cfg.dtype)
        Wd = [numerics.decode(w, cfg.dtype) for w in wnp]
        c0 = time.perf_counter()
        osats.err_curve(H, *Wd, t.astype(np.float64))
        cdt = time.perf_counter() - c0
        cores = len(os.sched_getaffinity(0))
        cpu = {"value": round(rows / cdt, 4), "unit": "calibration rows/s (20 candidates)", "cores": cores,
               "kind": "oracle",
               "sample": f"{rows} calibration rows x {K} candidates through the float64 oracle (Eq. 6 by "
                         f"masking), {cdt:.1f} s"}
    res = {
        "metric": "SATS calibration: Eq. 6 error curves of one layer", "value": round(n / dt, 1),
        "unit": "calibration rows/s (20 candidates)", "n_gpus": 1, "steps": steps, "warmup": args.warmup,
        "ms_per_step": round(dt * 1e3, 3), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16 (fp32 accumulate, p as bf16 hi + lo)", "data": "synthetic",
        "config": {"workload": f"sats_calib_{cfg.name}", "d": d, "d_ff": d_ff, "calibration_rows": n,
                   "candidates": K, "error_products": len(kcs)},
        "kernels": kern,
        "roofline": {"kernel": "cal_err_kernel", "bound": "mfma", "achieved": round(achieved, 1),
                     "peak": BF16_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / BF16_MFMA_PEAK_TFLOPS, 4), "traffic": None},
        "cpu_baseline": cpu,
        "realized_sparsity_at_candidates": [round(float(v), 5) for v in sp],
        "err_at_candidates": [round(float(v), 6) for v in err],
    }
    print(json.dumps(res), flush=True)


def bench_route(args):
    """Routing-table construction (Eq. 11-14) at the Llama-3.1 vocabulary (128256 ids):
    2^22 routing-corpus occurrences with base and sparse losses, 2^20 held-out ids,
    Zipf(1.1) ids, target routed fraction 0.5.  One step is one sats_route_table call."""
    import torch
    import paper_2607_08991_amd as sats
    from workloads import synth
    from oracle import route  # test infrastructure: the cpu_baseline leg only

    V, n, nh, r_tar = 128256, 1 << 22, 1 << 20, 0.5
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    log(f"[bench] generating a routing corpus of {n} occurrences")
    ids, lb, ls = synth.routing_corpus(11, n, V)
    held = synth.routing_corpus(11, nh, V, split=1)[0]
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    dids, dlb, dls, dheld = up(ids), up(lb), up(ls), up(held)
    table = torch.empty(V, dtype=torch.uint8, device=dev)
    for _ in range(max(1, args.warmup)):
        sats.sats_route_table(dlb, dls, dids, dheld, V, r_tar, table)
    steps = max(1, args.steps)
    # headline timing without per-kernel events; the kernels from a second,
    # identical region with events around the two accumulation launches
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        tau, r = sats.sats_route_table(dlb, dls, dids, dheld, V, r_tar, table)
    dt = (time.perf_counter() - t0) / steps
    kinds = (sats.SATS_K_ROUTE_ACCUM, sats.SATS_K_ROUTE_MERGE)
    for k in kinds:
        sats.sats_timing_begin(k, steps)
    for _ in range(steps):
        sats.sats_route_table(dlb, dls, dids, dheld, V, r_tar, table)
    kus = {}
    for k in kinds:
        tot, c = sats.sats_timing_end(k)
        kus[sats.sats_kernel_name(k)] = tot / c * 1e3
    alg = 12 * n  # one id and two float32 losses per occurrence, read once
    kernels = {}
    for name, us in kus.items():
        kernels[name] = {"avg_us": round(us, 2)}
    k_us = kus["route_part_kernel"]
    gbps = alg / (k_us * 1e-6) / 1e9
    kernels["route_part_kernel"].update({"algorithmic_bytes": alg, "achieved_gbps": round(gbps, 1)})
    kernels["route_merge_kernel"]["note"] = "adds the part kernel's per-chunk entries (implementation traffic)"
    cpu = None
    if not args.no_cpu:
        ns, nhs = 1 << 22, 1 << 17  # the whole routing split; the oracle's candidate loop is quadratic
        c0 = time.perf_counter()
        route.build(ids[:ns], lb[:ns], ls[:ns], held[:nhs], V, r_tar)
        cdt = time.perf_counter() - c0
        cpu = {"value": round(ns / cdt, 1), "unit": "routing occurrences/s", "cores": 1, "kind": "oracle",
               "sample": f"{ns} routing occurrences and {nhs} held-out ids through the oracle (Python loops "
                         f"over occurrences and candidate thresholds), {cdt:.1f} s"}
    res = {
        "metric": "routing-table construction (Eq. 11-14)", "value": round(n / dt, 1),
        "unit": "routing occurrences/s", "n_gpus": 1, "steps": steps, "warmup": args.warmup,
        "ms_per_step": round(dt * 1e3, 3), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32 losses, exact integer sums, f64 scores", "data": "synthetic",
        "config": {"workload": "route_table_llama_vocab", "vocab": V, "routing_occurrences": n,
                   "heldout_occurrences": nh, "ids": "Zipf(1.1)", "r_tar": r_tar},
        "tau": tau, "realized_routed_fraction": r,
        "kernels": kernels,
        "roofline": {"kernel": "route_part_kernel", "bound": "hbm", "achieved": round(gbps, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(gbps / HBM_PEAK_GBPS, 4), "traffic": None},
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(sharding is described in DESIGN.md); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    if args.copy_probe:
        copy_probe(args.copy_probe)
        return

    import torch
    import paper_2607_08991_amd as sats
    from workloads import get_config, synth

    sats.load()
    sats.sats_set_options(batch_path={"auto": sats.SATS_BATCH_AUTO, "mfma": sats.SATS_BATCH_MFMA,
                                      "split": sats.SATS_BATCH_SPLIT, "compact": sats.SATS_BATCH_COMPACT}[args.batch_path])
    if args.workload == "sats-calib":
        return bench_calib(args)
    if args.workload == "route-lut":
        return bench_route(args)
    cfg = get_config(args.workload)
    if cfg.n_layers != 1:
        return bench_stack(args, cfg)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    ts = thresholds_for(cfg)
    d, d_ff, L = cfg.d, cfg.d_ff, cfg.n_layers
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    esz = cfg.elem_bytes

    log(f"[bench] generating {cfg.name} weights")
    wnp = synth.layer_weights(cfg.seed, 0, d, d_ff, cfg.dtype)

    def up(a):
        a = np.ascontiguousarray(a)
        t = torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a)
        return t.view(tdt).to(dev) if a.dtype == np.uint16 else t.to(dev)

    base = [up(w) for w in wnp]
    base[0] = base[0].t().contiguous()  # the library takes W_gate one row per neuron
    R = args.lora_rank
    if R:  # the adapters travel with each weight copy
        base += [up(m) for m in synth.lora_adapters(cfg.seed, 0, d, d_ff, R, cfg.dtype)]
    copies = [base] + [[w.clone() for w in base] for _ in range(args.copies - 1)]
    xnp = synth.decode_x(cfg, args.tokens)
    X = up(xnp)
    lut = synth.config_lut(cfg)
    ids = torch.from_numpy(synth.token_ids(cfg, args.tokens)).to(dev)
    dlut = torch.from_numpy(lut).to(dev) if lut is not None else None
    thr = torch.from_numpy(ts).to(dev)
    out = torch.empty((args.tokens, d), dtype=tdt, device=dev)
    n = 1  # decode batch
    stream = torch.cuda.current_stream()

    # kept-row counts of every decode token (identical inputs -> identical counts in the timed run)
    cnt = torch.zeros((L, args.tokens), dtype=torch.int32, device=dev)
    route = torch.zeros(args.tokens, dtype=torch.uint8, device=dev)
    for i in range(args.tokens):
        if R:
            sats.sats_mlp_forward_lora(X[i:i + 1], ids[i:i + 1] if dlut is not None else None, *base[:3],
                                       base[3:], R, args.lora_scale, thr, dlut, out[i:i + 1], 1, d, d_ff, L,
                                       route_out=route[i:i + 1], active_count=cnt[:, i:i + 1])
        else:
            sats.sats_mlp_forward_inspect(X[i:i + 1], ids[i:i + 1] if dlut is not None else None,
                                          *base, thr, dlut, out[i:i + 1], 1, d, d_ff, L,
                                          route_out=route[i:i + 1], active_count=cnt[:, i:i + 1])
    torch.cuda.synchronize()
    kept = cnt.cpu().numpy().astype(np.float64)
    routed_base = route.cpu().numpy()

    def step_plain(s):
        i = s % args.tokens
        w = copies[s % args.copies]
        sats.sats_mlp_forward(X[i:i + 1], ids[i:i + 1] if dlut is not None else None, w[0], w[1],
                              w[2], thr, dlut, out[i:i + 1], n, d, d_ff, L, stream)

    def step_lora(s):
        i = s % args.tokens
        w = copies[s % args.copies]
        sats.sats_mlp_forward_lora(X[i:i + 1], ids[i:i + 1] if dlut is not None else None, w[0], w[1], w[2],
                                   w[3:], R, args.lora_scale, thr, dlut, out[i:i + 1], n, d, d_ff, L, stream)

    step_fwd = step_lora if R else step_plain

    def step_dense(s):
        i = s % args.tokens
        w = copies[s % args.copies]
        sats.sats_mlp_dense(X[i:i + 1], w[0], w[1], w[2], out[i:i + 1], n, d, d_ff, L, stream)

    def timed(fn, kinds=()):
        for s in range(args.warmup):
            fn(s)
        torch.cuda.synchronize()
        for k in kinds:
            sats.sats_timing_begin(k, args.steps)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for s in range(args.steps):
            fn(args.warmup + s)
        e1.record(stream)
        torch.cuda.synchronize()
        sats.sats_device_status(stream)  # raises if a bounded device-side wait gave up: the timing is void
        ms = e0.elapsed_time(e1) / args.steps
        kt = {}
        for k in kinds:
            tot, c = sats.sats_timing_end(k)
            if c:
                kt[sats.sats_kernel_name(k)] = (tot / c, c)
        return ms, kt

    log(f"[bench] timing {args.steps} steps (warmup {args.warmup}), {args.copies} weight copies")
    kinds = (sats.SATS_K_GATE, sats.SATS_K_UP, sats.SATS_K_DOWN, sats.SATS_K_DEC_LAYER, sats.SATS_K_DEC_LORA_V,
             sats.SATS_K_DEC_REDUCE, sats.SATS_K_DEC_REDUCE_LORA)
    # headline timing without per-kernel events (recording them costs a few us
    # per launch); per-kernel durations come from an identical second region
    ms, _ = timed(step_fwd)
    ms_ev, kt = timed(step_fwd, kinds)
    dense_ms = None
    if not args.no_dense:
        dense_ms, _ = timed(step_dense)
    plain_ms = timed(step_plain)[0] if R else None

    # algorithmic bytes: all of W_gate, the kept rows of W_up_T and W_down, x and out
    steps_idx = (args.warmup + np.arange(args.steps)) % args.tokens
    a_mean = float(kept[:, steps_idx].sum(axis=0).mean())           # kept rows per step (all layers)
    gate_bytes = d * d_ff * esz + n * d * esz
    updown_row = d * esz
    touched = L * d * d_ff * esz + 2 * updown_row * a_mean + 2 * n * d * esz
    # LoRA: A_gate, B_gate, A_up and B_down whole, the kept rows of B_up_T and A_down
    lora_bytes = L * (2 * d * R + R * d_ff + R * d) * esz + 2 * R * esz * a_mean if R else 0
    touched += lora_bytes
    gbps = touched / (ms * 1e-3) / 1e9
    sparsity = 1.0 - a_mean / (L * d_ff)

    up_bytes = updown_row * a_mean / L
    kern = {}
    # LoRA: B_gate at every column and B_up_T, A_down at the kept rows in the
    # layer launch; A_gate and A_up in the input launch; B_down in the reduction
    layer_lora = (R * d_ff * esz + 2 * R * esz * a_mean / L) if R else 0
    for name, (kms, c) in kt.items():
        b = {"gate_kernel": gate_bytes, "up_kernel": up_bytes, "down_kernel": up_bytes,
             "dec_layer_kernel": gate_bytes + 2 * up_bytes + layer_lora,
             "dec_lora_v_kernel": 2 * d * R * esz + n * d * esz,
             "dec_reduce_kernel": n * d * esz,
             "dec_reduce_lora_kernel": n * d * esz + R * d * esz}[name]
        kern[name] = {"avg_us": round(kms * 1e3, 3), "launches": c,
                      "algorithmic_bytes": int(b), "achieved_gbps": round(b / (kms * 1e-3) / 1e9, 1)}
    dom = max(kern, key=lambda k: kern[k]["avg_us"])
    dom_b = kern[dom]["algorithmic_bytes"]
    dom_gbps = dom_b / (kern[dom]["avg_us"] * 1e-6) / 1e9

    cpu = None
    if not args.no_cpu:
        log(f"[bench] timing the CPU oracle on {args.cpu_sample} tokens")
        ns = min(args.cpu_sample, 128) if R else args.cpu_sample  # the adapted oracle merges weights per token
        cpu = cpu_baseline(cfg, wnp, ts, synth.decode_x(cfg, ns), ns,
                           synth.lora_adapters(cfg.seed, 0, d, d_ff, R, cfg.dtype) if R else None, args.lora_scale)

    res = {
        "metric": METRIC,
        "value": round(1e3 / ms * n, 2),
        "unit": "tok/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": (f"{cfg.name}: one Llama-3.1-8B-shaped gated-MLP layer" if cfg.index == 1
                                else cfg.name) + (f", LoRA rank {R} on the sparse path" if R else ""),
                   "d": d, "d_ff": d_ff, "n_layers": L, "decode_batch": n,
                   "route": "all tokens sparse" if lut is None else "route_lut",
                   "threshold": [float(t) for t in ts], "target_sparsity": cfg.k_fixed,
                   "weight_copies_rotated": args.copies},
        "hbm_gbps_touched": round(gbps, 1),
        "hbm_frac_touched": round(gbps / HBM_PEAK_GBPS, 4),
        "touched_bytes_per_step": int(touched),
        "realized_sparsity": round(sparsity, 5),
        "realized_base_routed_fraction": float(routed_base.mean()),
        "ms_per_step_with_kernel_events": round(ms_ev, 6),
        "dense_ms_per_step": None if dense_ms is None else round(dense_ms, 6),
        "dense_hbm_gbps": None if dense_ms is None else
        round((3 * L * d * d_ff * esz + 2 * n * d * esz) / (dense_ms * 1e-3) / 1e9, 1),
        "speedup_vs_dense": None if dense_ms is None else round(dense_ms / ms, 4),
        "kernels": kern,
        "roofline": {"kernel": dom, "bound": "hbm", "achieved": round(dom_gbps, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(dom_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": counter_traffic(dom, "c2_llama_layer_bf16") if cfg.index == 1 and not R
                     else None},
        "cpu_baseline": cpu,
    }
    if R:
        res["lora"] = {"rank": R, "scale": args.lora_scale, "adapter_bytes_per_step": int(lora_bytes),
                       "plain_sparse_ms_per_step": round(plain_ms, 6),
                       "overhead_vs_plain_sparse": round(ms / plain_ms, 4)}
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
