#!/usr/bin/env python3
"""Tree-build throughput of the PCTree per-round builder on one MI355X.

One step = one full round of the hot path (Alg. 1): B sequential Markov
stages (batched parent-conditioned projection, row log-softmax, per-parent
top-k, path scores, frontier pruning), the global top-N and the emission of
tokens, parents, position ids and the ancestor mask.  Inputs are seeded
synthetic tensors of the Qwen3-4B large-block shape (V=151936, B=16, N=64,
k=8, r=256, bf16), resident in HBM before timing starts.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E peak, GB/s
METRIC = "tree-build rounds/sec + µs/round (V=151936,B=16,N=64); % peak HBM GB/s"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "round_kernel_traffic.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2608_02123_amd", "csrc", "pctree_kernels.hip")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_bytes(w, w_once=False):
    """Bytes one round must move (W and L_d streamed once per depth; the
    frontier's embedding rows and the depth features).  With ``w_once`` W
    counts once per round: the floor for a kernel that keeps W on chip
    across the B stages."""
    es = 2 if w.dtype == "bf16" else 4
    kk = min(w.k, w.V)
    sum_p = 1 + (w.B - 1) * kk  # frontier sizes b_0 = 1, b_d = k'
    return ((1 if w_once else w.B) * w.r * w.V * es  # W, shared by all requests
            + w.R * w.B * w.V * es          # L_d per request
            + w.R * sum_p * w.r * es        # E rows gathered for the frontier
            + w.R * w.B * w.r * 4)          # h_d


def spread(xs):
    """Median, 10th and 90th percentiles of a list of per-round times (us)."""
    if not xs:
        return None
    s = sorted(xs)

    def q(f):
        return s[min(len(s) - 1, int(round(f * (len(s) - 1))))]
    return {"median": q(0.5), "p10": q(0.1), "p90": q(0.9), "rounds": len(s)}


def time_rounds(launch, steps, cold_steps, flush):
    """Per-round durations (us) from events around each launch: ``steps``
    back-to-back (warm) rounds, then ``cold_steps`` rounds each after a write
    of ``flush`` (512 MiB, larger than the 256 MB Infinity Cache, as the
    target model's forward would evict W), outside the events."""
    import torch

    def pairs(n, before=None):
        ev = []
        for _ in range(n):
            if before is not None:
                before()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            launch()
            b.record()
            ev.append((a, b))
        torch.cuda.synchronize()
        return [a.elapsed_time(b) * 1000.0 for a, b in ev]

    warm = pairs(steps)
    cold = pairs(cold_steps, before=lambda: flush.add_(1)) if cold_steps else []
    return warm, cold


def time_config(P, name, steps, cold_steps, flush):
    """us/round (warm and cold) and the fraction of the HBM roofline of one
    more workload, with the same timing as the headline."""
    import torch
    from paper_2608_02123_amd.synth import CONFIGS, make_inputs

    w = CONFIGS[name]
    log(f"[bench] workload {name}")
    inp = make_inputs(w)
    dev = P.device_inputs(inp)
    b = P.TreeBuilder(w.V, w.B, w.N, w.k, w.r, w.R, P.BF16 if w.dtype == "bf16" else P.F32,
                      mask=True)
    b.bind(**dev)
    for _ in range(5):
        b.launch()
    torch.cuda.synchronize()
    warm, cold = time_rounds(b.launch, steps, cold_steps, flush)
    out = b.launch(check=True)
    nbytes = algorithmic_bytes(w)
    ws, cs = spread(warm), spread(cold)
    res = {"workload": f"V={w.V} B={w.B} N={w.N} k={w.k} r={w.r} R={w.R} {w.dtype}",
           "warm_us": ws, "cold_us": cs, "algorithmic_bytes": nbytes,
           "w_once_bytes": algorithmic_bytes(w, w_once=True),
           "frac": nbytes / (ws["median"] * 1e-6) / 1e9 / HBM_PEAK_GBS,
           "cold_frac": (nbytes / (cs["median"] * 1e-6) / 1e9 / HBM_PEAK_GBS) if cs else None,
           "count": [int(c) for c in out["count"].cpu()]}
    del b, dev, inp
    torch.cuda.empty_cache()
    return res


def kernel_hash():
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic():
    """HBM bytes per dominant-kernel launch from rocprofv3 counters, if taken on
    the current kernel source; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256_16") != kernel_hash():
        return None
    return t.get("bytes_per_launch")


def cpu_baseline(inp, w, seconds):
    """The CPU oracle as it stands, timed on this host on whole rounds."""
    import numpy as np
    from oracle import pctree_oracle as O

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # noqa: BLE001
        threads = 1
    W64 = inp["W"].astype(np.float64)
    n, t0 = 0, time.perf_counter()
    while True:
        O.build_tree(inp["L"][0], inp["E"], W64, inp["h"][0], int(inp["root"][0]),
                     int(inp["prefix_len"][0]), w.k, w.N, w.dtype)
        n += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    return {"value": n / el, "unit": "rounds/s", "cores": threads, "kind": "oracle",
            "sample": f"{n} whole rounds of request 0 of {w.name} (all "
                      f"{1 + (w.B - 1) * min(w.k, w.V)} child-logit rows materialised, float64) "
                      f"in {el:.1f} s; BLAS threads {threads}, os.cpu_count() {os.cpu_count()}"}


def _event_us(fn, reps):
    import torch

    fn()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        fn()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) * 1000.0 / reps


def time_verify(P, builder, w, inp, reps=200):
    """The verification steps after one round of the workload: retrieve rows,
    greedy acceptance against synthetic target predictions, and compaction of
    a Qwen3-4B-shaped KV cache (36 layers x K/V, 8 KV heads x 128 dims, bf16)."""
    import numpy as np
    import torch
    from paper_2608_02123_amd.synth import target_next

    log("[bench] verification steps")
    out = builder.launch()
    torch.cuda.synchronize()
    tok = out["token"].cpu().numpy()
    par = out["parent"].cpu().numpy()
    cnt = out["count"].cpu().numpy()
    rng = np.random.default_rng(1)
    tn = np.stack([target_next(rng, tok[i], par[i], int(cnt[i]), w.V, 0.8)
                   for i in range(w.R)])
    tn = torch.from_numpy(tn).cuda()
    groups, slot = 72, 8 * 128
    prefix = inp["prefix_len"]
    cap = int(prefix.max()) + w.N
    cache = torch.zeros(w.R, groups, cap, slot, dtype=torch.bfloat16, device="cuda")
    pre = torch.from_numpy(prefix).cuda()
    rows, nrows = P.build_retrieve(out["parent"], out["count"], w.B)
    acc = P.accept_greedy(out["token"], rows, nrows, tn)
    torch.cuda.synchronize()
    a_len = acc["accept_len"].cpu().numpy()
    nodes = acc["accept_node"].cpu().numpy()
    moved = sum(int(sum(1 for m in range(a_len[i] + 1) if nodes[i, m] != m)) for i in range(w.R))
    # the C entry points with their arguments marshalled once, so that the
    # events see the kernels rather than the Python wrappers
    import ctypes
    L = P.lib()
    vp = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    ra = (vp(out["parent"]), vp(out["count"]), w.R, w.N, w.B, vp(rows), vp(nrows), st)
    aa = (vp(out["token"]), vp(rows), vp(nrows), vp(tn), w.R, w.N, w.B, vp(acc["accept_len"]),
          vp(acc["accept_row"]), vp(acc["accept_node"]), vp(acc["bonus"]), st)
    es = cache.element_size()
    ca = (vp(cache), cache.stride(0) * es, cache.stride(1) * es, groups, cap, slot * es, vp(pre),
          vp(acc["accept_node"]), vp(acc["accept_len"]), w.R, w.N, w.B, st)
    us_r = _event_us(lambda: L.pctree_build_retrieve(*ra), reps)
    us_a = _event_us(lambda: L.pctree_accept_greedy(*aa), reps)
    us_c = _event_us(lambda: L.pctree_compact_kv(*ca), reps)
    attn = time_attention(P, out, w, prefix, reps)
    return {"retrieve_us": us_r, "accept_us": us_a, "compact_us": us_c,
            "accept_len": [int(x) for x in a_len], "nrows": [int(x) for x in nrows.cpu()],
            "compact_bytes": 2 * moved * groups * slot * 2,
            "kv": "72 groups (36 layers x K/V) x 8 heads x 128 dims bf16 per slot",
            "target": "synthetic: a child's token with p = 0.8 at each node, else uniform",
            "attention": attn}


def time_attention(P, out, w, prefix, reps):
    """One tree-masked attention layer of the target's verification forward on
    the round's own tree: Qwen3 attention shapes (32 query / 8 key-value heads,
    or 40 / 8 for the 14B batch), head dimension 128, bf16, over each
    request's prefix and tree slots."""
    import ctypes

    import numpy as np
    import torch
    from paper_2608_02123_amd import synth

    Hq, Hkv, D = synth.ATTN_SHAPES["qwen3_14b" if w.R > 1 else "qwen3_4b"]
    cnt = out["count"].cpu().numpy().astype(np.int64)
    pre = np.asarray(prefix, dtype=np.int64)
    C = int((pre + w.N).max())
    t = synth.make_attention_inputs(np.random.default_rng(3), w.R, w.N, Hq, Hkv, D, pre, cnt, C)
    t["k"] = np.nan_to_num(t["k"])  # slots nobody reads: zeros rather than NaN
    t["v"] = np.nan_to_num(t["v"])

    def up(a):
        return torch.from_numpy(synth.bf16_bits(a).view(np.int16)).cuda().view(torch.bfloat16)

    q, k, v = up(t["q"]), up(t["k"]), up(t["v"])
    att = P.TreeAttention(w.R, w.N, Hq, Hkv, D, C, D ** -0.5)
    pre_d = torch.from_numpy(pre.astype(np.int32)).cuda()
    res = att(q, k, v, out["mask"], out["count"], pre_d)
    torch.cuda.synchronize()
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    vp = lambda x: ctypes.c_void_p(x.data_ptr())  # noqa: E731
    args = (ctypes.byref(att.shape), vp(q), vp(k), vp(v), vp(out["mask"]), vp(out["count"]),
            vp(pre_d), vp(res), vp(att.workspace), att.ws_bytes, st)
    L = P.lib()
    us = _event_us(lambda: L.pctree_tree_attention(*args), reps)
    # algorithmic traffic: each admitted range of K and V read once per kv head,
    # the queries read and the outputs written once
    slots = int((pre + cnt).sum())
    nodes = int(cnt.sum())
    bytes_ = 2 * Hkv * slots * D * 2 + 2 * nodes * Hq * D * 2
    # flops: q.k and p.v over every admitted slot of every (node, head)
    mask = out["mask"].cpu().numpy().view(np.uint32)
    tree_adm = sum(int(sum(bin(int(x)).count("1") for x in mask[r, :cnt[r]].ravel()))
                   for r in range(w.R))
    adm = int(sum(pre[r] * cnt[r] for r in range(w.R))) + tree_adm
    flops = 4 * adm * Hq * D
    return {"us": us, "heads": f"{Hq}/{Hkv}x{D}", "capacity": C,
            "algorithmic_bytes": bytes_, "gbs": bytes_ / us / 1e3,
            "hbm_frac": bytes_ / us / 1e3 / HBM_PEAK_GBS,
            "flops": flops, "tflops": flops / us / 1e6, "mfma_frac": flops / us / 1e6 / 2500.0,
            "splits": att.ws_bytes > 0}


def time_sweeps(P, w, inp, dev, reps=30):
    """us/round of the two control scorings (Sec. 5.3) and of k and N sweeps
    (the paper's ablations over the branching factor and the budget)."""
    import torch

    log("[bench] sweeps")
    dt = P.BF16 if w.dtype == "bf16" else P.F32

    def us(k, N, mode=P.MODE_PARENT):
        b = P.TreeBuilder(w.V, w.B, N, k, w.r, w.R, dt, mask=True, mode=mode)
        b.bind(**dev)
        for _ in range(3):
            b.launch()
        return _event_us(b.launch, reps)

    return {
        "modes_us": {"parent": us(w.k, w.N), "shared": us(w.k, w.N, P.MODE_SHARED),
                     "independent": us(w.k, w.N, P.MODE_INDEPENDENT)},
        "k_us": {str(k): us(k, w.N) for k in (1, 2, 4, 8, 16)},
        "N_us": {str(N): us(w.k, N) for N in (8, 16, 32, 64, 128, 256)},
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="qwen4b_b16")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cold-steps", type=int, default=50)
    ap.add_argument("--configs", default="tiny,qwen4b_b7,qwen8b_b7,qwen14b_b16_r8",
                    help="other workloads timed in the same run (comma list; empty: none)")
    ap.add_argument("--config-steps", type=int, default=100)
    ap.add_argument("--no-verify", action="store_true",
                    help="skip timing the verification steps after the round")
    ap.add_argument("--sweep", action="store_true",
                    help="also time the two control scorings and k / N sweeps")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run three 256 MiB device-to-device passes (an elementwise "
                         "negation: 256 MiB read, 256 MiB written), the reference for HBM counters")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: no multi-GPU path is implemented (requests would "
              "shard across GPUs with no exchange between them)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_02123_amd import pctree as P
    from paper_2608_02123_amd.synth import CONFIGS, make_inputs

    w = CONFIGS[args.workload]
    if args.calibrate_copy:
        src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)  # reads 256 MiB, writes 256 MiB
        torch.cuda.synchronize()
        log("[bench] calibration passes done (3 x 256 MiB)")
    log(f"[bench] generating {w.name}")
    inp = make_inputs(w)
    torch.cuda.set_device(0)
    dev = P.device_inputs(inp)
    builder = P.TreeBuilder(w.V, w.B, w.N, w.k, w.r, w.R,
                            P.BF16 if w.dtype == "bf16" else P.F32, mask=True)
    builder.bind(**dev)
    log(f"[bench] warmup {args.warmup}")
    for _ in range(args.warmup):
        builder.launch()
    torch.cuda.synchronize()

    # timed region: K back-to-back rounds
    log(f"[bench] timing {args.steps} rounds")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        builder.launch()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = e0.elapsed_time(e1) / args.steps
    rounds_per_s = 1000.0 / ms

    # dominant kernel, timed with events around each of its launches
    log("[bench] kernel timing pass")
    P.profile_enable(True)
    for _ in range(args.steps):
        builder.launch()
    torch.cuda.synchronize()
    kms, launches, kname = P.profile_read()
    P.profile_enable(False)
    k_avg_s = kms / 1000.0 / max(launches, 1)
    bytes_round = algorithmic_bytes(w)
    # the persistent round kernel runs all B stages; a head launch runs one
    per_launch = bytes_round if kname == "round_kernel" else bytes_round / w.B
    achieved = per_launch / k_avg_s / 1e9

    # per-round spread, warm (back to back) and cold (W evicted from the
    # Infinity Cache before each round)
    log(f"[bench] per-round pass: {args.steps} warm, {args.cold_steps} cold")
    flush = torch.empty(512 << 20 if args.cold_steps else 1, dtype=torch.uint8, device="cuda")
    warm_us, cold_us = time_rounds(builder.launch, args.steps, args.cold_steps, flush)
    warm_sp, cold_sp = spread(warm_us), spread(cold_us)
    cold_med = cold_sp["median"] / 1000.0 if cold_sp else None  # ms

    verify = None if args.no_verify else time_verify(P, builder, w, inp)
    sweep = time_sweeps(P, w, inp, dev) if args.sweep else None
    configs = {}
    for name in [c for c in args.configs.split(",") if c and c != w.name]:
        configs[name] = time_config(P, name, args.config_steps, min(args.cold_steps, 30), flush)

    cpu = None
    if not args.no_cpu_baseline:
        log(f"[bench] cpu baseline (~{args.cpu_seconds:.0f} s)")
        cpu = cpu_baseline(inp, w, args.cpu_seconds)

    traffic = measured_traffic()
    w_once = algorithmic_bytes(w, w_once=True)
    line = {
        "metric": METRIC,
        "value": rounds_per_s,
        "unit": "rounds/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded; Qwen3-shaped base logits and random-init Markov head)",
        "config": {"workload": f"{w.name}: V={w.V} B={w.B} N={w.N} k={w.k} r={w.r} R={w.R} "
                               f"{w.dtype}", "global_batch": w.R, "seq_len": w.B,
                   "parallelism": "single GPU"},
        "us_per_round": ms * 1000.0,
        "round_hbm_frac": bytes_round / (ms / 1000.0) / 1e9 / HBM_PEAK_GBS,
        "round_us": {"warm": warm_sp, "cold": cold_sp},
        "cold_us_per_round": cold_med * 1000.0 if cold_med else None,
        "cold_rounds_per_s": 1000.0 / cold_med if cold_med else None,
        "cold_round_hbm_frac": (bytes_round / (cold_med / 1000.0) / 1e9 / HBM_PEAK_GBS
                                if cold_med else None),
        "algorithmic_bytes_per_round": bytes_round,
        "w_once_bytes_per_round": w_once,
        "roofline": {"bound": "hbm", "kernel": kname, "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": traffic, "bytes_per_launch": per_launch,
                     "avg_launch_us": k_avg_s * 1e6, "launches": launches,
                     # the same bytes over the median cold round (W evicted first)
                     "cold_frac": (bytes_round / (cold_med / 1000.0) / 1e9 / HBM_PEAK_GBS
                                   if cold_med else None),
                     # what the kernel really moves: counter bytes per launch
                     "traffic_frac": (traffic / k_avg_s / 1e9 / HBM_PEAK_GBS
                                      if traffic else None),
                     # the floor with W read once per round, over the same time
                     "w_once_bytes": w_once if kname == "round_kernel" else w_once / w.B,
                     "w_once_frac": ((w_once if kname == "round_kernel" else w_once / w.B)
                                     / k_avg_s / 1e9 / HBM_PEAK_GBS),
                     # the B dependent stages of one launch: time per stage
                     "stage_period_us": (k_avg_s * 1e6 / w.B if kname == "round_kernel"
                                         else k_avg_s * 1e6)},
        "cpu_baseline": cpu,
        "wall_s_timed_region": wall,
    }
    if verify is not None:
        line["verify"] = verify
    if sweep is not None:
        line["sweep"] = sweep
    if configs:
        line["configs"] = configs
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
