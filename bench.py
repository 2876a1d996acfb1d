#!/usr/bin/env python3
"""Benchmark of the batched routing scorer on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input,
every input already resident in HBM:
  1. ls_load_cache_state  -- rebuild every instance's prefix-cache hash table
  2. ls_score_batch       -- prefix overlap, features, reward model, argmin
  3. ls_update            -- one online SGD step of the reward model
The printed value is (request, instance) pairs scored per second of step time;
updates per second and per-kernel timings ride along.  Per-kernel durations
come from HIP events recorded by the library on the stream of each call.

    python bench.py [--steps K] [--warmup W] [--config large_batch] [--no-cpu-baseline]
                    [--copy-probe-mib M]

--copy-probe-mib runs M MiB device-to-device copies after the timed region; a
hardware-counter pass over the same command reads FETCH_SIZE / WRITE_SIZE of
that plain copy beside the scorer's kernels, which calibrates the counters.
"roofline.traffic" is filled from a committed counter record
(profiles/traffic_<kind>_<workload>.md) only while the sources of that kernel
still hash to the digest the record was taken at; otherwise it is null.
"""
import argparse
import glob
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "(request,instance) pairs scored/sec + online updates/sec; % HBM/MFMA roofline"

# MI355X published peaks (dense)
PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2500.0
# fp32 FMA on the vector ALUs without packed-fp32 instructions (disabled in this
# build): 256 CUs x 4 SIMDs x 16 lanes x 2 flop x 2.4 GHz
PEAK_VALU_FP32_TFLOPS = 256 * 4 * 16 * 2 * 2.4e9 / 1e12


# Kernels behind each timed kind (names as rocprofv3 prints them) and the
# sources they are compiled from.
KIND_KERNELS = {
    "score_pairs_mfma": (["ls::score_pairs_mfma_kernel"], ["k_score_mfma.hip", "k_common.h", "ls_internal.h"]),
    "table_build": (["ls::table_segment_kernel", "ls::table_overflow_kernel"], ["k_cache.hip", "ls_internal.h"]),
    "prefix_match": (["ls::group_insert_kernel", "ls::group_lcp_kernel", "ls::cont_filter_kernel",
                      "ls::cont_scan_kernel", "ls::cont_probe_kernel", "ls::prefix_leaders_kernel",
                      "ls::followers_resolve_kernel", "ls::followers_probe_kernel"], ["k_prefix.hip", "ls_internal.h"]),
    "rescore": (["ls::rescore_wave_kernel"], ["k_band.hip", "k_common.h", "ls_internal.h"]),
    "update": (["ls::dense_lane_kernel", "ls::wgrad_mfma_kernel", "ls::wgrad_direct_kernel", "ls::wgrad_reduce_kernel",
                "ls::delta_head_kernel", "ls::normalize_kernel", "ls::loss_grad_kernel", "ls::loss_final_kernel",
                "ls::sgd_kernel", "ls::refresh_compute_kernel"], ["k_update.hip", "k_score.hip", "ls_internal.h"]),
}


def sources_digest(kind):
    h = hashlib.sha256()
    for f in KIND_KERNELS[kind][1]:
        with open(os.path.join(ROOT, "paper_2606_00946_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_record(kind, workload):
    """HBM bytes per launch from a committed counter record, if it is current."""
    if kind not in KIND_KERNELS:
        return None
    digest = sources_digest(kind)
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "traffic_*.md"))):
        with open(path) as fh:
            for line in fh:
                if not line.startswith("record: "):
                    continue
                rec = json.loads(line[len("record: "):])
                if rec.get("kind") == kind and rec.get("workload") == workload and rec.get("digest") == digest:
                    return rec
    return None


def copy_probe(mib):
    import torch
    src = torch.ones(mib << 20, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"copy probe: 3 x {mib} MiB device-to-device")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def model_flops_per_pair(cfg):
    d, (h1, h2) = cfg.d, cfg.hidden
    return 2 * (d * h1 + h1 * h2 + h2)


def executed_flops_per_pair(cfg):
    """Flops of one pair as the scorers run it: layer 1 resumes the instance's
    partial (b1 and the instance columns, computed once per instance), so only
    the 5 request and pair columns are multiplied per pair."""
    d, (h1, h2) = cfg.d, cfg.hidden
    return 2 * (5 * h1 + h1 * h2 + h2)


def update_flops(cfg, B):
    d, (h1, h2) = cfg.d, cfg.hidden
    fwd = 2 * (d * h1 + h1 * h2 + h2)
    wgrad = 2 * (d * h1 + h1 * h2 + h2)
    igrad = 2 * (h1 * h2)                 # gradient into the first hidden layer
    return B * (fwd + wgrad + igrad)


def cpu_baseline(w, target_s=12.0):
    """The oracle, untuned, on a bounded sample of requests (all instances each)."""
    import oracle
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or (os.cpu_count() or 1)
    cfg = w.cfg
    mode = "bf16" if cfg.dtype == "bf16" else "fp32"
    rng = np.random.default_rng(7)

    def run(S):
        sel = np.sort(rng.choice(cfg.R, min(S, cfg.R), replace=False)).astype(np.int32)
        t = time.perf_counter()
        oracle.score(mode, cfg.d, cfg.hidden, w.params, w.mu, w.inv_sigma, w.req_off, w.req_hashes, w.prompt_len,
                     w.inst_feat, w.inst_off, w.inst_hashes, sel=sel, threads=threads)
        return len(sel), time.perf_counter() - t

    # two points separate the per-call cost (building the instance sets) from the per-request cost
    s0, t0 = run(16)
    s1, t1 = run(64)
    per_req = max((t1 - t0) / max(s1 - s0, 1), 1e-6)
    fixed = max(t0 - s0 * per_req, 0.0)
    S = int(min(cfg.R, max(64, (target_s - fixed) / per_req)))
    s1, t1 = run(S)
    return {
        "value": s1 * cfg.N / t1, "unit": "pairs/s", "cores": threads, "kind": "oracle",
        "sample": (f"{s1} of {cfg.R} requests x all {cfg.N} instances, {mode} oracle "
                   f"(set build + overlap + features + MLP + argmin), {t1:.1f} s wall"),
    }


ROUTE_POLICY = dict(heuristic=1, count_cols=(0, 1), theta_imbal=4.0, overload_k=0.5, n_samples=10000, n_min=1000,
                    epsilon=0.05, kv_col=4, tau_sat=0.3, tau_ben=64.0, k_filter=2, delta=0.01)


def time_route(ctx, w, dev_in, reps):
    """The full routing policy (fallback heuristic, exploration, K-filter, tie-break) on the same batch, timed
    on its own: it is a separate entry point and not part of the step above."""
    import torch

    from paper_2606_00946_amd import lodestar
    R, N = w.cfg.R, w.cfg.N
    pol = lodestar.make_policy(**ROUTE_POLICY)
    rnd = torch.from_numpy(np.random.default_rng(3).integers(0, 1 << 32, (R, 3), dtype=np.uint64)
                           .astype(np.uint32).view(np.int32)).cuda()
    chosen = torch.empty(R, dtype=torch.int32, device="cuda")
    status = torch.empty(R, dtype=torch.int32, device="cuda")
    ctx.ls_route_batch(pol, *dev_in, rnd, chosen, status)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        ctx.ls_route_batch(pol, *dev_in, rnd, chosen, status)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / reps
    st = status.cpu().numpy()
    return {"policy": "Alg. 4 with Alg. 1 fallback, epsilon 0.05, K-filter 2, delta 0.01",
            "ms_per_batch": round(ms, 4), "pairs_per_s": round(R * N / (ms / 1e3), 1),
            "explored": int(((st & 0x100) != 0).sum()), "kfilter": int(((st & 0x200) != 0).sum()),
            "tiebreak": int(((st & 0x400) != 0).sum())}


def time_online_learning(ctx, w):
    """The paper's data path at its own sizes (Section 4.3.2): FIFO and replay pool of 5000 each, a push of 1000
    logged samples into full pools (1000 coreset decisions), then a retraining round over the 10,000 samples."""
    import torch
    cfg = w.cfg
    rng = np.random.default_rng(11)
    x_all = torch.from_numpy(np.ascontiguousarray(w.upd_feats[:11000])).cuda()
    y_all = torch.from_numpy(np.ascontiguousarray(w.upd_ttft[:11000])).cuda()
    ctx.ls_buffer_init(5000, 5000)
    ctx.ls_buffer_push(x_all[:10000], y_all[:10000])        # fills FIFO and pool
    torch.cuda.synchronize()
    adm = torch.zeros(1, dtype=torch.int32, device="cuda")
    t0 = time.perf_counter()
    ctx.ls_buffer_push(x_all[10000:11000], y_all[10000:11000], adm)
    torch.cuda.synchronize()
    push_ms = (time.perf_counter() - t0) * 1e3
    perm = np.concatenate([rng.permutation(10000) for _ in range(5)]).astype(np.int32)
    t0 = time.perf_counter()
    ctx.ls_train_round(5, 256, w.lr, perm)
    torch.cuda.synchronize()
    train_ms = (time.perf_counter() - t0) * 1e3
    return {"fifo": 5000, "replay": 5000, "push_1000_ms": round(push_ms, 3), "admitted": int(adm.item()),
            "train_round_ms": round(train_ms, 3), "train_round": "5 epochs x 10000 samples, minibatch 256",
            "train_samples_per_s": round(5 * 10000 / (train_ms / 1e3), 1)}


def time_maintenance(w, inst_h, req_off, req_h, chosen, reps):
    """Prefix-index maintenance (Section 2: the gateway records each routed request's blocks on its instance,
    engines evict least recently used blocks): the step's routed batch committed into the loaded state with exact
    LRU eviction to the loaded capacity, then the tables rebuilt.  Each commit runs on a fresh load, untimed."""
    import torch

    from paper_2606_00946_amd import lodestar
    cfg = w.cfg
    ctx = lodestar.Context(cfg.d, cfg.hidden, cfg.dtype, device=0)
    ctx.ls_set_model(w.params, w.mu, w.inv_sigma)
    ctx.ls_set_cache_capacity(np.diff(w.inst_off))
    n_hashes = int(w.req_off[-1])
    wall, kinds = 0.0, {}
    for i in range(reps + 1):
        ctx.ls_load_cache_state(w.inst_off, inst_h)
        torch.cuda.synchronize()
        if i > 0:
            ctx.ls_profile_enable(True)
        t0 = time.perf_counter()
        ctx.ls_commit_routes(req_off, req_h, chosen, n_hashes=n_hashes)
        torch.cuda.synchronize()
        if i > 0:
            wall += time.perf_counter() - t0
            for k, v in ctx.ls_profile_read().items():
                kinds[k] = kinds.get(k, 0.0) + v[1]
            ctx.ls_profile_enable(False)
    off, _, _ = ctx.ls_read_cache_state()
    ctx.close()
    ms = wall * 1e3 / reps
    return {"commit_ms": round(ms, 4), "kernel_ms": {k: round(v / reps, 4) for k, v in kinds.items()},
            "routed_blocks": n_hashes, "cached_blocks_after": int(off[-1]),
            "requests_per_s": round(w.cfg.R / (ms / 1e3), 1)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="large_batch")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe-mib", type=int, default=0)
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the scorer shards by request with no collective, and this build "
              "runs on a single MI355X; use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2606_00946_amd import lodestar, synth

    torch.cuda.set_device(0)
    t = time.perf_counter()
    w = synth.generate(args.config)
    cfg = w.cfg
    log(f"generated {cfg.name}: R={cfg.R} N={cfg.N} hashes={w.req_hashes.size} cached={w.inst_hashes.size} "
        f"({time.perf_counter() - t:.1f} s)")

    def dev(a):
        a = np.ascontiguousarray(a)
        return torch.from_numpy(a.view(np.int64) if a.dtype == np.uint64 else a).cuda()

    ctx = lodestar.Context(cfg.d, cfg.hidden, cfg.dtype, device=0)
    ctx.ls_set_model(w.params, w.mu, w.inv_sigma)
    inst_h = dev(w.inst_hashes)
    req_off, req_h, plen, feat = dev(w.req_off), dev(w.req_hashes), dev(w.prompt_len), dev(w.inst_feat)
    upd_x, upd_y = dev(w.upd_feats), dev(w.upd_ttft)
    R, N, B = cfg.R, cfg.N, cfg.update_batch
    chosen = torch.empty(R, dtype=torch.int32, device="cuda")
    min_ttft = torch.empty(R, dtype=torch.float32, device="cuda")
    overlap = torch.empty(R * N, dtype=torch.int32, device="cuda")
    loss = torch.empty(1, dtype=torch.float32, device="cuda")

    def step():
        ctx.ls_load_cache_state(w.inst_off, inst_h)
        ctx.ls_score_batch(req_off, req_h, plen, feat, chosen, min_ttft, None, overlap, None)
        ctx.ls_update(upd_x, upd_y, w.lr, loss, None)

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log(f"warmup step {i + 1}/{args.warmup} done")
    ctx.ls_profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    prof = ctx.ls_profile_read()
    ctx.ls_profile_enable(False)
    log(f"timed {args.steps} steps: {(t1 - t0) * 1e3 / args.steps:.3f} ms/step")

    ms_step = (t1 - t0) * 1e3 / args.steps
    pairs_per_s = R * N / (ms_step / 1e3)
    phases = {k: round(v[1] / args.steps, 4) for k, v in prof.items()}

    # algorithmic work of each kernel kind per launch
    n = np.diff(w.req_off)
    ov = overlap.cpu().numpy().reshape(R, N).astype(np.int64)
    probes = int(np.minimum(ov + 1, n[:, None]).sum())
    k1_bytes = 64 * probes + 8 * int(n.sum()) + 4 * R * N
    model_tflop = model_flops_per_pair(cfg) * R * N / 1e12
    exec_tflop = executed_flops_per_pair(cfg) * R * N / 1e12
    roof = {
        "prefix_match": ("hbm", k1_bytes / 1e9, PEAK_HBM_GBS, "GB/s"),
        "score_pairs": ("alu", exec_tflop, PEAK_VALU_FP32_TFLOPS, "TFLOP/s"),
        "score_pairs_mfma": ("mfma", exec_tflop, PEAK_BF16_TFLOPS, "TFLOP/s"),
        "update": ("alu", update_flops(cfg, B) / 1e12, PEAK_VALU_FP32_TFLOPS, "TFLOP/s"),
        "table_build": ("hbm", (8 + 64) * int(w.inst_hashes.size) / 1e9, PEAK_HBM_GBS, "GB/s"),
    }
    dom = max((k for k in prof if k in roof), key=lambda k: prof[k][1])
    bound, work, peak, unit = roof[dom]
    avg_s = prof[dom][1] / prof[dom][0] / 1e3
    achieved = work / avg_s
    # the unfactorised model's flops over the same time, for comparison
    model_rate = round(model_tflop / avg_s, 3) if dom in ("score_pairs", "score_pairs_mfma") else None
    rec = traffic_record(dom, cfg.name)
    traffic = None if rec is None else round(rec["bytes_per_launch"] / 1e9, 4)
    result = {
        "metric": METRIC,
        "value": round(pairs_per_s, 1),
        "unit": "pairs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": cfg.name, "requests": R, "instances": N, "update_batch": B,
                   "cached_blocks": int(w.inst_hashes.size), "prompt_blocks": int(n.sum()),
                   "predictor": f"{cfg.d}-{cfg.hidden[0]}-{cfg.hidden[1]}-1 {cfg.dtype}"},
        "updates_per_s": round(1e3 / ms_step, 3),
        "update_samples_per_s": round(B * 1e3 / ms_step, 1),
        "kernel_ms_per_step": phases,
        "roofline": {"kernel": dom, "bound": bound, "achieved": round(achieved, 3), "peak": round(peak, 1),
                     "unit": unit, "frac": round(achieved / peak, 4), "traffic": traffic,
                     "traffic_unit": "GB per launch", "digest": sources_digest(dom) if dom in KIND_KERNELS else None,
                     "model_flop_rate": model_rate},
        "useful_probes": probes,
    }
    result["route"] = time_route(ctx, w, (req_off, req_h, plen, feat), args.steps)
    result["online_learning"] = time_online_learning(ctx, w)
    result["maintenance"] = time_maintenance(w, inst_h, req_off, req_h, chosen, max(1, min(args.steps, 5)))
    ctx.close()
    if args.copy_probe_mib > 0:
        copy_probe(args.copy_probe_mib)
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
