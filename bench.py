#!/usr/bin/env python3
"""Benchmark of the batched routing scorer on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input,
every input already resident in HBM:
  1. ls_load_cache_state  -- rebuild every instance's prefix-cache hash table
  2. ls_score_batch       -- prefix overlap, features, reward model, argmin
  3. ls_update            -- one online SGD step of the reward model
The printed value is (request, instance) pairs scored per second of step time.
Beside it: pairs per second of the scoring call alone (R N / t_score), the
update's own steps and samples per second, per-kernel timings and rooflines, and
one entry per other workload (scoring and update only, as the cache state of a
serving router changes far less often than its batches).  Per-kernel durations
come from HIP events recorded by the library on the stream of each call.

    python bench.py [--steps K] [--warmup W] [--config large_batch] [--no-cpu-baseline]
                    [--no-other-configs] [--copy-probe-mib M]

--copy-probe-mib runs M MiB device-to-device copies after the timed region; a
hardware-counter pass over the same command reads FETCH_SIZE / WRITE_SIZE of
that plain copy beside the kernels, which calibrates the counters.
"traffic" is filled from a committed counter record
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
# fp32 on the matrix cores (dense), where the canonical chains run as K=1 steps
PEAK_FP32_MFMA_TFLOPS = 157.3


# Kernels behind each timed kind (names as rocprofv3 prints them) and the
# sources they are compiled from.
KIND_KERNELS = {
    "score_pairs_mfma": (["ls::score_pairs_mfma_kernel"], ["k_score_mfma.hip", "k_common.h", "ls_internal.h"]),
    "table_build": (["ls::seg_inst_kernel", "ls::part_kernel", "ls::table_segment_kernel", "ls::table_overflow_kernel"],
                    ["k_cache.hip", "ls_internal.h"]),
    "prefix_match": (["ls::group_insert_kernel", "ls::group_lcp_kernel", "ls::cont_scan_kernel",
                      "ls::leaders_first_kernel", "ls::leaders_rest_kernel",
                      "ls::followers_resolve_kernel", "ls::followers_probe_kernel"], ["k_prefix.hip", "ls_internal.h"]),
    "rescore": (["ls::rescore_chain_mfma_kernel", "ls::rescore_wave_kernel"],
                ["k_score_chain.hip", "k_band.hip", "k_common.h", "k_policy.h", "ls_internal.h"]),
    "score_pairs": (["ls::score_chain_mfma_kernel", "ls::score_pairs_kernel"],
                    ["k_score_chain.hip", "k_score.hip", "k_common.h", "ls_internal.h"]),
    "update": (["ls::normalize_kernel", "ls::normalize_b16_kernel", "ls::dense_mfma_kernel", "ls::dense_lane_kernel", "ls::dense_small_kernel",
                "ls::layer_fwd_kernel",
                "ls::loss_grad_kernel", "ls::loss_final_kernel", "ls::wgrad_direct_kernel", "ls::wgrad_row_kernel",
                "ls::wgrad_reduce_wave_kernel", "ls::wgrad_reduce_kernel", "ls::wgrad_mfma_kernel",
                "ls::delta_head_kernel", "ls::delta_head_b16_kernel", "ls::backprop_hidden_kernel", "ls::gemm_nt_splitk_kernel",
                "ls::splitk_reduce_kernel", "ls::rowsum_kernel", "ls::sgd_kernel", "ls::refresh_compute_kernel",
                "ls::prepare_mfma_kernel"],
               ["k_update.hip", "k_score.hip", "k_score_mfma.hip", "k_common.h", "k_policy.h", "ls_internal.h"]),
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


def chain_flops(cfg, B):
    """Flops of the update's canonical fma chains: the forward layers and head,
    and the gradient into the first hidden layer."""
    d, (h1, h2) = cfg.d, cfg.hidden
    return B * (2 * (d * h1 + h1 * h2 + h2) + 2 * h1 * h2)


def cpu_baseline(w, target_s=12.0, single_requests=256):
    """The oracle, untuned, on a bounded sample of requests (all instances each):
    on every host core, then on one thread over the first `single_requests`
    requests."""
    import oracle
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or (os.cpu_count() or 1)
    cfg = w.cfg
    mode = "bf16" if cfg.dtype == "bf16" else "fp32"
    rng = np.random.default_rng(7)

    def run(sel, nthreads):
        t = time.perf_counter()
        oracle.score(mode, cfg.d, cfg.hidden, w.params, w.mu, w.inv_sigma, w.req_off, w.req_hashes, w.prompt_len,
                     w.inst_feat, w.inst_off, w.inst_hashes, sel=sel, threads=nthreads)
        return len(sel), time.perf_counter() - t

    pick = lambda S: np.sort(rng.choice(cfg.R, min(S, cfg.R), replace=False)).astype(np.int32)
    # two points separate the per-call cost (building the instance sets) from the per-request cost
    s0, t0 = run(pick(16), threads)
    s1, t1 = run(pick(64), threads)
    per_req = max((t1 - t0) / max(s1 - s0, 1), 1e-6)
    fixed = max(t0 - s0 * per_req, 0.0)
    S = int(min(cfg.R, max(64, (target_s - fixed) / per_req)))
    s1, t1 = run(pick(S), threads)
    sg = min(single_requests, cfg.R)
    s2, t2 = run(np.arange(sg, dtype=np.int32), 1)
    return {
        "value": s1 * cfg.N / t1, "unit": "pairs/s", "cores": threads, "kind": "oracle",
        "sample": (f"{s1} of {cfg.R} requests x all {cfg.N} instances, {mode} oracle "
                   f"(set build + overlap + features + MLP + argmin), {t1:.1f} s wall"),
        "single_thread": {"value": s2 * cfg.N / t2, "unit": "pairs/s", "cores": 1,
                          "sample": f"first {s2} requests x all {cfg.N} instances, {mode} oracle, {t2:.1f} s wall "
                                    "(per-call set build included)"},
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
    # 11,000 logged rows (the workload's update rows, repeated if it has fewer)
    x_all = torch.from_numpy(np.ascontiguousarray(np.resize(w.upd_feats, (11000, cfg.d)))).cuda()
    y_all = torch.from_numpy(np.ascontiguousarray(np.resize(w.upd_ttft, 11000))).cuda()
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


def k1_algorithmic_bytes(w, ov):
    """Bytes the prefix-overlap step must move for this batch with shared
    prefixes answered once (Section 2: reuse is strictly sequential, so a request
    that shares its first c blocks with a longer request of the batch has that
    request's overlap wherever it is below c):
      every request hash read once (8 B), the overlap matrix written once (4 B
      per pair), and one 64-B bucket per useful probe -- for each group of
      requests with the same first block, the longest one (lowest id on ties)
      probes min(l + 1, n) blocks per instance; every other request, with
      common prefix c with it, probes min(l - c + 1, n - c) blocks on the
      instances where the longer one's run reaches c, none elsewhere.
    Speculative probes past a miss and table lines read twice are overhead."""
    req_off, h = w.req_off, w.req_hashes
    R, N = ov.shape
    n = np.diff(req_off)
    has = n > 0
    first = np.where(has, h[np.minimum(req_off[:-1], max(h.size - 1, 0))], 0)
    order = np.lexsort((np.arange(R), -n, first))            # by first hash, longest first, lowest id
    probes = 0
    i = 0
    while i < R:
        j = i
        r0 = order[i]
        while j < R and first[order[j]] == first[r0] and has[order[j]] == has[r0]:
            j += 1
        if has[r0]:
            lead = r0
            hl = h[req_off[lead]:req_off[lead + 1]]
            ll = ov[lead]
            probes += int(np.minimum(ll + 1, n[lead]).sum())
            for k in range(i + 1, j):
                f = order[k]
                hf = h[req_off[f]:req_off[f + 1]]
                m = min(hf.size, hl.size)
                diff = np.flatnonzero(hf[:m] != hl[:m])
                c = int(diff[0]) if diff.size else m
                if c >= n[f]:
                    continue
                reach = ll >= c
                probes += int(np.minimum(ov[f][reach] - c + 1, n[f] - c).sum())
        i = j
    return 64 * probes + 8 * int(n.sum()) + 4 * R * N, probes


def roofline_entry(kind, bound, work, peak, unit, calls, total_ms, cfg_name, extra=None):
    """achieved = algorithmic work per call / the kind's average device time per
    call (all of its launch groups within one call of the entry point)."""
    avg_s = total_ms / max(calls, 1) / 1e3
    achieved = work / avg_s if avg_s > 0 else 0.0
    rec = traffic_record(kind, cfg_name)
    out = {"bound": bound, "achieved": round(achieved, 3), "peak": round(peak, 1), "unit": unit,
           "frac": round(achieved / peak, 4), "avg_ms": round(avg_s * 1e3, 4),
           "traffic": None if rec is None else round(rec["bytes_per_launch"] / 1e9, 4),
           "traffic_unit": "GB per launch",
           "digest": sources_digest(kind) if kind in KIND_KERNELS else None}
    if extra:
        out.update(extra)
    return out


def scoring_rooflines(cfg, prof, steps, exec_tflop, model_tflop, k1_gb):
    """Rooflines of the scoring kernels from one profile of `steps` scoring calls:
    K1 on HBM, the bf16 scorer on the matrix cores at the bf16 peak, and the
    canonical fp32 chains (K=1 fp32 matrix-core steps) at the fp32 matrix-core
    peak."""
    out = {}
    if "prefix_match" in prof:
        out["prefix_match"] = roofline_entry("prefix_match", "hbm", k1_gb, PEAK_HBM_GBS, "GB/s", steps,
                                             prof["prefix_match"][1], cfg.name)
    for kind, bound, peak in (("score_pairs_mfma", "mfma", PEAK_BF16_TFLOPS),
                              ("score_pairs", "mfma", PEAK_FP32_MFMA_TFLOPS)):
        if kind in prof:
            ms = prof[kind][1]
            out[kind] = roofline_entry(kind, bound, exec_tflop, peak, "TFLOP/s", steps, ms, cfg.name,
                                       {"model_flop_rate": round(model_tflop / (ms / steps / 1e3), 3)})
    return out


SCORE_KINDS = ("prefix_match", "instance_partial", "score_pairs", "score_pairs_mfma", "band_select", "rescore",
               "argmin")


def time_prefix_closed(w, inst_h, ins, overlap_ref, steps):
    """The scoring call with the caches declared prefix-closed (ls_set_prefix_closed: K1 finds each run's end
    by search, exact when every cached block's predecessor in the prompt is cached as well -- Section 2: prefix
    reuse is strictly sequential and engines evict least recently used blocks, tail first; the synthetic caches
    are built so): K1's and the call's device time, and whether every overlap equals the general path's."""
    import torch

    from paper_2606_00946_amd import lodestar
    cfg = w.cfg
    R, N = cfg.R, cfg.N
    ctx = lodestar.Context(cfg.d, cfg.hidden, cfg.dtype, device=0)
    ctx.ls_set_model(w.params, w.mu, w.inv_sigma)
    ctx.ls_set_prefix_closed(True)
    ctx.ls_load_cache_state(w.inst_off, inst_h)
    chosen = torch.empty(R, dtype=torch.int32, device="cuda")
    overlap = torch.empty(R * N, dtype=torch.int32, device="cuda")
    ctx.ls_score_batch(*ins, chosen, None, None, overlap, None)
    torch.cuda.synchronize()
    ctx.ls_profile_enable(True)
    for _ in range(steps):
        ctx.ls_score_batch(*ins, chosen, None, None, overlap, None)
    torch.cuda.synchronize()
    prof = ctx.ls_profile_read()
    ctx.ls_profile_enable(False)
    ctx.close()
    ms = {k: v[1] / steps for k, v in prof.items()}
    t_score = sum(ms.get(k, 0.0) for k in SCORE_KINDS)
    return {"prefix_match_ms": round(ms.get("prefix_match", 0.0), 4), "score_ms": round(t_score, 4),
            "score_pairs_per_s": round(R * N / (t_score / 1e3), 1),
            "overlaps_equal_general": bool(torch.equal(overlap, overlap_ref))}


def run_other_config(name, steps, warmup):
    """Scoring and update of another workload: pairs/s of the scoring call, the
    update's steps/s, per-kernel times and the rooflines of K1 and the scorer."""
    import torch

    from paper_2606_00946_amd import lodestar, synth
    w = synth.generate(name)
    cfg = w.cfg
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a.view(np.int64) if a.dtype == np.uint64 else a)).cuda()
    ctx = lodestar.Context(cfg.d, cfg.hidden, cfg.dtype, device=0)
    ctx.ls_set_model(w.params, w.mu, w.inv_sigma)
    inst_h = dev(w.inst_hashes)
    ctx.ls_load_cache_state(w.inst_off, inst_h)
    ins = (dev(w.req_off), dev(w.req_hashes), dev(w.prompt_len), dev(w.inst_feat))
    x, y = dev(w.upd_feats), dev(w.upd_ttft)
    R, N, B = cfg.R, cfg.N, cfg.update_batch
    chosen = torch.empty(R, dtype=torch.int32, device="cuda")
    min_ttft = torch.empty(R, dtype=torch.float32, device="cuda")
    overlap = torch.empty(R * N, dtype=torch.int32, device="cuda")

    def step():
        ctx.ls_score_batch(*ins, chosen, min_ttft, None, overlap, None)
        ctx.ls_update(x, y, w.lr)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    ctx.ls_profile_enable(True)
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / steps
    prof = ctx.ls_profile_read()
    ctx.ls_profile_enable(False)
    ctx.close()
    closed = time_prefix_closed(w, inst_h, ins, overlap, steps)
    ms = {k: v[1] / steps for k, v in prof.items()}
    t_score = sum(ms.get(k, 0.0) for k in SCORE_KINDS)
    t_upd = ms.get("update", 0.0)
    ov = overlap.cpu().numpy().reshape(R, N).astype(np.int64)
    k1_bytes, probes = k1_algorithmic_bytes(w, ov)
    rl = scoring_rooflines(cfg, prof, steps, executed_flops_per_pair(cfg) * R * N / 1e12,
                           model_flops_per_pair(cfg) * R * N / 1e12, k1_bytes / 1e9)
    if "update" in prof:
        rl["update"] = roofline_entry("update", "mfma" if cfg.dtype == "bf16" else "alu", update_flops(cfg, B) / 1e12,
                                      PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_VALU_FP32_TFLOPS,
                                      "TFLOP/s", steps, prof["update"][1], cfg.name)
    return {"requests": R, "instances": N, "predictor": f"{cfg.d}-" + "-".join(map(str, cfg.hidden)) + f"-1 {cfg.dtype}",
            "update_batch": B, "score_pairs_per_s": round(R * N / (t_score / 1e3), 1),
            "score_ms": round(t_score, 4), "updates_per_s": round(1e3 / t_upd, 2) if t_upd else None,
            "update_samples_per_s": round(B * 1e3 / t_upd, 1) if t_upd else None,
            "wall_ms_per_step": round(wall_ms, 4), "kernel_ms": {k: round(v, 4) for k, v in ms.items()},
            "useful_probes": probes, "rooflines": rl, "prefix_closed": closed}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="large_batch")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-configs", action="store_true")
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
    t_score = sum(v[1] for k, v in prof.items() if k in SCORE_KINDS) / args.steps
    t_upd = prof["update"][1] / args.steps if "update" in prof else None

    # algorithmic work of each kernel kind per launch
    n = np.diff(w.req_off)
    ov = overlap.cpu().numpy().reshape(R, N).astype(np.int64)
    k1_bytes, probes = k1_algorithmic_bytes(w, ov)
    exec_tflop = executed_flops_per_pair(cfg) * R * N / 1e12
    model_tflop = model_flops_per_pair(cfg) * R * N / 1e12
    steps = args.steps
    rooflines = scoring_rooflines(cfg, prof, steps, exec_tflop, model_tflop, k1_bytes / 1e9)
    if "update" in prof:
        t_u = prof["update"][1] / steps / 1e3
        # the canonical chains (forward layers and hidden backprop) run as K=1 fp32
        # matrix-core steps, the weight gradients as bf16 matrix-core products: the
        # floor prices each part at its own peak
        chain_tflop = chain_flops(cfg, B) / 1e12
        grad_tflop = update_flops(cfg, B) / 1e12 - chain_tflop
        floor_ms = (chain_tflop / PEAK_FP32_MFMA_TFLOPS + grad_tflop / PEAK_BF16_TFLOPS) * 1e3
        rooflines["update"] = roofline_entry("update", "mfma" if cfg.dtype == "bf16" else "alu",
                                             update_flops(cfg, B) / 1e12,
                                             PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_VALU_FP32_TFLOPS,
                                             "TFLOP/s", steps, prof["update"][1], cfg.name,
                                             {"chain_tflop_per_s": round(chain_tflop / t_u, 3),
                                              "chain_frac_fp32_mfma": round(chain_tflop / t_u / PEAK_FP32_MFMA_TFLOPS, 4),
                                              "floor_ms_at_peaks": round(floor_ms, 4),
                                              "floor_frac": round(floor_ms / (t_u * 1e3), 4)})
    if "table_build" in prof:
        # each cached key read once (8 B) and its table written once (two 8-byte slots per key at half load)
        rooflines["table_build"] = roofline_entry("table_build", "hbm", (8 + 16) * int(w.inst_hashes.size) / 1e9,
                                                  PEAK_HBM_GBS, "GB/s", steps, prof["table_build"][1], cfg.name)
    dom = max((k for k in rooflines), key=lambda k: prof[k][1])
    roof = dict(rooflines[dom])
    roof = {"kernel": dom, **roof}

    # candidates the band sends to canonical rescoring, per request (after the timed region)
    band = None
    tt = torch.empty(R * N, dtype=torch.float32, device="cuda")
    ee = torch.empty(R * N, dtype=torch.float32, device="cuda")
    bb = torch.empty(R * N, dtype=torch.uint8, device="cuda")
    try:
        ctx.ls_fast_scores(req_off, req_h, plen, feat, tt, ee, bb)
        torch.cuda.synchronize()
        band = round(float(bb.sum(dtype=torch.int64).item()) / R, 4)
    except lodestar.LodestarError:
        pass                                      # no matrix-core path for this model
    del tt, ee, bb

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
        "score_pairs_per_s": round(R * N / (t_score / 1e3), 1),
        "score_ms": round(t_score, 4),
        "updates_per_s": round(1e3 / t_upd, 3) if t_upd else None,
        "update_samples_per_s": round(B * 1e3 / t_upd, 1) if t_upd else None,
        "kernel_ms_per_step": phases,
        "roofline": roof,
        "rooflines": rooflines,
        "useful_probes": probes,
        "band_candidates_per_request": band,
    }
    result["route"] = time_route(ctx, w, (req_off, req_h, plen, feat), args.steps)
    result["online_learning"] = time_online_learning(ctx, w)
    result["maintenance"] = time_maintenance(w, inst_h, req_off, req_h, chosen, max(1, min(args.steps, 5)))
    ctx.close()
    result["prefix_closed"] = time_prefix_closed(w, inst_h, (req_off, req_h, plen, feat), overlap, args.steps)
    del inst_h, req_off, req_h, plen, feat, upd_x, upd_y, overlap
    torch.cuda.empty_cache()
    if not args.no_other_configs:
        others = {}
        for name in ("tiny", "homogeneous", "heterogeneous", "long_context"):
            if name == cfg.name:
                continue
            others[name] = run_other_config(name, args.steps, max(1, args.warmup))
            log(f"{name}: {others[name]['score_pairs_per_s']:.4g} pairs/s, {others[name]['score_ms']} ms scoring")
            torch.cuda.empty_cache()
        result["other_configs"] = others
    if args.copy_probe_mib > 0:
        copy_probe(args.copy_probe_mib)
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
