"""The bench's work models and roofline arithmetic, on the CPU.

Every fraction the bench reports divides algorithmic work by a measured time.
These tests pin the work side: the flops per pair and per update step against
counts built from the layer shapes, K1's useful-probe byte model against
hand-counted cases (the overlaps cross-checked with the oracle), and the
roofline arithmetic.  The bench must also refuse to run on more than one GPU."""
import os
import subprocess
import sys
import types

import numpy as np

import bench
import oracle
from paper_2606_00946_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _layers(cfg):
    d, (h1, h2) = cfg.d, cfg.hidden
    return d, h1, h2, [(d, h1), (h1, h2), (h2, 1)]


def test_flops_per_pair_from_layer_shapes():
    for cfg in synth.CONFIGS.values():
        d, h1, _, shapes = _layers(cfg)
        macs = sum(i * o for i, o in shapes)
        assert bench.model_flops_per_pair(cfg) == 2 * macs
        # layer 1 resumes each instance's partial (b1 and its d - 5 columns):
        # only the 5 request and pair columns are multiplied per pair
        assert bench.executed_flops_per_pair(cfg) == 2 * (macs - (d - 5) * h1)
    large = synth.CONFIGS["large_batch"]
    assert bench.model_flops_per_pair(large) == 164_352
    assert bench.executed_flops_per_pair(large) == 134_144


def test_update_flops_from_layer_shapes():
    for cfg in synth.CONFIGS.values():
        B = cfg.update_batch
        _, h1, h2, shapes = _layers(cfg)
        macs = sum(i * o for i, o in shapes)
        forward, weight_grads = 2 * macs * B, 2 * macs * B
        # the gradient into the first hidden layer goes back through W2; the
        # head's into the second is an elementwise product
        input_grad = 2 * h1 * h2 * B
        assert bench.update_flops(cfg, B) == forward + weight_grads + input_grad
        assert bench.chain_flops(cfg, B) == forward + input_grad
    large = synth.CONFIGS["large_batch"]
    assert round(bench.update_flops(large, 65536) / 1e9, 1) == 30.1
    assert round(bench.chain_flops(large, 65536) / 1e9, 1) == 19.4


def _workload(requests, caches):
    req_off = np.zeros(len(requests) + 1, np.int64)
    req_off[1:] = np.cumsum([len(r) for r in requests])
    inst_off = np.zeros(len(caches) + 1, np.int64)
    inst_off[1:] = np.cumsum([len(c) for c in caches])
    cat = lambda xs: np.array([v for x in xs for v in x], np.uint64)
    return types.SimpleNamespace(req_off=req_off, req_hashes=cat(requests), inst_off=inst_off,
                                 inst_hashes=cat(caches))


def _k1(requests, caches, want_ov):
    w = _workload(requests, caches)
    ov = oracle.overlap(w.req_off, w.req_hashes, w.inst_off, w.inst_hashes)
    np.testing.assert_array_equal(ov, np.array(want_ov, np.int32))
    return bench.k1_algorithmic_bytes(w, ov.astype(np.int64))


def test_k1_useful_probes_hand_counted():
    # r0 and r1 share their first block, r0 is the longer (the group's leader);
    # r2 is alone.  Leader r0 probes min(l + 1, n): 4 on instance 0 (a run of 3
    # ending at block 3), 2 on instance 1.  Follower r1 shares c = 2 blocks with
    # r0; only instance 0's run reaches c, where r1 probes min(2 - 2 + 1, 3 - 2)
    # = 1.  r2 misses its first block on both instances: 1 + 1.  9 probes.
    caches = [[1, 2, 3], [1, 5]]
    requests = [[1, 2, 3, 4], [1, 2, 9], [7, 8]]
    nbytes, probes = _k1(requests, caches, [[3, 1], [2, 1], [0, 0]])
    assert probes == 9
    assert nbytes == 64 * 9 + 8 * (4 + 3 + 2) + 4 * 3 * 2


def test_k1_identical_and_empty_requests():
    # identical requests: the lower id leads (2 probes: a run of 2 = n), the
    # other shares all of its blocks and probes nothing
    nbytes, probes = _k1([[5, 6], [5, 6]], [[5, 6]], [[2], [2]])
    assert probes == 2 and nbytes == 64 * 2 + 8 * 4 + 4 * 2
    # an empty request probes nothing; a one-block request that misses probes once
    nbytes, probes = _k1([[], [3]], [[4]], [[0], [0]])
    assert probes == 1 and nbytes == 64 + 8 + 4 * 2


def test_roofline_arithmetic():
    # 1 GB per call, 4 calls in 1 ms: 0.25 ms per call, 4 TB/s, half of 8 TB/s
    r = bench.roofline_entry("prefix_match", "hbm", 1.0, 8000.0, "GB/s", 4, 1.0, "no_such_workload")
    assert r["avg_ms"] == 0.25 and r["achieved"] == 4000.0 and r["frac"] == 0.5
    assert r["traffic"] is None                      # no counter record for this workload
    assert r["digest"] == bench.sources_digest("prefix_match")


def test_bench_refuses_more_than_one_gpu():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert p.returncode == 2
    assert "one GPU" in p.stderr or "single MI355X" in p.stderr
