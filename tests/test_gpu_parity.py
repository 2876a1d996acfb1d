"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Bars: overlap counts, chosen instances and feature rows bit-exact; scores
bit-identical to the oracle in the kernel's precision (fp32 fma chains, or bf16
operands with fp32 sums) and within 1e-4 relative of the double-precision
definition for fp32 models; gradients within 1e-4 relative of the oracle whose
forward pass (and so every ReLU mask) runs in the kernel's precision and whose
backward sums are double (per tensor in norm, and per element against
max(|ref|, 0.1 RMS of the tensor)), loss within 1e-5 relative.
"""
import functools

import numpy as np
import pytest

import oracle
import oracle_pins
from gpu_helpers import GpuRun, band_check, fp32_bound_ok, grad_ok, layer_slices, note, rel_ok, to_dev, uses_fast_path
from paper_2606_00946_amd import lodestar, synth

pytestmark = pytest.mark.gpu

CONFIGS = ["tiny", "homogeneous", "heterogeneous", "long_context", "large_batch"]
FULL_SCORE = {"tiny", "homogeneous", "heterogeneous", "long_context"}   # the oracle scores every pair


@functools.lru_cache(maxsize=2)
def workload(name, R=None, N=None):
    return synth.generate(name, R=R, N=N)


def mode_of(w):
    return "bf16" if w.cfg.dtype == "bf16" else "fp32"


def sampled(w, k=96, seed=0):
    R = w.cfg.R
    if w.cfg.name in FULL_SCORE and R * w.cfg.N <= 600_000:
        return np.arange(R, dtype=np.int32)
    rng = np.random.default_rng(seed)
    sel = np.unique(np.concatenate([[0, R - 1], rng.choice(R, k, replace=False)]))
    return sel.astype(np.int32)


def oracle_score(w, mode, sel):
    return oracle.score(mode, w.cfg.d, w.cfg.hidden, w.params, w.mu, w.inv_sigma, w.req_off, w.req_hashes,
                        w.prompt_len, w.inst_feat, w.inst_off, w.inst_hashes, sel=sel, threads=16)


def check_scoring(w, out, sel, exact=False, run=None):
    """`out` is a call that asked for the score matrix, so every score is the
    canonical one: overlaps, decisions, min_ttft, feature rows and scores
    bit-exact against the oracle in the kernel's precision on the selected
    requests (and fp32 scores within 1e-4 of the double-precision definition).
    With `run` on a context whose bf16 model runs on the matrix cores, the
    matrix-core call's decisions, minima, overlaps and rows must equal the
    canonical call's on every request, and every fast score must lie within
    E/8 of the canonical one (the bound the decision relies on, with a margin)."""
    mode = mode_of(w)
    ref = oracle_score(w, mode, sel)
    np.testing.assert_array_equal(out["overlap"][sel], ref["overlap"])
    np.testing.assert_array_equal(out["chosen"][sel], ref["chosen"])
    np.testing.assert_array_equal(out["min_ttft"][sel].view(np.uint32), ref["min_ttft"].astype(np.float32).view(np.uint32))
    np.testing.assert_array_equal(out["feat"][sel], ref["feat"].astype(np.float32))
    got = out["scores"][sel]
    want = ref["scores"].astype(np.float32)
    mism = np.argwhere(got.view(np.uint32) != want.view(np.uint32))
    assert mism.size == 0, f"{len(mism)} scores differ from the oracle, first {mism[:3]}"
    if mode == "fp32":
        ref64 = oracle_score(w, "f64", sel)
        ok, worst = fp32_bound_ok(w, sel, out["overlap"][sel], got, ref64["scores"])
        assert ok, f"scores vs double-precision definition: {worst} times the bar"
    if run is not None and uses_fast_path(w.cfg.d, w.cfg.hidden, w.cfg.dtype, exact):
        check_fast_path(w, run, out)
    return ref


def check_fast_path(w, run, canon, what=None):
    """The matrix-core path against a canonical call on the same context."""
    fast = run.score(with_scores=False)
    for k in ("overlap", "chosen", "feat"):
        np.testing.assert_array_equal(fast[k], canon[k], err_msg=k)
    np.testing.assert_array_equal(fast["min_ttft"].view(np.uint32), canon["min_ttft"].view(np.uint32))
    band_check(run.fast_scores(), canon["scores"], what or f"{w.cfg.name} R={w.cfg.R} N={w.cfg.N}")


@pytest.mark.parametrize("name", CONFIGS)
def test_score_parity(name):
    w = workload(name)
    note(f"score parity {name} R={w.cfg.R} N={w.cfg.N}")
    run = GpuRun(w)
    out = run.score()
    assert np.all(out["chosen"] >= 0) and np.all(out["chosen"] < w.cfg.N)
    sel = sampled(w)
    check_scoring(w, out, sel, run=run)
    if w.cfg.R * w.cfg.N <= 600_000:                 # every overlap, not only the sampled requests
        ov = oracle.overlap(w.req_off, w.req_hashes, w.inst_off, w.inst_hashes, threads=16)
        np.testing.assert_array_equal(out["overlap"], ov)
    # invariants that hold at any size
    n = np.diff(w.req_off)
    assert np.all(out["overlap"] >= 0) and np.all(out["overlap"] <= n[:, None])
    row = np.arange(w.cfg.R)
    assert np.array_equal(out["min_ttft"], out["scores"][row, out["chosen"]])
    assert np.all(out["scores"][row, out["chosen"]][:, None] <= out["scores"])
    run.ctx.close()


def _trained_large(kind):
    """The Large-batch model as it stands after online training on the GPU:
    'initial' (the seeded model), 'sgd25' (25 ls_update steps on the update rows
    at the workload's learning rate, as the bench applies), or 'round' (a
    retraining round over a FIFO and replay pool of 5000 each: 5 epochs of
    minibatch 256 in a seeded order)."""
    import torch
    w = workload("large_batch")
    if kind == "initial":
        return w.params
    cfg = w.cfg
    ctx = lodestar.Context(cfg.d, cfg.hidden, cfg.dtype)
    ctx.ls_set_model(w.params, w.mu, w.inv_sigma)
    x, y = to_dev(w.upd_feats), to_dev(w.upd_ttft)
    if kind == "sgd25":
        for _ in range(25):
            ctx.ls_update(x, y, w.lr)
    else:
        ctx.ls_buffer_init(5000, 5000)
        ctx.ls_buffer_push(x[:11000].contiguous(), y[:11000].contiguous())
        st = ctx.ls_buffer_state()
        n = int(st[0]) + int(st[2])
        perm = np.concatenate([np.random.default_rng(e).permutation(n) for e in range(5)]).astype(np.int32)
        ctx.ls_train_round(5, 256, w.lr, perm)
    torch.cuda.synchronize()
    p = ctx.ls_get_model()[0]
    ctx.close()
    assert not np.array_equal(p, w.params)
    return p


@pytest.mark.parametrize("kind", ["initial", "sgd25", "round"])
def test_large_batch_full_size_oracle_parity(kind):
    """All 65,536 x 256 Large-batch pairs against the oracle (bf16 mode, every
    request), for the seeded model and for two trained ones: overlaps, decisions,
    minima and feature rows of the matrix-core path, and every canonical score,
    bit-exact; every fast score within E/8 of its canonical value."""
    w = workload("large_batch")
    note(f"large_batch full-size oracle parity, model {kind}")
    params = _trained_large(kind)
    run = GpuRun(w, params=params)
    canon = run.score()
    fast = run.score(with_scores=False)
    bounds = run.fast_scores()
    run.ctx.close()
    note(f"large_batch full-size oracle parity, model {kind}: oracle on 16 threads")
    ref = oracle.score("bf16", w.cfg.d, w.cfg.hidden, params, w.mu, w.inv_sigma, w.req_off, w.req_hashes,
                       w.prompt_len, w.inst_feat, w.inst_off, w.inst_hashes, threads=16)
    for res in (canon, fast):
        np.testing.assert_array_equal(res["overlap"], ref["overlap"])
        np.testing.assert_array_equal(res["chosen"], ref["chosen"])
        np.testing.assert_array_equal(res["min_ttft"].view(np.uint32),
                                      ref["min_ttft"].astype(np.float32).view(np.uint32))
        np.testing.assert_array_equal(res["feat"], ref["feat"].astype(np.float32))
    want = ref["scores"].astype(np.float32)
    n_bad = int(np.count_nonzero(canon["scores"].view(np.uint32) != want.view(np.uint32)))
    assert n_bad == 0, f"{n_bad} canonical scores differ from the oracle"
    band_check(bounds, want, f"large_batch model {kind}")


@pytest.mark.parametrize("base,R,N,cap", [("large_batch", 37, 13, None), ("large_batch", 130, 65, None),
                                          ("large_batch", 2, 256, None), ("large_batch", 224, 640, 2000),
                                          ("homogeneous", 70, 45, None), ("homogeneous", 9, 300, None),
                                          ("tiny", 40, 33, None)])
def test_bf16_matrix_core_ragged(base, R, N, cap):
    """The matrix-core scorer at each hidden width (256, 128, 64) on ragged
    shapes -- a partial last group of 16 instances, a partial last block of 32
    requests, fewer units than CUs, and (224 x 640: 280 units on 256
    workgroups) workgroups whose units span two instance groups, so that the
    partials in LDS are reloaded mid-run -- with every request checked:
    decisions and minima exact, scores within the band."""
    cfg = synth.dataclasses.replace(synth.CONFIGS[base], dtype="bf16", R=R, N=N)
    if cap is not None:
        cfg = synth.dataclasses.replace(cfg, capacity=(cap,))
    w = synth.generate(cfg)
    assert uses_fast_path(cfg.d, cfg.hidden, cfg.dtype)
    note(f"bf16 matrix-core ragged {base} d={cfg.d} h={cfg.hidden} R={R} N={N}")
    run = GpuRun(w)
    check_scoring(w, run.score(), np.arange(R, dtype=np.int32), run=run)
    run.ctx.close()


def test_bf16_exact_mode_matches_oracle_bitwise():
    """ls_set_exact_scores: every bf16 score on the canonical chain, bit-identical to the oracle."""
    w = workload("large_batch")
    note("bf16 exact mode large_batch")
    run = GpuRun(w, exact=True)
    out = run.score(with_scores=False)
    sel = sampled(w, k=24)
    ref = oracle_score(w, "bf16", sel)
    np.testing.assert_array_equal(out["chosen"][sel], ref["chosen"])
    np.testing.assert_array_equal(out["min_ttft"][sel].view(np.uint32), ref["min_ttft"].astype(np.float32).view(np.uint32))
    np.testing.assert_array_equal(out["feat"][sel], ref["feat"].astype(np.float32))
    run.ctx.close()


def _check_update(w, feats=None, ttft=None):
    """One SGD step through the C ABI against the oracle's, per parameter tensor."""
    feats = w.upd_feats if feats is None else feats
    ttft = w.upd_ttft if ttft is None else ttft
    run = GpuRun(w)
    got = run.update(feats, ttft)
    # ReLU masks are decided in the kernel's precision on both sides (the oracle's
    # forward runs the same fp32 chains); the backward sums are double in the oracle
    mode = mode_of(w)
    ref = oracle.update(mode, w.cfg.d, w.cfg.hidden, w.params, w.mu, w.inv_sigma, feats, ttft, w.lr)
    assert abs(got["loss"] - ref["loss"]) <= 1e-5 * abs(ref["loss"]), (got["loss"], ref["loss"])
    if mode == "fp32":
        # against the double-precision definition only masks of pre-activations
        # within rounding of zero can differ
        ref64 = oracle.update("f64", w.cfg.d, w.cfg.hidden, w.params, w.mu, w.inv_sigma, feats, ttft, w.lr)
        assert np.linalg.norm(got["grad"] - ref64["grad"]) <= 1e-3 * np.linalg.norm(ref64["grad"])
    report = []
    for lname, a, b in layer_slices(w.cfg.d, w.cfg.hidden):
        g, r = got["grad"][a:b], ref["grad"][a:b]
        nrm = np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-30)
        assert nrm <= 1e-4, f"{lname}: norm-wise relative gradient error {nrm}"
        ok, worst, worst3 = grad_ok(g, r)
        assert ok, f"{lname}: elementwise gradient error {worst}"
        report.append(f"{lname} {worst:.1e} ({worst3:.1e} at a 1e-3 floor)")
        # the step: W' - W against the oracle's, allowing one ulp of W' for the final rounding
        dg = got["params"][a:b].astype(np.float64) - w.params[a:b].astype(np.float64)
        dr = ref["params"][a:b].astype(np.float64) - w.params[a:b].astype(np.float64)
        ulp = np.spacing(np.abs(ref["params"][a:b])).astype(np.float64)
        assert np.all(np.abs(dg - dr) <= 1e-4 * np.abs(dr) + ulp), lname
    print(f"update B={feats.shape[0]} worst elementwise gradient error: " + ", ".join(report), flush=True)
    run.ctx.close()


@pytest.mark.parametrize("name", CONFIGS)
def test_update_parity(name):
    w = workload(name)
    note(f"update parity {name} B={w.cfg.update_batch}")
    _check_update(w)


@pytest.mark.parametrize("B", [77, 1030, 1032])
def test_update_parity_bf16_ragged_batch(B):
    """bf16 update at batch sizes that leave a ragged split-K chunk, aligned and not."""
    w = workload("large_batch")
    note(f"bf16 update ragged B={B}")
    _check_update(w, w.upd_feats[:B], w.upd_ttft[:B])


def _golden_model(dtype):
    """The dyadic two-pair example on a d = 8 row: the 3 instance columns carry
    the example, the 5 derived columns have zero weights."""
    g = oracle_pins.golden("mlp_two_pair_example.json")
    W1 = np.zeros((2, 8)); W1[:, :3] = g["W1"]
    layers = [(W1, g["b1"]), (g["W2"], g["b2"]), (g["W3"], g["b3"])]
    params = oracle_pins._pack(layers)
    return g, params


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_golden_two_pair_example(dtype):
    import torch
    note(f"golden two-pair example {dtype}")
    g, params = _golden_model(dtype)
    ctx = lodestar.Context(8, [2, 2], dtype)
    ctx.ls_set_model(params, np.zeros(8, np.float32), np.ones(8, np.float32))
    ctx.ls_load_cache_state(np.array([0, 2, 3], np.int64), to_dev(np.array([5, 6, 5], np.uint64)))
    inst = to_dev(np.array(g["x"], np.float32))
    req_off = to_dev(np.array([0, 2], np.int64))
    req_h = to_dev(np.array([5, 6], np.uint64))
    plen = to_dev(np.array([40], np.int32))
    chosen = torch.zeros(1, dtype=torch.int32, device="cuda")
    mn = torch.zeros(1, dtype=torch.float32, device="cuda")
    sc = torch.zeros(2, dtype=torch.float32, device="cuda")
    ov = torch.zeros(2, dtype=torch.int32, device="cuda")
    ft = torch.zeros(8, dtype=torch.float32, device="cuda")
    ctx.ls_score_batch(req_off, req_h, plen, inst, chosen, mn, sc, ov, ft)
    torch.cuda.synchronize()
    assert sc.cpu().tolist() == g["scores"]
    assert chosen.item() == g["chosen"] and mn.item() == g["scores"][0]
    assert ov.cpu().tolist() == [2, 1]
    np.testing.assert_array_equal(ft.cpu().numpy(), np.array([1, 2, 0.5, 40, 2, 2, 32 / 40, 8], np.float32))
    # one SGD step on the two pairs (derived columns zero)
    sg = g["sgd"]
    feats = np.zeros((2, 8), np.float32); feats[:, :3] = g["x"]
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    grad = torch.zeros(ctx.n_params, dtype=torch.float32, device="cuda")
    ctx.ls_update(to_dev(feats), to_dev(np.array(sg["ttft"], np.float32)), sg["lr"], loss, grad)
    torch.cuda.synchronize()
    assert loss.item() == sg["loss"]
    dW1 = np.zeros((2, 8)); dW1[:, :3] = sg["dW1"]
    want_grad = oracle_pins._pack([(dW1, sg["db1"]), (sg["dW2"], sg["db2"]), (sg["dW3"], sg["db3"])])
    np.testing.assert_array_equal(grad.cpu().numpy(), want_grad)
    W1n = np.zeros((2, 8)); W1n[:, :3] = sg["W1_new"]
    want = oracle_pins._pack([(W1n, sg["b1_new"]), (sg["W2_new"], sg["b2_new"]), (sg["W3_new"], sg["b3_new"])])
    np.testing.assert_array_equal(ctx.ls_get_model()[0], want)
    ctx.close()


def _adversarial_workload():
    """Hand-built cache state and requests covering the edge cases of the overlap."""
    E = (1 << 64) - 1
    caches = [
        [],                                  # empty cache
        [11, 22, 33, 44, 55, 66, 77, 88],    # everything of request 1
        [11, 22, 44, 55],                    # a gap at 33
        [0, E, 11, 11, 22, 22],              # 0, the all-ones key, duplicates
        [E],                                 # only the all-ones key
        [22, 33, 44],                        # missing the first block
        list(range(1000, 1400)),             # unrelated, forces several buckets
    ]
    reqs = [
        ([], 10),                            # prompt shorter than one block
        ([11, 22, 33, 44, 55, 66, 77, 88], 140),
        ([11, 22, 33, 44], 64),
        ([0, E, 11, 22, 5], 80),
        ([E, E, 7], 50),
        ([E], 0),                            # L = 0 (kappa defined as 0)
        (list(range(1000, 1300)), 4800),     # long run inside one instance
        ([11], 16),
    ]
    inst_off, inst_h = oracle_pins._csr(caches)
    req_off, req_h = oracle_pins._csr([r for r, _ in reqs])
    L = np.array([l for _, l in reqs], np.int32)
    return inst_off, inst_h, req_off, req_h, L


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_adversarial_overlaps_and_features(dtype):
    note(f"adversarial overlaps {dtype}")
    inst_off, inst_h, req_off, req_h, L = _adversarial_workload()
    base = workload("tiny")
    N, R = len(inst_off) - 1, len(req_off) - 1
    rng = np.random.default_rng(4)
    d = base.cfg.d
    w = synth.Workload(cfg=synth.dataclasses.replace(base.cfg, R=R, N=N, dtype=dtype), req_off=req_off,
                       req_hashes=req_h, prompt_len=L, req_group=np.zeros(R, np.int32), inst_off=inst_off,
                       inst_hashes=inst_h, inst_feat=rng.uniform(0, 4, (N, d - 5)).astype(np.float32),
                       params=base.params, mu=base.mu, inv_sigma=base.inv_sigma, upd_feats=base.upd_feats,
                       upd_ttft=base.upd_ttft, lr=base.lr)
    run = GpuRun(w)
    out = run.score()
    want = np.array([[oracle_pins._brute_overlap(r, c) for c in
                      [list(inst_h[inst_off[i]:inst_off[i + 1]]) for i in range(N)]]
                     for r in [list(req_h[req_off[k]:req_off[k + 1]]) for k in range(R)]])
    np.testing.assert_array_equal(out["overlap"], want)
    check_scoring(w, out, np.arange(R, dtype=np.int32), run=run)


_PHI = 0x9E3779B97F4A7C15
_PHI_INV = pow(_PHI, -1, 1 << 64)


def _bucket(key, nb):
    """Home bucket of a key in a table of nb buckets (the library's bucket rule)."""
    return (((key * _PHI) % (1 << 64) >> 32) * nb) >> 32


def _keys_homed_at(rng, b, nb, count):
    """Distinct keys whose home bucket in a table of nb buckets is b."""
    lo = -(-(b << 32) // nb)
    hi = -(-((b + 1) << 32) // nb)
    out = set()
    while len(out) < count:
        h = (int(rng.integers(lo, hi)) << 32) | int(rng.integers(0, 1 << 32))
        k = (h * _PHI_INV) % (1 << 64)
        assert _bucket(k, nb) == b
        if k != (1 << 64) - 1:
            out.add(k)
    return sorted(out)


@pytest.mark.parametrize("case", ["queued", "requeue_all"])
def test_table_overflow_paths(case):
    """Keys piled onto the last bucket of a table segment and of the whole table
    overflow the segment being built; the build must still place every key where
    a lookup finds it, through the overflow queue or, when more keys overflow
    than the queue holds, through re-insertion of every key."""
    note(f"table overflow {case}")
    rng = np.random.default_rng(11)
    seg = 2048
    if case == "queued":
        cnt = 12000                          # 3000 buckets: segments of 2048 and 952
        nb = (cnt + 3) // 4
        at_seg_end = _keys_homed_at(rng, seg - 1, nb, 60)
        at_tab_end = _keys_homed_at(rng, nb - 1, nb, 60)
        rest = [int(x) for x in rng.integers(0, 1 << 63, cnt - 120)]
        big = rest[:5000] + at_seg_end + rest[5000:] + at_tab_end
        piles = [at_seg_end, at_tab_end]
    else:
        cnt = 20000                          # every key homed at the last bucket of segment 0
        nb = (cnt + 3) // 4
        pile = _keys_homed_at(rng, seg - 1, nb, cnt)
        big = list(pile)
        piles = [pile[:300], pile[-300:]]
    caches = [big, big[:7000], [int(x) for x in rng.integers(0, 1 << 63, 50)]]
    absent = [_keys_homed_at(np.random.default_rng(99), seg - 1, nb, 2)[0],
              _keys_homed_at(np.random.default_rng(98), nb - 1, nb, 2)[0]]
    absent = [k for k in absent if k not in set(big)]
    reqs = []
    for p in piles:
        reqs.append(p)                       # a run made of overflowed keys only
        reqs.append(p[:25] + absent[:1] + p[25:40])
        reqs.append(list(reversed(p[:50])))
    reqs.append(big[:200])
    reqs.append(big[4990:5100])
    reqs.append(absent + big[:10])
    inst_off, inst_h = oracle_pins._csr(caches)
    req_off, req_h = oracle_pins._csr(reqs)
    L = np.array([16 * len(r) + 3 for r in reqs], np.int32)
    base = workload("tiny")
    N, R, d = len(caches), len(reqs), base.cfg.d
    w = synth.Workload(cfg=synth.dataclasses.replace(base.cfg, R=R, N=N), req_off=req_off, req_hashes=req_h,
                       prompt_len=L, req_group=np.zeros(R, np.int32), inst_off=inst_off, inst_hashes=inst_h,
                       inst_feat=np.random.default_rng(5).uniform(0, 4, (N, d - 5)).astype(np.float32),
                       params=base.params, mu=base.mu, inv_sigma=base.inv_sigma, upd_feats=base.upd_feats,
                       upd_ttft=base.upd_ttft, lr=base.lr)
    run = GpuRun(w)
    out = run.score()
    want = oracle.overlap(req_off, req_h, inst_off, inst_h)
    np.testing.assert_array_equal(out["overlap"], want)
    assert out["overlap"][0, 0] == len(piles[0])
    check_scoring(w, out, np.arange(R, dtype=np.int32), run=run)


_FP_MUL = 0xD6E8FEB86659FD93
_FP_MUL_INV = pow(_FP_MUL, -1, 1 << 64)


def _fp_twin(key):
    """A different key with the same 32-bit fingerprint as `key` under the
    library's fingerprint rule (high word of key * _FP_MUL mod 2^64): the low
    bit of the product flipped and mapped back."""
    return (((key * _FP_MUL) % (1 << 64) ^ 1) * _FP_MUL_INV) % (1 << 64)


def _semi_join_workload(case):
    """Instance 0 holds a shared chain A and a pile of keys homed in its first
    table segment, placed last in its input; requests lead with A + 3 blocks and
    follow with A + a continuation.  run_overflow: the pile overfills the
    segment's run, so its later keys reach the table only through the overflow
    pass, and the continuations are taken among them.  requeue_all: a pile so
    large that the overflow queue itself overflows.  collisions: continuations
    whose fingerprint some other cached key shares, cached or not.
    widely_cached: every cached continuation also on eight more instances, more
    (continuation, instance) matches than the pair table of a batch this size
    holds.  Instance 3 holds A and every third cached continuation."""
    rng = np.random.default_rng({"run_overflow": 41, "requeue_all": 42, "collisions": 43, "widely_cached": 44}[case])
    filler = lambda k: [int(x) for x in rng.integers(0, 1 << 63, k)]
    A = filler(5)
    cnt = 30000
    nb = (cnt + 3) // 4
    P = {"run_overflow": 15000, "requeue_all": 25000, "collisions": 0, "widely_cached": 15000}[case]
    pile = set()
    while len(pile) < P:
        b = int(rng.integers(0, 2048))
        pile.update(_keys_homed_at(rng, b, nb, 1))
    pile = [k for k in pile if k not in set(A)]
    rng.shuffle(pile)
    conts, cached_conts = [], set()
    if case == "collisions":
        X = filler(60)                        # not cached; their twins are
        Y = filler(60)                        # cached; their twins are continuations too
        twins_x = [_fp_twin(k) for k in X]
        big = A + twins_x + Y + filler(cnt - 5 - 120)
        conts = X + Y + [_fp_twin(k) for k in Y]
        cached_conts = set(Y)
    else:
        big = A + filler(cnt - 5 - len(pile)) + pile
        conts = pile[-300:] + filler(40)      # late pile keys, and keys cached nowhere
        cached_conts = set(pile[-300:])
    held = [k for k in conts if k in cached_conts]
    caches = [big, A[:3] + filler(200), [], A + held[::3] + filler(100)]
    if case == "widely_cached":
        caches += [A + held + filler(50) for _ in range(8)]
    reqs = [(A + filler(3), 16 * 8)]          # the leader (longest of group A)
    for k in conts:
        reqs.append((A + [k], 16 * 6 + 5))
    for k in conts[:50]:
        reqs.append((A + [k] + A[:1], 16 * 7))
    inst_off, inst_h = oracle_pins._csr(caches)
    req_off, req_h = oracle_pins._csr([r for r, _ in reqs])
    L = np.array([l for _, l in reqs], np.int32)
    return inst_off, inst_h, req_off, req_h, L, cached_conts, conts


@pytest.mark.parametrize("mode", [1, 2])
@pytest.mark.parametrize("case", ["run_overflow", "requeue_all", "collisions", "widely_cached"])
def test_semi_join_fingerprints(case, mode):
    """The semi-join over the fingerprints a table build leaves: continuations
    cached only through the build's overflow pass, a build whose overflow queue
    overflowed (its keys then are not all listed, so every continuation counts
    as cached), fingerprints shared by distinct keys, and continuations cached
    on many instances (more matches than the pair table holds).  With the join
    on (mode 1) and off (mode 2), every overlap equals the oracle's."""
    note(f"semi-join fingerprints {case}, join mode {mode}")
    inst_off, inst_h, req_off, req_h, L, cached_conts, conts = _semi_join_workload(case)
    base = workload("tiny")
    N, R, d = len(inst_off) - 1, len(req_off) - 1, base.cfg.d
    w = synth.Workload(cfg=synth.dataclasses.replace(base.cfg, R=R, N=N), req_off=req_off, req_hashes=req_h,
                       prompt_len=L, req_group=np.zeros(R, np.int32), inst_off=inst_off, inst_hashes=inst_h,
                       inst_feat=np.random.default_rng(9).uniform(0, 4, (N, d - 5)).astype(np.float32),
                       params=base.params, mu=base.mu, inv_sigma=base.inv_sigma, upd_feats=base.upd_feats,
                       upd_ttft=base.upd_ttft, lr=base.lr)
    run = GpuRun(w, prefix_join=mode)
    out = run.score()
    want = oracle.overlap(req_off, req_h, inst_off, inst_h)
    np.testing.assert_array_equal(out["overlap"], want)
    # the continuations that are cached extend the run on instance 0, the others stop it at A
    got0 = want[1:1 + len(conts), 0]
    assert np.array_equal(got0 >= 6, np.array([k in cached_conts for k in conts]))
    assert int(np.count_nonzero(got0 >= 6)) == len(cached_conts) > 0
    got3 = want[1:1 + len(conts), 3]
    assert 0 < int(np.count_nonzero(got3 >= 6)) < len(cached_conts)
    check_scoring(w, out, np.arange(R, dtype=np.int32), run=run)
    run.ctx.close()


def _follower_workload(rng):
    """A shared chain A with followers that leave it at different blocks and
    continue with hashes cached on some instances, on none, or equal to the
    all-ones key; plus unrelated keys so the tables span several buckets."""
    E = (1 << 64) - 1
    A = [int(x) for x in rng.integers(0, 1 << 63, 12)]
    X, Y, Z, W2, V = (int(x) for x in rng.integers(0, 1 << 63, 5))
    filler = lambda k: [int(x) for x in rng.integers(0, 1 << 63, k)]
    caches = [
        A[:10] + filler(300),                 # the whole leader chain
        A[:5] + filler(300),                  # part of it
        A[:10] + [X, Y] + filler(300),        # the chain and one follower's continuation
        [],                                   # nothing
        A[:3] + [E] + filler(300),            # the all-ones key after A[:3]
        [X] + A[:6] + filler(300),            # X without the prefix before it
        A[:2] + [W2, V] + filler(300),        # a continuation after two blocks
    ]
    reqs = [
        (A[:10], 170),                        # leader of group A
        (A[:6] + [X, Y, Z], 150),             # continuation cached on instance 2 only
        (A[:4] + [Z], 90),                    # continuation cached nowhere
        (A[:3] + [E, Z], 85),                 # continuation is the all-ones key
        (A[:10], 160),                        # same prompt as the leader
        (A[:7], 120),                         # ends inside the common prefix
        (A[:2] + [W2, V, X], 99),             # continuation cached on instance 6
        (A[:1] + [Z] * 3, 70),                # leaves after one block
        ([X, Y], 40),                         # its own group
        (A[:10] + [Y], 180),                  # longer than the leader: becomes the leader
    ]
    for _ in range(40):                       # more followers with private tails
        k = int(rng.integers(0, 11))
        reqs.append((A[:k] + filler(int(rng.integers(0, 4))), 16 * 16))
    inst_off, inst_h = oracle_pins._csr(caches)
    req_off, req_h = oracle_pins._csr([r for r, _ in reqs])
    L = np.array([max(l, 16 * len(r)) for r, l in reqs], np.int32)
    return inst_off, inst_h, req_off, req_h, L


@pytest.mark.parametrize("pad", [False, True])
@pytest.mark.parametrize("mode", [0, 1, 2])
def test_followers_and_continuations(mode, pad):
    """Followers resolved from the leader, through the semi-join of their
    continuation hashes (mode 1), or by probing (mode 2): identical overlaps.
    pad adds an eighth (empty) cache, so that N % 4 == 0 and followers are
    resolved four instances per thread (mixed hit and miss lanes in one word)."""
    note(f"followers and continuations, join mode {mode}, padded {pad}")
    inst_off, inst_h, req_off, req_h, L = _follower_workload(np.random.default_rng(21))
    if pad:
        inst_off = np.append(inst_off, inst_off[-1])
    base = workload("tiny")
    N, R, d = len(inst_off) - 1, len(req_off) - 1, base.cfg.d
    w = synth.Workload(cfg=synth.dataclasses.replace(base.cfg, R=R, N=N), req_off=req_off, req_hashes=req_h,
                       prompt_len=L, req_group=np.zeros(R, np.int32), inst_off=inst_off, inst_hashes=inst_h,
                       inst_feat=np.random.default_rng(6).uniform(0, 4, (N, d - 5)).astype(np.float32),
                       params=base.params, mu=base.mu, inv_sigma=base.inv_sigma, upd_feats=base.upd_feats,
                       upd_ttft=base.upd_ttft, lr=base.lr)
    run = GpuRun(w, prefix_join=mode)
    out = run.score()
    want = oracle.overlap(req_off, req_h, inst_off, inst_h)
    np.testing.assert_array_equal(out["overlap"], want)
    assert want[1, 2] == 8 and want[1, 0] == 6 and want[6, 6] == 4
    check_scoring(w, out, np.arange(R, dtype=np.int32), run=run)


@pytest.mark.parametrize("mode", [1, 2])
def test_long_runs(mode):
    """Prompts of thousands of blocks: the leaders' runs are extended 256
    positions per round (prompts of 1024 blocks or more) and common prefixes
    compared up to 128 positions per round.  Runs that end at a gap deep in the
    prompt, at the all-ones key, at a window boundary, at the prompt's end, and
    followers that leave the leader deep in the chain."""
    note(f"long runs, join mode {mode}")
    rng = np.random.default_rng(33)
    E = (1 << 64) - 1
    A = [int(x) for x in rng.integers(0, 1 << 63, 3000)]
    A[2222] = E                                  # the all-ones key inside the chain
    filler = lambda k: [int(x) for x in rng.integers(0, 1 << 63, k)]
    caches = [
        A[:1700] + A[1701:2500] + filler(50),    # gap at 1700
        A + filler(10),                          # the whole chain, all-ones key included
        A[:1000],                                # ends at 1000
        A[:2222] + A[2223:],                     # everything but the all-ones key
        [E] + A[:256] + A[257:2048],             # gap at a window boundary
        A[:16 + 256 + 1],                        # run of 273 blocks
        [],
        A[:3000:2],                              # every other block: run 1
    ]
    reqs = [(A, 16 * 3000),                      # the leader
            (A[:2900] + filler(30), 16 * 2930),   # leaves the chain at 2900
            (A[:1300] + filler(5), 16 * 1305),    # leaves at 1300
            (A[:2222], 16 * 2222),               # ends just before the all-ones key
            (A[:2500], 16 * 2500 + 9),
            (filler(1200), 16 * 1200),           # a long prompt of its own group
            (A[:40], 16 * 40)]                   # short follower
    inst_off, inst_h = oracle_pins._csr(caches)
    req_off, req_h = oracle_pins._csr([r for r, _ in reqs])
    L = np.array([l for _, l in reqs], np.int32)
    base = workload("tiny")
    N, R, d = len(inst_off) - 1, len(req_off) - 1, base.cfg.d
    w = synth.Workload(cfg=synth.dataclasses.replace(base.cfg, R=R, N=N), req_off=req_off, req_hashes=req_h,
                       prompt_len=L, req_group=np.zeros(R, np.int32), inst_off=inst_off, inst_hashes=inst_h,
                       inst_feat=np.random.default_rng(8).uniform(0, 4, (N, d - 5)).astype(np.float32),
                       params=base.params, mu=base.mu, inv_sigma=base.inv_sigma, upd_feats=base.upd_feats,
                       upd_ttft=base.upd_ttft, lr=base.lr)
    run = GpuRun(w, prefix_join=mode)
    out = run.score()
    want = oracle.overlap(req_off, req_h, inst_off, inst_h)
    np.testing.assert_array_equal(out["overlap"], want)
    assert list(want[0]) == [1700, 3000, 1000, 2222, 256, 273, 0, 1]
    check_scoring(w, out, np.arange(R, dtype=np.int32), run=run)


@pytest.mark.parametrize("mode", [1, 2])
def test_join_modes_agree_on_a_full_workload(mode):
    """The homogeneous workload with the semi-join forced on and off."""
    w = workload("homogeneous")
    note(f"homogeneous overlaps, join mode {mode}")
    out = GpuRun(w, prefix_join=mode).score()
    sel = sampled(w, k=48)
    want = oracle.overlap(w.req_off, w.req_hashes, w.inst_off, w.inst_hashes, sel=sel)
    np.testing.assert_array_equal(out["overlap"][sel], want)


@pytest.mark.parametrize("name", CONFIGS)
def test_prefix_closed_search(name):
    """The run-end search for prefix-closed caches (the synthetic caches are,
    see test_inputs_cpu.py) gives the oracle's overlaps and decisions."""
    w = workload(name)
    note(f"prefix-closed search {name}")
    run = GpuRun(w, prefix_closed=True)
    out = run.score()
    sel = sampled(w)
    want = oracle.overlap(w.req_off, w.req_hashes, w.inst_off, w.inst_hashes, sel=sel)
    np.testing.assert_array_equal(out["overlap"][sel], want)
    check_scoring(w, out, sel, run=run)


@pytest.mark.parametrize("name", ["large_batch", "long_context", "heterogeneous", "tiny"])
def test_prefix_closed_equals_general_at_full_size(name):
    """Every overlap, decision and minimum of the full batch with the caches
    declared prefix-closed (leaders' run-end search from block 1, followers
    galloping from their common prefix) equals the general walk's: the
    synthetic caches are prefix-closed, so both are exact.  Long-context and
    Tiny also take the wave-per-request common-prefix pass."""
    w = workload(name)
    note(f"prefix-closed against the general walk at full size {name}")
    outs = []
    for closed in (False, True):
        run = GpuRun(w, prefix_closed=closed)
        outs.append(run.score(with_scores=False))
        run.ctx.close()
    for k in ("overlap", "chosen", "min_ttft"):
        a, b = np.asarray(outs[0][k]), np.asarray(outs[1][k])
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), k


def test_ties_go_to_lowest_instance():
    """Instances with identical state and cache score identically; the lowest id wins."""
    note("exact ties")
    base = workload("tiny")
    cfg = base.cfg
    N = cfg.N
    lists = [base.inst_hashes[base.inst_off[i]:base.inst_off[i + 1]] for i in range(N)]
    feat = base.inst_feat.copy()
    for i in range(N):                       # instances come in identical pairs (i, i ^ 1)
        lists[i] = lists[i & ~1]
        feat[i] = feat[i & ~1]
    inst_off = np.zeros(N + 1, np.int64); inst_off[1:] = np.cumsum([len(x) for x in lists])
    w = synth.dataclasses.replace(base, inst_off=inst_off, inst_hashes=np.concatenate(lists), inst_feat=feat)
    run = GpuRun(w)
    out = run.score()
    assert np.all(out["chosen"] % 2 == 0)
    np.testing.assert_array_equal(out["scores"][:, 0::2], out["scores"][:, 1::2])
    check_scoring(w, out, np.arange(cfg.R, dtype=np.int32), run=run)


@pytest.mark.parametrize("R,N", [(1, 1), (37, 13), (5, 300), (130, 65)])
def test_ragged_shapes(R, N):
    note(f"ragged shapes R={R} N={N}")
    w = workload("homogeneous", R=R, N=N)
    out = GpuRun(w).score()
    check_scoring(w, out, np.arange(R, dtype=np.int32))
    got = GpuRun(w).update(w.upd_feats[:77], w.upd_ttft[:77])
    ref = oracle.update("fp32", w.cfg.d, w.cfg.hidden, w.params, w.mu, w.inv_sigma, w.upd_feats[:77],
                        w.upd_ttft[:77], w.lr)
    ok, worst, _ = grad_ok(got["grad"], ref["grad"])
    assert ok, worst


def test_deterministic_and_reload():
    """Two contexts, two runs each: identical bits; the model round-trips bitwise."""
    note("determinism and reload")
    w = workload("heterogeneous")
    a, b = GpuRun(w), GpuRun(w)
    oa, ob = a.score(), b.score()
    for k in ("scores", "overlap", "chosen", "feat"):
        assert np.array_equal(oa[k].view(np.uint8), ob[k].view(np.uint8)), k
    p, mu, s = a.ctx.ls_get_model()
    assert np.array_equal(p.view(np.uint32), w.params.view(np.uint32))
    assert np.array_equal(mu, w.mu) and np.array_equal(s, w.inv_sigma)
    ua, ub = a.update(), b.update()
    assert np.array_equal(ua["grad"].view(np.uint32), ub["grad"].view(np.uint32))
    assert np.array_equal(ua["params"].view(np.uint32), ub["params"].view(np.uint32))
    # a model read back and installed elsewhere scores identically
    c = GpuRun(w, params=ua["params"])
    assert np.array_equal(c.score()["scores"].view(np.uint32), a.score()["scores"].view(np.uint32))


@pytest.mark.parametrize("name", ["homogeneous", "large_batch"])
def test_results_independent_of_launch_geometry(name):
    """The same batch and update with the launches sized for the whole GPU, for
    37 compute units and for 8 (ls_set_cu_limit): persistent kernels then walk
    many more units per workgroup, grid-stride loops many more items per thread.
    Every output is bitwise the same."""
    w = workload(name)
    results = []
    for cus in (0, 37, 8):
        note(f"launch geometry {name}: {cus or 'all'} compute units")
        run = GpuRun(w)
        run.ctx.ls_set_cu_limit(cus)
        res = {"canon": run.score()}
        if uses_fast_path(w.cfg.d, w.cfg.hidden, w.cfg.dtype):
            res["fast"] = run.score(with_scores=False)
            res["bounds"] = run.fast_scores()
        res["update"] = run.update()
        run.ctx.close()
        results.append(res)
    flat = lambda r: [(f"{k}.{j}", np.ascontiguousarray(v).view(np.uint8)) for k, d in r.items() for j, v in d.items()
                      if isinstance(v, np.ndarray)]
    base = flat(results[0])
    for other in results[1:]:
        for (ka, a), (kb, b) in zip(base, flat(other)):
            assert ka == kb and np.array_equal(a, b), ka


def test_abi_errors_on_device():
    import torch
    note("ABI error paths")
    w = workload("tiny")
    cfg = w.cfg
    ctx = lodestar.Context(cfg.d, cfg.hidden, cfg.dtype)
    req_off, req_h = to_dev(w.req_off), to_dev(w.req_hashes)
    plen, feat = to_dev(w.prompt_len), to_dev(w.inst_feat)
    chosen = torch.zeros(cfg.R, dtype=torch.int32, device="cuda")
    with pytest.raises(lodestar.LodestarError) as e:
        ctx.ls_score_batch(req_off, req_h, plen, feat, chosen)
    assert e.value.code == lodestar.LS_ERR_STATE
    ctx.ls_set_model(w.params, w.mu, w.inv_sigma)
    with pytest.raises(lodestar.LodestarError) as e:
        ctx.ls_score_batch(req_off, req_h, plen, feat, chosen)
    assert e.value.code == lodestar.LS_ERR_STATE and "cache" in str(e.value)
    ctx.ls_load_cache_state(w.inst_off, to_dev(w.inst_hashes))
    lib = ctx.lib
    import ctypes
    P = ctypes.c_void_p
    ptr = lambda t: P(t.data_ptr())
    assert lib.ls_score_batch(ctx.h, cfg.R, cfg.N + 1, ptr(req_off), ptr(req_h), ptr(plen), ptr(feat), ptr(chosen),
                              None, None, None, None, None) == lodestar.LS_ERR_STATE
    assert lib.ls_score_batch(ctx.h, cfg.R, cfg.N, ptr(req_off), ptr(req_h), ptr(plen), ptr(feat), None,
                              None, None, None, None, None) == lodestar.LS_ERR_INVALID
    assert lib.ls_score_batch(ctx.h, -1, cfg.N, *([None] * 10)) == lodestar.LS_ERR_INVALID
    assert lib.ls_score_batch(ctx.h, 0, cfg.N, *([None] * 10)) == lodestar.LS_OK
    params = np.ascontiguousarray(w.params)
    assert lib.ls_set_model(ctx.h, params.ctypes.data_as(P), params.size - 1, params.ctypes.data_as(P),
                            params.ctypes.data_as(P), None) == lodestar.LS_ERR_INVALID
    bad_off = np.array([0, 5, 3], np.int64)
    assert lib.ls_load_cache_state(ctx.h, 2, bad_off.ctypes.data_as(P), ptr(req_h), None) == lodestar.LS_ERR_INVALID
    assert lib.ls_update(ctx.h, 0, ptr(feat), ptr(feat), 0.1, None, None, None) == lodestar.LS_ERR_INVALID
    assert lib.ls_update(ctx.h, 4, ptr(feat), ptr(feat), float("nan"), None, None, None) == lodestar.LS_ERR_INVALID
    assert lib.ls_set_chain_kernels(ctx.h, 2) == lodestar.LS_ERR_INVALID
    assert lib.ls_set_chain_kernels(ctx.h, -1) == lodestar.LS_ERR_INVALID
    assert lib.ls_set_chain_kernels(None, 0) == lodestar.LS_ERR_INVALID
    # the context still works after rejected calls
    ctx.ls_score_batch(req_off, req_h, plen, feat, chosen)
    torch.cuda.synchronize()
    ctx.close()
