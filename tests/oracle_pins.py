"""Pins for the CPU oracle: checks against facts fixed outside the oracle.

Each ``pin_*`` function raises AssertionError when the oracle disagrees with a
hand-derived fixture, a closed form, an invariant of the definition, a library
routine on a special case, or brute force on tiny inputs.  The same functions
run against the real oracle (test_oracle_pins.py) and against deliberately
broken copies of it (test_oracle_mutants.py), which must each fail at least one.
"""
from __future__ import annotations

import itertools
import json
import os

import numpy as np

import oracle

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def golden(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def _csr(lists, dtype=np.uint64):
    off = np.zeros(len(lists) + 1, dtype=np.int64)
    off[1:] = np.cumsum([len(x) for x in lists])
    flat = np.array([v for x in lists for v in x], dtype=dtype) if off[-1] else np.zeros(0, dtype)
    return off, flat


def _pack(layers):
    """layers: list of (W [out, in], b [out]) -> flat fp32 in the oracle's packing."""
    return np.concatenate([np.concatenate([np.asarray(W, np.float64).ravel(), np.asarray(b, np.float64)])
                           for W, b in layers]).astype(np.float32)


def _brute_overlap(req, cache):
    """Largest k such that every one of the first k request blocks is cached."""
    s = set(int(v) for v in cache)
    best = 0
    for k in range(len(req) + 1):
        if all(int(h) in s for h in req[:k]):
            best = k
    return best


# ---------------------------------------------------------------------------
# bfloat16 rounding
# ---------------------------------------------------------------------------
def pin_bf16_definition():
    f = np.float32
    hand = [
        (1.0, 1.0),
        (1.00390625, 1.0),                      # 1 + 2^-8: tie -> even mantissa (1.0)
        (1.01171875, 1.015625),                 # 1 + 3*2^-8: tie -> even (1 + 2^-6)
        (float(np.nextafter(f(1.00390625), f(2))), 1.0078125),   # just above the tie rounds up
        (float(np.nextafter(f(1.00390625), f(0))), 1.0),         # just below rounds down
        (-2.0078125, -2.0),                     # -(2 + 2^-7): tie -> even
        (2.0 ** -149, 0.0),                     # smallest subnormal vanishes
        (2.0 ** -134, 0.0),                     # half the subnormal quantum 2^-133: tie -> 0
        (3 * 2.0 ** -134, 2.0 ** -132),         # 1.5 quanta: tie -> even (2 quanta)
        (float(np.finfo(np.float32).max), float("inf")),
        (-0.0, -0.0),
    ]
    for x, want in hand:
        got = float(oracle.bf16_round(np.float32(x)))
        assert got == want and np.signbit(got) == np.signbit(want), (x, got, want)
    assert np.isnan(oracle.bf16_round(np.float32("nan")))
    # torch's float -> bfloat16 conversion is round-to-nearest-even as well
    import torch
    rng = np.random.default_rng(7)
    vals = np.concatenate([
        rng.standard_normal(3000).astype(np.float32),
        (rng.standard_normal(500) * 1e-39).astype(np.float32),
        (rng.integers(1, 1 << 16, 500).astype(np.uint32) << np.uint32(16) | np.uint32(0x8000)).view(np.float32),
    ])
    vals = vals[np.isfinite(vals)]
    ref = torch.from_numpy(vals).to(torch.bfloat16).to(torch.float32).numpy()
    ours = oracle.bf16_round(vals)
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))


# ---------------------------------------------------------------------------
# prefix overlap
# ---------------------------------------------------------------------------
def pin_overlap_worked_example():
    g = golden("prefix_worked_example.json")
    caches = [c["cache"] for c in g["cases"]]
    inst_off, inst_h = _csr(caches)
    req_off, req_h = _csr([g["request_hashes"]])
    ov = oracle.overlap(req_off, req_h, inst_off, inst_h)[0]
    assert list(ov) == [c["overlap"] for c in g["cases"]], ov
    for c, o in zip(g["cases"], ov):
        x = oracle.features("fp32", np.zeros(1, np.float32), g["prompt_len"], g["n_blocks"], o)
        assert x[3] == o == c["hit_tokens"] // g["block_tokens"]
        assert x[4] == float(np.float32(c["hit_tokens"]) / np.float32(g["prompt_len"]))
        assert x[5] == g["prompt_len"] - c["hit_tokens"]


def pin_overlap_bruteforce_exhaustive():
    """Every request over a 5-letter alphabet up to 4 blocks against every cache subset."""
    alphabet = [0, 1, 2, 3, (1 << 64) - 1]
    reqs = [list(t) for k in range(5) for t in itertools.product(alphabet, repeat=k)]
    caches = [[a for bit, a in enumerate(alphabet) if m >> bit & 1] for m in range(1 << len(alphabet))]
    req_off, req_h = _csr(reqs)
    inst_off, inst_h = _csr(caches)
    ov = oracle.overlap(req_off, req_h, inst_off, inst_h)
    for r, req in enumerate(reqs):
        for i, cache in enumerate(caches):
            assert ov[r, i] == _brute_overlap(req, cache), (req, cache, ov[r, i])


def pin_overlap_invariants(seed=3, trials=60):
    rng = np.random.default_rng(seed)
    for _ in range(trials):
        n = int(rng.integers(0, 12))
        req = rng.integers(0, 20, n).astype(np.uint64)
        cache = rng.choice(20, int(rng.integers(0, 20)), replace=False).astype(np.uint64)
        extra = rng.integers(0, 20, 5).astype(np.uint64)
        bigger = np.concatenate([cache, extra])
        perm_dup = np.concatenate([cache[::-1], cache[: len(cache) // 2]])
        full = np.concatenate([cache, req])
        k = int(rng.integers(0, n + 1))
        reqs = [req, req[:k]]
        caches = [cache, bigger, perm_dup, full]
        ov = oracle.overlap(*_csr([list(r) for r in reqs]), *_csr([list(c) for c in caches]))
        l = ov[0, 0]
        assert 0 <= l <= n
        assert ov[0, 1] >= l                         # monotone in cache contents
        assert ov[0, 2] == l                         # order and duplicates of the cache are irrelevant
        assert ov[0, 3] == n                         # a cache holding every block gives a full run
        assert ov[1, 0] == min(l, k)                 # truncating the request truncates the run
        if n and int(req[0]) not in set(cache.tolist()):
            assert l == 0
        assert l == _brute_overlap(list(req), list(cache))


# ---------------------------------------------------------------------------
# features
# ---------------------------------------------------------------------------
def pin_features_closed_form():
    row = np.array([3.0, -1.5, 0.25], np.float32)
    x = oracle.features("fp32", row, 64, 4, 2)
    assert list(x) == [3.0, -1.5, 0.25, 64.0, 4.0, 2.0, 0.5, 32.0]
    x = oracle.features("f64", row, 87, 5, 2)
    assert x[6] == 32.0 / 87.0 and x[7] == 55.0
    x = oracle.features("fp32", row, 87, 5, 2)
    assert x[6] == float(np.float32(32.0) / np.float32(87.0))
    x = oracle.features("bf16", row, 0, 0, 0)
    assert x[6] == 0.0 and x[7] == 0.0
    x = oracle.features("f64", row, 8191, 511, 511)
    assert x[6] == 8176.0 / 8191.0 and x[7] == 15.0


# ---------------------------------------------------------------------------
# forward pass and argmin
# ---------------------------------------------------------------------------
def _golden_net():
    g = golden("mlp_two_pair_example.json")
    params = _pack([(g["W1"], g["b1"]), (g["W2"], g["b2"]), (g["W3"], g["b3"])])
    return g, params


def pin_forward_golden():
    g, params = _golden_net()
    d = g["d"]
    mu = np.zeros(d, np.float32); s = np.ones(d, np.float32)
    for mode in ("f64", "fp32", "bf16"):
        t = oracle.forward(mode, d, g["hidden"], params, mu, s, np.array(g["x"]))
        assert list(t) == g["scores"], (mode, t)
        assert oracle.argmin(t)[0] == g["chosen"]
    # normalisation: x' = x * 2 + 1 with mu = 1 and inv_sigma = 0.5 gives the same inputs back
    xs = np.array(g["x"]) * 2.0 + 1.0
    t = oracle.forward("fp32", d, g["hidden"], params, np.ones(d, np.float32), np.full(d, 0.5, np.float32), xs)
    assert list(t) == g["scores"]


def pin_forward_bf16_rounding_points():
    """One-unit nets (d = 1, hidden = [1]) in which exactly one quantity is not a
    bfloat16 number, so each rounding point of the bf16 mode shows by itself.
    Values are powers-of-two sums worked by hand; the fp32 mode keeps them."""
    one = np.ones(1, np.float32); zero = np.zeros(1, np.float32)
    cases = [
        # (x, W1, b1, W2, b2, bf16 result, fp32 result)
        (1 + 2**-8 + 2**-10, 1.0, 0.0, 1.0, 0.0, 1 + 2**-7, 1 + 2**-8 + 2**-10),   # input rounds up (0.625 quanta)
        (1.0, 1 + 2**-10, 0.0, 1.0, 0.0, 1.0, 1 + 2**-10),                         # layer-1 weight rounds down
        (3.0, 1 + 2**-7, 0.0, 1.0, 0.0, 3 + 2**-5, 3 + 3 * 2**-7),                  # activation 3.0234375: tie -> 3.03125
        (1.0, 1.0, 0.0, 1 + 2**-10, 0.0, 1.0, 1 + 2**-10),                         # head weight rounds down
        (1.0, 1.0, 2**-12, 1.0, 2**-12, 1 + 2**-12, 1 + 2**-11),                  # activation rounds, biases do not
    ]
    for x, w1, b1, w2, b2, want_bf, want_32 in cases:
        params = np.array([w1, b1, w2, b2], np.float32)
        t_bf = oracle.forward("bf16", 1, [1], params, zero, one, np.array([[x]]))[0]
        t_32 = oracle.forward("fp32", 1, [1], params, zero, one, np.array([[x]]))[0]
        assert t_bf == want_bf and t_32 == want_32, (x, w1, b1, w2, b2, t_bf, t_32)


def pin_forward_linear_special_case(seed=5):
    """Positive weights, biases and inputs keep every ReLU open: the net is the
    affine map W3 (W2 (W1 x + b1) + b2) + b3."""
    rng = np.random.default_rng(seed)
    d, hidden = 7, [9, 6]
    dims = [d, *hidden, 1]
    layers = [(rng.uniform(0.1, 1.0, (dims[i + 1], dims[i])), rng.uniform(0.0, 0.5, dims[i + 1]))
              for i in range(3)]
    params = _pack(layers)
    mu = rng.uniform(-1, 0, d).astype(np.float32)
    s = rng.uniform(0.5, 2, d).astype(np.float32)
    x = rng.uniform(0, 3, (11, d))
    t = oracle.forward("f64", d, hidden, params, mu, s, x)
    W = [np.asarray(L[0], np.float32).astype(np.float64) for L in layers]
    b = [np.asarray(L[1], np.float32).astype(np.float64) for L in layers]
    xt = (x - mu.astype(np.float64)) * s.astype(np.float64)
    ref = (W[2] @ (W[1] @ (W[0] @ xt.T + b[0][:, None]) + b[1][:, None]) + b[2][:, None])[0]
    assert np.allclose(t, ref, rtol=1e-12, atol=0), (t, ref)


def pin_forward_relu_closed():
    """A last hidden layer pushed far negative outputs zeros: t = b_out exactly."""
    rng = np.random.default_rng(9)
    d, hidden = 6, [8, 5]
    layers = [(rng.standard_normal((8, 6)), rng.standard_normal(8)),
              (rng.uniform(-1, 0, (5, 8)), np.full(5, -50.0)),
              (rng.standard_normal((1, 5)), np.array([0.375]))]
    params = _pack(layers)
    x = rng.uniform(-1, 1, (9, d))
    for mode in ("f64", "fp32", "bf16"):
        t = oracle.forward(mode, d, hidden, params, np.zeros(d, np.float32), np.ones(d, np.float32), x)
        assert np.all(t == 0.375), (mode, t)


def pin_forward_lowp_bound(seed=11):
    """The fp32 chain stays within the classic dot-product error bound of the
    double-precision definition (gamma_K per layer, propagated with |W|)."""
    rng = np.random.default_rng(seed)
    d, hidden = 16, [32, 24]
    dims = [d, *hidden, 1]
    layers = [(rng.normal(0, np.sqrt(2 / dims[i]), (dims[i + 1], dims[i])), rng.uniform(-0.1, 0.1, dims[i + 1]))
              for i in range(3)]
    params = _pack(layers)
    mu = np.zeros(d, np.float32); s = np.ones(d, np.float32)
    x = rng.standard_normal((200, d)).astype(np.float32).astype(np.float64)
    t64 = oracle.forward("f64", d, hidden, params, mu, s, x)
    t32 = oracle.forward("fp32", d, hidden, params, mu, s, x)
    # crude rigorous-enough bound: relative 1e-5 of the magnitude of |W| |a| sums
    absnet = _pack([(np.abs(np.asarray(W, np.float32)), np.abs(np.asarray(b, np.float32))) for W, b in layers])
    mag = oracle.forward("f64", d, hidden, absnet, mu, s, np.abs(x))
    assert np.all(np.abs(t32 - t64) <= 1e-5 * mag + 1e-30), np.max(np.abs(t32 - t64) / mag)
    assert not np.array_equal(t32, t64)              # the modes really do differ in rounding


def pin_argmin_rules():
    nan, inf = float("nan"), float("inf")
    cases = [
        ([3.0, 1.0, 2.0], 1),
        ([1.0, 1.0, 0.5, 0.5], 2),                # exact tie -> lowest id
        ([0.0, -0.0], 0), ([-0.0, 0.0], 0),       # signed zeros compare equal
        ([nan, inf, 5.0], 2),
        ([nan, inf], 1),                          # NaN ranks after +inf
        ([nan, nan, nan], 0),                     # all NaN -> instance 0
        ([-inf, -inf], 0),
        ([7.0], 0),
    ]
    for s, want in cases:
        got, m = oracle.argmin(np.array(s))
        assert got == want, (s, got)
        assert (np.isnan(m) and np.isnan(s[want])) or m == s[want]


# ---------------------------------------------------------------------------
# online update
# ---------------------------------------------------------------------------
def _check_grad(res, want, d, hidden):
    shapes = [(2, 3), (2,), (2, 2), (2,), (1, 2), (1,)]
    names = ["dW1", "db1", "dW2", "db2", "dW3", "db3"]
    off = 0
    for name, shp in zip(names, shapes):
        n = int(np.prod(shp))
        got = res["grad"][off:off + n]
        assert np.array_equal(got, np.asarray(want[name], np.float64).ravel()), (name, got, want[name])
        off += n


def pin_update_golden():
    g, params = _golden_net()
    d = g["d"]
    mu = np.zeros(d, np.float32); s = np.ones(d, np.float32)
    sg = g["sgd"]
    for mode in ("f64", "fp32", "bf16"):
        res = oracle.update(mode, d, g["hidden"], params, mu, s, np.array(g["x"]), np.array(sg["ttft"]), sg["lr"])
        assert res["loss"] == sg["loss"], (mode, res["loss"])
        _check_grad(res, sg, d, g["hidden"])
        want = _pack([(sg["W1_new"], sg["b1_new"]), (sg["W2_new"], sg["b2_new"]), (sg["W3_new"], sg["b3_new"])])
        assert np.array_equal(res["params"], want), (mode, res["params"], want)
    one = g["sgd_first_sample_only"]
    res = oracle.update("f64", d, g["hidden"], params, mu, s, np.array(g["x"][:1]), np.array(one["ttft"]), 0.25)
    assert res["loss"] == one["loss"]
    _check_grad(res, one, d, g["hidden"])


def pin_update_bf16_rounding_points():
    """One-unit net, one sample (d = 1, hidden = [1], x = 1, W1 = 1, b = 0,
    head weight w = 1 + 2^-7).  t = w, g = 2 (t - y); the hidden-unit gradient
    is w * g.  In bf16 mode g and w * g are rounded to bfloat16 before they
    multiply anything; in f64 mode nothing is.  Values worked by hand."""
    w = 1 + 2**-7
    params = np.array([1.0, 0.0, w, 0.0], np.float32)
    one = np.ones(1, np.float32); zero = np.zeros(1, np.float32)
    x = np.ones((1, 1), np.float32)
    cases = [
        # y, mode, loss, [dW1, db1, dW2, db2]
        (0.0, "bf16", 1.01568603515625, [2.03125, 2.03125, 2.015625, 2.015625]),        # w*g = 2.0313720703125 rounds
        (0.0, "f64", 1.01568603515625, [2.0313720703125, 2.0313720703125, 2.015625, 2.015625]),
        (2**-9, "bf16", 1.011753082275390625, [2.03125, 2.03125, 2.015625, 2.015625]),  # g = 2.01171875 rounds up
        (2**-9, "f64", 1.011753082275390625, [2.027435302734375, 2.027435302734375, 2.01171875, 2.01171875]),
    ]
    for y, mode, loss, grad in cases:
        res = oracle.update(mode, 1, [1], params, zero, one, x, np.array([y], np.float32), 0.0)
        assert res["loss"] == loss and list(res["grad"]) == grad, (y, mode, res["loss"], res["grad"])


def pin_update_invariants(seed=13):
    rng = np.random.default_rng(seed)
    d, hidden = 6, [7, 5]
    dims = [d, *hidden, 1]
    params = _pack([(rng.normal(0, 0.6, (dims[i + 1], dims[i])), rng.uniform(-0.2, 0.2, dims[i + 1])) for i in range(3)])
    mu = rng.normal(0, 1, d).astype(np.float32); s = rng.uniform(0.5, 2, d).astype(np.float32)
    x = rng.normal(0, 2, (8, d)).astype(np.float32); y = rng.uniform(0, 2, 8).astype(np.float32)
    r0 = oracle.update("f64", d, hidden, params, mu, s, x, y, 0.0)
    assert np.array_equal(r0["params"], params)                    # lr = 0 leaves the model unchanged
    # the batch gradient is the mean of single-sample gradients
    parts = [oracle.update("f64", d, hidden, params, mu, s, x[b:b + 1], y[b:b + 1], 0.1)["grad"] for b in range(8)]
    assert np.allclose(r0["grad"], np.mean(parts, axis=0), rtol=1e-12, atol=1e-15)
    # the step moves against the gradient
    r1 = oracle.update("f64", d, hidden, params, mu, s, x, y, 1e-3)
    dp = r1["params"].astype(np.float64) - params.astype(np.float64)
    assert np.sum(dp * r0["grad"]) < 0
    # loss agrees with the forward pass of the same precision
    for mode in ("f64", "fp32", "bf16"):
        t = oracle.forward(mode, d, hidden, params, mu, s, x.astype(np.float64))
        r = oracle.update(mode, d, hidden, params, mu, s, x, y, 0.0)
        assert np.isclose(r["loss"], np.mean((t - y.astype(np.float64)) ** 2), rtol=1e-13), mode


def pin_update_finite_difference(seed=17):
    """Central differences of the forward-pass loss, in double precision."""
    rng = np.random.default_rng(seed)
    d, hidden = 5, [6, 4]
    dims = [d, *hidden, 1]
    params = _pack([(rng.normal(0, 0.8, (dims[i + 1], dims[i])), rng.uniform(-0.3, 0.3, dims[i + 1])) for i in range(3)])
    mu = rng.normal(0, 0.5, d).astype(np.float32); s = rng.uniform(0.5, 1.5, d).astype(np.float32)
    x = rng.normal(0, 2, (6, d)); y = rng.uniform(-1, 1, 6)
    res = oracle.update("f64", d, hidden, params, mu, s, x.astype(np.float32), y.astype(np.float32), 0.0)

    def loss(p):
        t = oracle.forward("f64", d, hidden, p, mu, s, x.astype(np.float32).astype(np.float64))
        return np.mean((t - y.astype(np.float32).astype(np.float64)) ** 2)

    h = 2.0 ** -14
    fd = np.zeros(params.shape[0])
    for k in range(params.shape[0]):
        pp = params.copy(); pm = params.copy()
        pp[k] += np.float32(h); pm[k] -= np.float32(h)
        fd[k] = (loss(pp) - loss(pm)) / (float(pp[k]) - float(pm[k]))
    err = np.abs(fd - res["grad"]) / np.maximum(np.abs(res["grad"]), 1e-6)
    assert np.mean(err < 1e-6) >= 0.95 and np.median(err) < 1e-8, (np.sort(err)[-5:], np.median(err))


# ---------------------------------------------------------------------------
# the whole scoring pass against an independent numpy pipeline on tiny inputs
# ---------------------------------------------------------------------------
def pin_score_pipeline_bruteforce(seed=19):
    rng = np.random.default_rng(seed)
    N, R, d_inst, hidden = 5, 9, 3, [6, 4]
    d = d_inst + 5
    caches = [list(rng.choice(12, int(rng.integers(0, 12)), replace=False)) for _ in range(N)]
    reqs = [list(rng.integers(0, 12, int(rng.integers(0, 8)))) for _ in range(R)]
    L = np.array([16 * len(r) + int(rng.integers(0, 16)) for r in reqs], np.int32)
    feat = rng.uniform(0, 4, (N, d_inst)).astype(np.float32)
    dims = [d, *hidden, 1]
    layers = [(rng.normal(0, 0.7, (dims[i + 1], dims[i])), rng.uniform(-0.2, 0.2, dims[i + 1])) for i in range(3)]
    params = _pack(layers)
    mu = rng.normal(0, 1, d).astype(np.float32); s = rng.uniform(0.2, 1, d).astype(np.float32)
    req_off, req_h = _csr(reqs); inst_off, inst_h = _csr(caches)
    out = oracle.score("f64", d, hidden, params, mu, s, req_off, req_h, L, feat, inst_off, inst_h)
    W = [np.asarray(Lr[0], np.float32).astype(np.float64) for Lr in layers]
    b = [np.asarray(Lr[1], np.float32).astype(np.float64) for Lr in layers]
    for r in range(R):
        ov = np.array([_brute_overlap(reqs[r], c) for c in caches])
        assert np.array_equal(out["overlap"][r], ov)
        x = np.concatenate([feat.astype(np.float64),
                            np.full((N, 1), float(L[r])), np.full((N, 1), float(len(reqs[r]))),
                            ov[:, None].astype(np.float64),
                            (16.0 * ov / L[r])[:, None] if L[r] else np.zeros((N, 1)),
                            (L[r] - 16.0 * ov)[:, None]], axis=1)
        a = (x - mu.astype(np.float64)) * s.astype(np.float64)
        for l in range(3):
            a = a @ W[l].T + b[l]
            if l < 2:
                a = np.maximum(a, 0.0)
        t = a[:, 0]
        assert np.allclose(out["scores"][r], t, rtol=1e-12, atol=1e-14), (out["scores"][r], t)
        best = int(np.lexsort((np.arange(N), t))[0])
        assert out["chosen"][r] == best and out["min_ttft"][r] == out["scores"][r][best]
        assert np.array_equal(out["feat"][r], x[best])


# ---------------------------------------------------------------------------
# routing policy: splitmix64, rendezvous hashing, Alg. 1 / Alg. 2, Alg. 3 / Alg. 4
# ---------------------------------------------------------------------------
_GAMMA = 0x9E3779B97F4A7C15
_M64 = (1 << 64) - 1


def pin_splitmix64_published():
    """splitmix64 seeded with 0: the first three outputs of the published generator."""
    want = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    assert [oracle.splitmix64_mix((_GAMMA * (k + 1)) & _M64) for k in range(3)] == want


def pin_hrw_topk(seed=23, trials=40):
    """Rendezvous top-K by brute-force sorting of the weights; adding an
    instance moves at most one key slot, and only to the new instance."""
    rng = np.random.default_rng(seed)
    for _ in range(trials):
        N = int(rng.integers(1, 40)); K = int(rng.integers(1, 6)); key = int(rng.integers(0, 1 << 63)) * 2 + 1
        w = [oracle.splitmix64_mix((key + _GAMMA * (i + 1)) & _M64) for i in range(N + 1)]
        brute = sorted(range(N), key=lambda i: (-w[i], i))[:K]
        got = list(oracle.hrw_topk(N, key, K))
        assert got == brute, (got, brute)
        grown = set(oracle.hrw_topk(N + 1, key, K))
        assert grown - set(got) <= {N} and len(grown ^ set(got)) <= 2


def _brute_alg1(m, c, theta, k):
    """Alg. 1 as printed: imbalance check, then sort by (match desc, count asc)
    and take the first instance not above mean + k * std."""
    N = len(c)
    least = min(range(N), key=lambda i: (c[i], i))
    if max(c) - min(c) > theta:
        return least
    mu = sum(c) / N
    sigma = (sum((x - mu) ** 2 for x in c) / N) ** 0.5
    for i in sorted(range(N), key=lambda i: (-float(m[i]), c[i], i)):
        if c[i] <= mu + k * sigma:
            return i
    return least


def _brute_alg2(m, c, tau):
    N = len(c)
    best = min(range(N), key=lambda i: (-float(m[i]), i))
    if float(m[best]) > tau:
        return best
    return min(range(N), key=lambda i: (c[i], i))


def pin_heuristics_hand():
    f = np.float32
    assert oracle.heuristic(1, f([0.9, 0.5, 0.1]), [10.0, 0.0, 5.0], theta=5.0, k=1.0) == 1      # imbalanced
    # balanced: mean 2, std 0.816, k = 0 -> counts <= 2 qualify; best match among them is instance 2
    assert oracle.heuristic(1, f([0.9, 0.5, 0.9]), [3.0, 2.0, 1.0], theta=10.0, k=0.0) == 2
    # a count exactly at the limit qualifies (mean 2, k = 0)
    assert oracle.heuristic(1, f([0.1, 0.9, 0.3]), [1.0, 2.0, 3.0], theta=10.0, k=0.0) == 1
    # nobody qualifies (negative k): least loaded
    assert oracle.heuristic(1, f([0.9, 0.5, 0.1]), [2.0, 1.0, 3.0], theta=10.0, k=-5.0) == 1
    m = f([0.2, 0.6, 0.6])
    assert oracle.heuristic(2, m, [5.0, 1.0, 0.0], tau=0.5) == 1                                  # above threshold
    assert oracle.heuristic(2, m, [5.0, 1.0, 0.0], tau=float(f(0.6))) == 2                         # equal: not above
    assert oracle.heuristic(2, m, [5.0, 1.0, 0.0], tau=0.7) == 2


def pin_heuristics_bruteforce(seed=29, trials=300):
    rng = np.random.default_rng(seed)
    for _ in range(trials):
        N = int(rng.integers(1, 9))
        m = np.float32(rng.choice([0.0, 0.25, 0.5, 0.75, 1.0], N))
        c = [float(v) for v in rng.integers(0, 6, N)]
        theta = float(rng.choice([1.0, 3.0, 100.0])); k = float(rng.choice([-1.0, 0.0, 0.5, 1.0]))
        tau = float(rng.choice([0.0, 0.25, 0.5, 0.9]))
        assert oracle.heuristic(1, m, c, theta=theta, k=k) == _brute_alg1(m, c, theta, k)
        assert oracle.heuristic(2, m, c, tau=tau) == _brute_alg2(m, c, tau)


def _route_case(seed=31, R=12, N=8, dup=False):
    """A small workload with the oracle's own (pinned) overlaps and scores."""
    from paper_2606_00946_amd import synth
    w = synth.generate("tiny", R=R, N=N)
    feat = w.inst_feat.copy()
    inst_lists = [w.inst_hashes[w.inst_off[i]:w.inst_off[i + 1]] for i in range(N)]
    if dup:                                        # instances in identical pairs -> exact score ties
        for i in range(N):
            inst_lists[i] = inst_lists[i & ~1]
            feat[i] = feat[i & ~1]
    inst_off = np.zeros(N + 1, np.int64); inst_off[1:] = np.cumsum([len(x) for x in inst_lists])
    inst_h = np.concatenate(inst_lists)
    rnd = np.random.default_rng(seed).integers(0, 1 << 32, (R, 3), dtype=np.uint64).astype(np.uint32)
    res = oracle.score("fp32", w.cfg.d, w.cfg.hidden, w.params, w.mu, w.inv_sigma, w.req_off, w.req_hashes,
                       w.prompt_len, feat, inst_off, inst_h)
    sc, ch = res["scores"], res["chosen"]
    ov = oracle.overlap(w.req_off, w.req_hashes, inst_off, inst_h)
    return w, feat, inst_off, inst_h, rnd, sc, ch, ov


def _run_route(case, **pol):
    w, feat, inst_off, inst_h, rnd, _, _, _ = case
    return oracle.route("fp32", w.cfg.d, w.cfg.hidden, w.params, w.mu, w.inv_sigma, w.req_off, w.req_hashes,
                        w.prompt_len, feat, inst_off, inst_h, oracle.policy(**pol), rnd)


def _scaled(u, n):
    return (int(u) * int(n)) >> 32


def pin_route_branches():
    case = _route_case()
    w, feat, inst_off, inst_h, rnd, sc, ch, ov = case
    R, N = w.cfg.R, w.cfg.N
    d_inst = w.cfg.d - 5
    counts = (0, 1)
    cnt = [float(feat[i, 0]) + float(feat[i, 1]) for i in range(N)]
    L = w.prompt_len
    kappa = np.array([[np.float32(0.0) if L[r] == 0 else np.float32(np.float32(16 * ov[r, i]) / np.float32(L[r]))
                       for i in range(N)] for r in range(R)], np.float32)
    base = dict(heuristic=1, count_cols=counts, theta_imbal=4.0, overload_k=0.5, n_samples=100, n_min=10)
    heur_want = [_brute_alg1(kappa[r], cnt, 4.0, 0.5) for r in range(R)]
    # plain greedy: the argmin of the scores
    c_, st, hr = _run_route(case, **base)
    assert list(c_) == list(ch) and all(st == oracle.ROUTE_OK) and list(hr) == heur_want
    # cold start: heuristic for everybody; n_samples == n_min is not a cold start
    c_, st, _ = _run_route(case, **{**base, "n_samples": 9})
    assert all(st == oracle.ROUTE_COLD_START) and list(c_) == heur_want
    c_, st, _ = _run_route(case, **{**base, "n_samples": 10})
    assert all(st == oracle.ROUTE_OK)
    # out-of-range instance column: every request falls back; a bound equal to the value is in range
    lo = np.full(w.cfg.d, -np.inf, np.float32); hi = np.full(w.cfg.d, np.inf, np.float32)
    hi2 = hi.copy(); hi2[2] = np.nextafter(np.float32(feat[:, 2].max()), np.float32(-np.inf))
    c_, st, _ = _run_route(case, **base, lo=lo, hi=hi2)
    assert all(st == oracle.ROUTE_OOD) and list(c_) == heur_want
    lo3 = lo.copy(); lo3[2] = np.float32(feat[:, 2].min())
    _, st, _ = _run_route(case, **base, lo=lo3, hi=hi)
    assert all(st == oracle.ROUTE_OK)
    # out-of-range request column (prompt length): only the long prompts fall back
    hi4 = hi.copy(); hi4[d_inst] = np.float32(np.median(L))
    c_, st, _ = _run_route(case, **base, lo=lo, hi=hi4)
    for r in range(R):
        assert (st[r] == oracle.ROUTE_OOD) == (L[r] > hi4[d_inst])
    # exploration: epsilon = 1 always, epsilon = 0 never; the draw is compared with floor(eps * 2^32)
    c_, st, _ = _run_route(case, **base, epsilon=1.0)
    assert all(st == oracle.ROUTE_EXPLORED) and list(c_) == [_scaled(rnd[r, 1], N) for r in range(R)]
    rnd[0, 0] = 1 << 31; rnd[1, 0] = (1 << 31) - 1
    _, st, _ = _run_route(case, **base, epsilon=0.5)
    assert st[0] == oracle.ROUTE_OK and st[1] == oracle.ROUTE_EXPLORED
    # tie-break: a huge margin makes every instance near-best
    c_, st, _ = _run_route(case, **base, delta=1e30)
    assert all(st == oracle.ROUTE_TIEBREAK) and list(c_) == [_scaled(rnd[r, 2], N) for r in range(R)]
    # K-filter forced on (saturation and benefit thresholds below any value)
    kf = dict(base, kv_col=4, tau_sat=-1.0, tau_ben=-1.0)
    first = [int(w.req_hashes[w.req_off[r]]) for r in range(R)]
    c_, st, _ = _run_route(case, **kf, k_filter=1)
    assert all(st == oracle.ROUTE_KFILTER)
    assert list(c_) == [int(oracle.hrw_topk(N, first[r], 1)[0]) for r in range(R)]
    c_, st, _ = _run_route(case, **kf, k_filter=N)
    assert list(c_) == list(ch)
    # with K = 2 and a huge margin the tie-break stays inside the filtered pair
    c_, st, _ = _run_route(case, **kf, k_filter=2, delta=1e30)
    for r in range(R):
        pair = sorted(oracle.hrw_topk(N, first[r], 2))
        assert c_[r] == pair[_scaled(rnd[r, 2], 2)] and st[r] == oracle.ROUTE_KFILTER | oracle.ROUTE_TIEBREAK
    # benefit threshold above every kappa * L: the filter stays off
    c_, st, _ = _run_route(case, **dict(kf, tau_ben=1e30), k_filter=1)
    assert list(c_) == list(ch) and all(st == oracle.ROUTE_OK)
    # Alg. 2 as the fallback heuristic
    _, _, hr = _run_route(case, **dict(base, heuristic=2, prefix_tau=0.25))
    assert list(hr) == [_brute_alg2(kappa[r], cnt, float(np.float32(0.25))) for r in range(R)]


def pin_route_exact_ties():
    """Duplicated instances tie exactly; a zero margin picks uniformly among the tied ones."""
    case = _route_case(dup=True)
    w, feat, inst_off, inst_h, rnd, sc, ch, ov = case
    c_, st, _ = _run_route(case, heuristic=1, count_cols=(0, 1), n_samples=1, n_min=0, delta=0.0)
    for r in range(w.cfg.R):
        tied = [i for i in range(w.cfg.N) if sc[r, i] == sc[r].min()]
        assert len(tied) >= 2
        assert c_[r] == tied[_scaled(rnd[r, 2], len(tied))] and st[r] == oracle.ROUTE_TIEBREAK


# ---------------------------------------------------------------------------
# online-learning data path: embeddings, FIFO, gradient-coreset admission, round
# ---------------------------------------------------------------------------
def _tiny_model():
    from paper_2606_00946_amd import synth
    return synth.generate("tiny")


def _numpy_forward_f64(w, x):
    """(t, last hidden activations) in double, from the packed parameters."""
    d, (h1, h2) = w.cfg.d, w.cfg.hidden
    p = w.params.astype(np.float64)
    o = 0
    W1 = p[o:o + h1 * d].reshape(h1, d); o += h1 * d
    b1 = p[o:o + h1]; o += h1
    W2 = p[o:o + h2 * h1].reshape(h2, h1); o += h2 * h1
    b2 = p[o:o + h2]; o += h2
    W3 = p[o:o + h2]; o += h2
    b3 = p[o]
    xt = (x.astype(np.float64) - w.mu) * w.inv_sigma
    a1 = np.maximum(xt @ W1.T + b1, 0)
    a2 = np.maximum(a1 @ W2.T + b2, 0)
    return a2 @ W3 + b3, a2


def pin_embedding_definition():
    w = _tiny_model()
    x, y = w.upd_feats[:50], w.upd_ttft[:50]
    e = oracle.embed("fp32", w.cfg.d, w.cfg.hidden, w.params, w.mu, w.inv_sigma, x, y)
    t, a2 = _numpy_forward_f64(w, x)
    ref = (t - y.astype(np.float64))[:, None] * a2
    assert e.shape == ref.shape
    assert np.linalg.norm(e - ref) <= 1e-4 * np.linalg.norm(ref)
    # a zero residual gives a zero embedding
    tk = oracle.forward("fp32", w.cfg.d, w.cfg.hidden, w.params, w.mu, w.inv_sigma, x).astype(np.float32)
    assert np.all(oracle.embed("fp32", w.cfg.d, w.cfg.hidden, w.params, w.mu, w.inv_sigma, x, tk) == 0.0)


def _stream(w, n, dup_every=5):
    """n update rows with every dup_every-th a copy of an earlier one (exact ties)."""
    x = w.upd_feats[:n].copy(); y = w.upd_ttft[:n].copy()
    for k in range(dup_every, n, dup_every):
        x[k] = x[k // 2]; y[k] = y[k // 2]
    return x, y


def _sq(a, b):
    s = 0.0
    for u, v in zip(a, b):
        s += (u - v) * (u - v)
    return s


def _check_buffer_stream(w, x, y, F, P, chunks):
    """Push x in the given chunk sizes and compare the FIFO and the pool with a
    brute-force replay that recomputes every nearest-neighbour distance."""
    cfg = w.cfg
    buf = oracle.Buffer(cfg.d, F, P)
    pool, fifo, evicted, s = [], [], 0, 0
    for k in chunks:
        chunk = list(range(s, min(s + k, len(x))))
        cands = []
        for b in chunk:
            if len(fifo) == F:
                cands.append(fifo.pop(0))
            fifo.append(b)
        rows = pool + cands
        if rows:
            E = oracle.embed("fp32", cfg.d, cfg.hidden, w.params, w.mu, w.inv_sigma, x[rows], y[rows])
            emb = {r: list(E[q]) for q, r in enumerate(rows)}
        for c in cands:
            if len(pool) < P:
                pool.append(c)
                continue
            dc = min(_sq(emb[c], emb[m]) for m in pool)
            nn = [min(_sq(emb[pool[a]], emb[pool[b]]) for b in range(len(pool)) if b != a) for a in range(len(pool))]
            js = min(range(len(pool)), key=lambda a: (nn[a], a))
            if dc > nn[js]:
                pool[js] = c
        oracle.buffer_push("fp32", cfg.hidden, w.params, w.mu, w.inv_sigma, buf, x[chunk], y[chunk])
        evicted += len(cands)
        fx, fy = buf.fifo_rows()
        np.testing.assert_array_equal(fx, x[fifo]); np.testing.assert_array_equal(fy, y[fifo])
        rx, ry = buf.replay_rows()
        assert int(buf.rep_count[0]) == min(P, evicted)
        np.testing.assert_array_equal(rx, x[pool]); np.testing.assert_array_equal(ry, y[pool])
        s += k


def pin_buffer_fifo_and_gcr(seed=37):
    """FIFO keeps the newest rows in order; the pool follows the admission rule."""
    w = _tiny_model()
    x, y = _stream(w, 90)
    rng = np.random.default_rng(seed)
    _check_buffer_stream(w, x, y, 12, 6, [int(v) for v in rng.integers(1, 9, 40)])
    # an exact tie: the pool holds a duplicated pair (distance 0) and a candidate
    # duplicates another member (distance 0): it must not be admitted
    a, b, z = w.upd_feats[0], w.upd_feats[1], w.upd_feats[2]
    ya, yb, yz = w.upd_ttft[0], w.upd_ttft[1], w.upd_ttft[2]
    x2 = np.stack([a, a, b, b, z]); y2 = np.array([ya, ya, yb, yb, yz], np.float32)
    _check_buffer_stream(w, x2, y2, 1, 3, [1] * 5)


def pin_train_round_composition():
    """A round is minibatch SGD over the FIFO (oldest first) then the pool, in
    the given order, the last minibatch possibly shorter."""
    w = _tiny_model()
    cfg = w.cfg
    buf = oracle.Buffer(cfg.d, 10, 4)
    x, y = w.upd_feats[:23], w.upd_ttft[:23]
    oracle.buffer_push("fp32", cfg.hidden, w.params, w.mu, w.inv_sigma, buf, x, y)
    fx, fy = buf.fifo_rows(); rx, ry = buf.replay_rows()
    X = np.concatenate([fx, rx]); Y = np.concatenate([fy, ry])
    n = X.shape[0]
    perm = np.concatenate([np.random.default_rng(e).permutation(n) for e in range(2)]).astype(np.int32)
    got, _ = oracle.train_round("fp32", cfg.hidden, w.params, w.mu, w.inv_sigma, buf, 2, 4, 0.05, perm)
    p = w.params.copy()
    for e in range(2):
        order = perm[e * n:(e + 1) * n]
        for s0 in range(0, n, 4):
            idx = order[s0:s0 + 4]
            p = oracle.update("fp32", cfg.d, cfg.hidden, p, w.mu, w.inv_sigma, X[idx], Y[idx], 0.05)["params"]
    np.testing.assert_array_equal(got, p)
    same, _ = oracle.train_round("fp32", cfg.hidden, w.params, w.mu, w.inv_sigma, buf, 0, 4, 0.05)
    np.testing.assert_array_equal(same, w.params)


# ---------------------------------------------------------------------------
# prefix-index maintenance (Section 2: the gateway records routed prefixes,
# engines evict least recently used blocks)
# ---------------------------------------------------------------------------
def _lists(off, h, st):
    return [list(zip(h[off[i]:off[i + 1]].tolist(), st[off[i]:off[i + 1]].tolist())) for i in range(len(off) - 1)]


def pin_commit_worked_example():
    """LRU worked by hand, capacity 3: a new batch evicts the oldest entries; within
    a request the head is newer than the tail; touching a cached block refreshes it;
    requests sent nowhere change nothing; capacity 0 keeps nothing."""
    x, y, z, a, b, c = 101, 102, 103, 201, 202, 301
    off, h = _csr([[x, y, z], [c]])
    st = oracle.initial_stamps(off)
    cap = [3, 0]
    # epoch 1: request 0 = [a, b] -> instance 0; request 1 = [c] -> nowhere (-1)
    off, h, st = oracle.commit(off, h, st, cap, *_csr([[a, b], [c]]), [0, -1], 1)
    assert _lists(off, h, st)[0] == [(a, oracle.stamp(1, 0, 0)), (b, oracle.stamp(1, 0, 1)), (z, 3)]
    assert _lists(off, h, st)[1] == []                    # capacity 0 empties instance 1
    # epoch 2: request 0 = [c] -> instance 1 (capacity 0), request 1 = [y, a] -> instance 0:
    # y comes back, a is refreshed, b (epoch 1) now beats z (loaded), z goes
    off, h, st = oracle.commit(off, h, st, cap, *_csr([[c], [y, a]]), [1, 0], 2)
    got = _lists(off, h, st)
    assert [k for k, _ in got[0]] == [y, a, b]
    assert got[0][0][1] == oracle.stamp(2, 1, 0) and got[0][1][1] == oracle.stamp(2, 1, 1)
    assert got[0][2][1] == oracle.stamp(1, 0, 1)
    assert oracle.stamp(2, 0, 0) > oracle.stamp(1, 5, 0) > oracle.stamp(1, 4, 0) > oracle.stamp(1, 4, 1)


def _lru_reference(state, cap, reqs, chosen):
    """Per-access LRU lists (an OrderedDict per instance, most recent at the end):
    the batch's accesses in order of recency -- requests in order, each request's
    blocks from its tail to its head -- then each instance trimmed from its
    least recent end."""
    from collections import OrderedDict
    for r, blocks in enumerate(reqs):
        i = chosen[r]
        if not 0 <= i < len(state):
            continue
        for blk in reversed(blocks):
            state[i].pop(blk, None)
            state[i][blk] = True
    for i, d in enumerate(state):
        while len(d) > cap[i]:
            d.popitem(last=False)
    return state


def pin_commit_matches_lru_lists():
    """Against a per-access LRU simulation on random small batches: repeated blocks
    within and across requests, the all-ones hash, requests routed nowhere or out of
    range, capacities from 0 up, several commits in a row."""
    from collections import OrderedDict
    rng = np.random.default_rng(77)
    for trial in range(6):
        N = int(rng.integers(1, 5))
        cap = rng.integers(0, 9, N).tolist()
        pool = np.array(rng.integers(1, 40, 30).tolist() + [2**64 - 1], dtype=np.uint64)
        lists0 = [[int(v) for v in dict.fromkeys(rng.choice(pool, int(rng.integers(0, 8))).tolist())]
                  for _ in range(N)]
        state = [OrderedDict((k, True) for k in l) for l in lists0]
        off, h = _csr(lists0)
        st = oracle.initial_stamps(off)
        for epoch in range(1, 5):
            R = int(rng.integers(0, 7))
            reqs = [[int(v) for v in rng.choice(pool, int(rng.integers(0, 6)))] for _ in range(R)]
            chosen = rng.integers(-1, N + 1, R).astype(np.int32)
            state = _lru_reference(state, cap, reqs, chosen)
            roff, rh = _csr(reqs) if R else (np.zeros(1, np.int64), np.zeros(0, np.uint64))
            off, h, st = oracle.commit(off, h, st, cap, roff, rh, chosen, epoch)
            got = _lists(off, h, st)
            for i in range(N):
                assert [k for k, _ in got[i]] == list(reversed(state[i])), (trial, epoch, i)
                stamps = [v for _, v in got[i]]
                assert stamps == sorted(stamps, reverse=True) and len(set(stamps)) == len(stamps)


def _chain(parent_hash, token_block):
    """A block's hash: a 64-bit mix of its parent's hash and its own tokens."""
    z = (parent_hash * 0x100000001B3 ^ (token_block + 0x9E3779B97F4A7C15)) & (2**64 - 1)
    z = ((z ^ (z >> 31)) * 0xD6E8FEB86659FD93) & (2**64 - 1)
    return z ^ (z >> 29)


def pin_commit_keeps_prefixes():
    """Tail-first eviction keeps every instance's cache closed under prefixes: with
    chained block hashes (a block's hash covers all earlier blocks), after any
    sequence of commits every cached block's parent block is cached too."""
    rng = np.random.default_rng(5)
    N = 3
    cap = [12, 20, 7]
    parent = {}
    prefixes = []                                        # shared request prefixes
    for g in range(4):
        hsh, blocks = 0, []
        for t in range(int(rng.integers(2, 6))):
            nh = _chain(hsh, 1000 * g + t)
            parent[nh] = hsh
            blocks.append(nh)
            hsh = nh
        prefixes.append(blocks)
    off, h = _csr([[] for _ in range(N)])
    st = oracle.initial_stamps(off)
    uid = 0
    for epoch in range(1, 9):
        reqs = []
        for _ in range(int(rng.integers(1, 6))):
            g = int(rng.integers(0, len(prefixes)))
            blocks = list(prefixes[g][:int(rng.integers(1, len(prefixes[g]) + 1))])
            hsh = blocks[-1]
            for _t in range(int(rng.integers(0, 5))):       # a private suffix
                uid += 1
                nh = _chain(hsh, 10**6 + uid)
                parent[nh] = hsh
                blocks.append(nh)
                hsh = nh
            reqs.append(blocks)
        chosen = rng.integers(0, N, len(reqs)).astype(np.int32)
        off, h, st = oracle.commit(off, h, st, cap, *_csr(reqs), chosen, epoch)
        for i, entries in enumerate(_lists(off, h, st)):
            cached = {k for k, _ in entries}
            assert len(cached) <= cap[i]
            for k in cached:
                p = parent[k]
                assert p == 0 or p in cached, (epoch, i)
        assert int(off[-1]) > 0


# ---------------------------------------------------------------------------
# dropout while training (Section 4.1: the predictor uses dropout 0.1)
# ---------------------------------------------------------------------------
def _one_unit_net():
    """d = 6 inputs, one hidden unit, head: z = 0.5 x0 + 0.25, t = 1 + 2 relu(z)."""
    W1 = np.zeros((1, 6)); W1[0, 0] = 0.5
    return _pack([(W1, [0.25]), ([[2.0]], [1.0])])


def pin_dropout_closed_form():
    """Inverted dropout on a single hidden unit with x0 = 1 (z = 0.75): a kept unit is
    scaled by 1/(1-p), so t = 1 + 2 * 0.75 / (1-p); a dropped one gives t = 1.  The
    observed dropped fraction matches p (binomial bound), and masks differ between
    the rows of one call."""
    params = _one_unit_net()
    mu, isg = np.zeros(6, np.float32), np.ones(6, np.float32)
    x = np.zeros((1, 6), np.float32); x[0, 0] = 1.0
    for mode in ("f64", "fp32", "bf16"):
        vals = []
        for step in range(400):
            out = oracle.update(mode, 6, [1], params, mu, isg, x, [0.0], 0.0, dropout=(0.5, 99, step))
            vals.append(out["loss"])                      # y = 0: loss = t^2
        vals = np.array(vals)
        assert set(np.unique(vals)) == {1.0, 16.0}, (mode, np.unique(vals))
        assert abs((vals == 1.0).mean() - 0.5) < 5 * 0.025, mode
    # p = 0.1: the fp32 scale is the fp32 value of 1/0.9
    s = np.float32(1.0 / 0.9)
    kept_t = np.float32(1.0) + np.float32(2.0) * (np.float32(0.75) * s)
    vals = np.array([oracle.update("fp32", 6, [1], params, mu, isg, x, [0.0], 0.0, dropout=(0.1, 7, k))["loss"]
                     for k in range(3000)])
    assert abs((vals == 1.0).mean() - 0.1) < 5 * np.sqrt(0.09 / 3000)
    assert np.all((vals == 1.0) | (vals == float(kept_t) ** 2))
    # p = 0 is no dropout at all
    plain = oracle.update("fp32", 6, [1], params, mu, isg, x, [0.0], 0.0)
    assert oracle.update("fp32", 6, [1], params, mu, isg, x, [0.0], 0.0, dropout=(0.0, 5, 3))["loss"] == plain["loss"]
    # 64 identical rows in one call: some kept, some dropped (the row is part of the draw)
    X = np.repeat(x, 64, axis=0)
    losses = [oracle.update("f64", 6, [1], params, mu, isg, X, np.zeros(64), 0.0, dropout=(0.5, 3, k))["loss"]
              for k in range(4)]
    assert all(1.0 < l < 16.0 for l in losses), losses


def pin_dropout_gradient_fd():
    """The gradient with dropout is the gradient of the masked network's loss: central
    finite differences of the double-precision loss with the same masks (same seed
    and step), over two hidden layers."""
    rng = np.random.default_rng(12)
    d, hidden, B = 7, [5, 4], 6
    n = oracle.param_count(d, hidden)
    params = (rng.standard_normal(n) * 0.5).astype(np.float32)
    mu = rng.standard_normal(d).astype(np.float32) * 0.1
    isg = (1.0 + rng.random(d)).astype(np.float32)
    X = rng.standard_normal((B, d)).astype(np.float32)
    Y = rng.standard_normal(B).astype(np.float32)
    drop = (0.3, 1234, 17)
    g = oracle.update("f64", d, hidden, params, mu, isg, X, Y, 0.0, dropout=drop)["grad"]
    assert np.count_nonzero(g) > 0
    h = 1e-3
    worst = 0.0
    for t in rng.choice(n, 24, replace=False):
        pp, pm = params.astype(np.float64).copy(), params.astype(np.float64).copy()
        pp[t] += h; pm[t] -= h
        lp = oracle.update("f64", d, hidden, pp.astype(np.float32), mu, isg, X, Y, 0.0, dropout=drop)["loss"]
        lm = oracle.update("f64", d, hidden, pm.astype(np.float32), mu, isg, X, Y, 0.0, dropout=drop)["loss"]
        # the float32 parameters hold pp / pm exactly only up to rounding: use the rounded step
        step = float(np.float32(pp[t])) - float(np.float32(pm[t]))
        fd = (lp - lm) / step
        worst = max(worst, abs(fd - g[t]) / max(1e-3, abs(g[t])))
    assert worst < 2e-3, worst


def pin_train_round_dropout_is_update_sequence():
    """A retraining round with dropout is the sequence of dropout updates over its
    minibatches, minibatch u drawing the masks of update call first_step + u."""
    from paper_2606_00946_amd import synth
    w = synth.generate("tiny")
    cfg = w.cfg
    buf = oracle.Buffer(cfg.d, 10, 4)
    x, y = w.upd_feats[:20], w.upd_ttft[:20]
    oracle.buffer_push("fp32", cfg.hidden, w.params, w.mu, w.inv_sigma, buf, x, y)
    fx, fy = buf.fifo_rows(); rx, ry = buf.replay_rows()
    X = np.concatenate([fx, rx]); Y = np.concatenate([fy, ry])
    n = X.shape[0]
    got, _ = oracle.train_round("fp32", cfg.hidden, w.params, w.mu, w.inv_sigma, buf, 2, 4, 0.05,
                                dropout=(0.2, 55, 100))
    p = w.params.copy()
    step = 100
    for e in range(2):
        for s0 in range(0, n, 4):
            p = oracle.update("fp32", cfg.d, cfg.hidden, p, w.mu, w.inv_sigma, X[s0:s0 + 4], Y[s0:s0 + 4], 0.05,
                              dropout=(0.2, 55, step))["params"]
            step += 1
    np.testing.assert_array_equal(got, p)
    plain, _ = oracle.train_round("fp32", cfg.hidden, w.params, w.mu, w.inv_sigma, buf, 2, 4, 0.05)
    assert not np.array_equal(got, plain)


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_") and callable(v)]
