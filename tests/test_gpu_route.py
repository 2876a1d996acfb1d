"""Routing policy (Alg. 3 / Alg. 4 with the Alg. 1 / Alg. 2 heuristics) through
the C ABI, against the oracle: the routed instance, the status code and the
heuristic's choice are compared exactly, on every workload and on the bf16
matrix-core path (where the candidate band must cover every pair a policy
decision can depend on)."""
import functools

import numpy as np
import pytest

import oracle
from gpu_helpers import note, to_dev
from paper_2606_00946_amd import lodestar, synth

pytestmark = pytest.mark.gpu

BASE = dict(heuristic=1, count_cols=(0, 1), theta_imbal=4.0, overload_k=0.5, n_samples=100, n_min=10)


@functools.lru_cache(maxsize=None)
def workload(name):
    return synth.generate(name)


def policies(w):
    L = w.prompt_len
    d_inst = w.cfg.d - 5
    lo = np.full(w.cfg.d, -np.inf, np.float32)
    hi = np.full(w.cfg.d, np.inf, np.float32)
    hi_req = hi.copy()
    hi_req[d_inst] = np.float32(np.median(L))                 # long prompts are out of range
    return {
        "greedy": dict(BASE),
        "cold_start": dict(BASE, n_samples=5),
        "explore": dict(BASE, epsilon=0.3),
        "tiebreak": dict(BASE, delta=0.02),
        "wide_tiebreak": dict(BASE, delta=0.3),
        "kfilter": dict(BASE, kv_col=4, tau_sat=0.3, tau_ben=64.0, k_filter=2, delta=0.01),
        "kfilter_tiebreak": dict(BASE, kv_col=4, tau_sat=0.3, tau_ben=64.0, k_filter=4, delta=0.3),
        "alg2": dict(BASE, heuristic=2, prefix_tau=0.2, epsilon=0.1),
        "ood_requests": dict(BASE, lo=lo, hi=hi_req, delta=0.0),
    }


def run_route(w, pol, rnd, exact=False):
    import torch
    cfg = w.cfg
    ctx = lodestar.Context(cfg.d, cfg.hidden, cfg.dtype)
    if exact:
        ctx.ls_set_exact_scores(True)
    ctx.ls_set_model(w.params, w.mu, w.inv_sigma)
    inst_h = to_dev(w.inst_hashes)
    ctx.ls_load_cache_state(w.inst_off, inst_h)
    R = cfg.R
    chosen = torch.full((R,), -7, dtype=torch.int32, device="cuda")
    status = torch.full((R,), -7, dtype=torch.int32, device="cuda")
    heur = torch.full((R,), -7, dtype=torch.int32, device="cuda")
    feat = torch.zeros(R * cfg.d, dtype=torch.float32, device="cuda")
    ctx.ls_route_batch(lodestar.make_policy(**pol), to_dev(w.req_off), to_dev(w.req_hashes),
                       to_dev(w.prompt_len.astype(np.int32)), to_dev(w.inst_feat.astype(np.float32)),
                       to_dev(rnd.view(np.int32)), chosen, status, heur, feat)
    torch.cuda.synchronize()
    out = chosen.cpu().numpy(), status.cpu().numpy(), heur.cpu().numpy(), feat.cpu().numpy().reshape(R, cfg.d)
    ctx.close()
    return out


def mode_of(w):
    return "bf16" if w.cfg.dtype == "bf16" else "fp32"


def sample(w, k):
    R = w.cfg.R
    if R <= k:
        return np.arange(R, dtype=np.int32)
    rng = np.random.default_rng(5)
    return np.unique(np.concatenate([[0, R - 1], rng.choice(R, k, replace=False)])).astype(np.int32)


@pytest.mark.parametrize("name,k", [("tiny", 64), ("homogeneous", 64), ("large_batch", 40)])
def test_route_matches_oracle(name, k):
    w = workload(name)
    cfg = w.cfg
    rnd = np.random.default_rng(17).integers(0, 1 << 32, (cfg.R, 3), dtype=np.uint64).astype(np.uint32)
    sel = sample(w, k)
    ov = None
    for pname, pol in policies(w).items():
        note(f"route {name} policy {pname}")
        chosen, status, heur, feat = run_route(w, pol, rnd)
        want = oracle.route(mode_of(w), cfg.d, cfg.hidden, w.params, w.mu, w.inv_sigma, w.req_off, w.req_hashes,
                            w.prompt_len, w.inst_feat, w.inst_off, w.inst_hashes, oracle.policy(**pol), rnd, sel=sel)
        np.testing.assert_array_equal(heur[sel], want[2], err_msg=f"{name}/{pname} heuristic")
        np.testing.assert_array_equal(status[sel], want[1], err_msg=f"{name}/{pname} status")
        np.testing.assert_array_equal(chosen[sel], want[0], err_msg=f"{name}/{pname} chosen")
        if ov is None:
            ov = oracle.overlap(w.req_off, w.req_hashes, w.inst_off, w.inst_hashes, sel=sel)
        d_inst = cfg.d - 5
        for q, r in enumerate(sel):
            i = chosen[r]
            row = np.zeros(cfg.d)
            oracle._load().lso_features(1, d_inst, oracle._ptr(np.ascontiguousarray(w.inst_feat[i], np.float32)),
                                        int(w.prompt_len[r]), int(w.req_off[r + 1] - w.req_off[r]), int(ov[q, i]),
                                        oracle._ptr(row))
            np.testing.assert_array_equal(feat[r], row.astype(np.float32), err_msg=f"{name}/{pname} feat row {r}")
        kinds = status[sel] & 0xFF
        print(f"{name}/{pname}: ok {int((kinds == 0).sum())} cold {int((kinds == 1).sum())} "
              f"ood {int((kinds == 2).sum())} explored {int(((status[sel] & 0x100) != 0).sum())} "
              f"kfilter {int(((status[sel] & 0x200) != 0).sum())} tiebreak {int(((status[sel] & 0x400) != 0).sum())}",
              flush=True)


def test_route_exact_mode_large():
    """The all-canonical path routes identically to the matrix-core path."""
    w = workload("large_batch")
    rnd = np.random.default_rng(23).integers(0, 1 << 32, (w.cfg.R, 3), dtype=np.uint64).astype(np.uint32)
    pol = policies(w)["kfilter"]
    note("route large_batch fast vs exact")
    fast = run_route(w, pol, rnd)
    exact = run_route(w, pol, rnd, exact=True)
    for a, b in zip(fast[:3], exact[:3]):
        np.testing.assert_array_equal(a, b)


def test_route_policy_errors():
    import torch
    w = workload("tiny")
    cfg = w.cfg
    note("route policy errors")
    ctx = lodestar.Context(cfg.d, cfg.hidden, cfg.dtype)
    ctx.ls_set_model(w.params, w.mu, w.inv_sigma)
    ctx.ls_load_cache_state(w.inst_off, to_dev(w.inst_hashes))
    R = cfg.R
    args = (to_dev(w.req_off), to_dev(w.req_hashes), to_dev(w.prompt_len.astype(np.int32)),
            to_dev(w.inst_feat.astype(np.float32)))
    chosen = torch.zeros(R, dtype=torch.int32, device="cuda")
    rnd = to_dev(np.zeros(3 * R, np.int32))
    bad = [dict(BASE, heuristic=3), dict(BASE, count_cols=(0, cfg.d)), dict(BASE, kv_col=cfg.d),
           dict(BASE, k_filter=9), dict(BASE, epsilon=1.5), dict(BASE, theta_imbal=float("nan"))]
    for pol in bad:
        with pytest.raises(lodestar.LodestarError) as e:
            ctx.ls_route_batch(lodestar.make_policy(**pol), *args, rnd, chosen)
        assert e.value.code == lodestar.LS_ERR_INVALID
    with pytest.raises(lodestar.LodestarError) as e:            # exploration needs random words
        ctx.ls_route_batch(lodestar.make_policy(**dict(BASE, epsilon=0.1)), *args, None, chosen)
    assert e.value.code == lodestar.LS_ERR_INVALID
    ctx.close()
