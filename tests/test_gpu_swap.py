"""Double-buffered retraining through the C ABI (Section 4.3.1: training never
stalls routing, a new model replaces the serving one at once; Section 4.3.2).

While the shadow model trains on its own stream, scores on the serving stream
must stay bit-identical to the live model's; after ls_swap_model they must be
bit-identical to those of a fresh context holding the trained weights, the
trained weights must follow the oracle's retraining rounds, the replay pool's
embeddings must have come from the shadow, and training must continue from
the model that now serves."""
import dataclasses

import numpy as np
import pytest

import oracle
from gpu_helpers import GpuRun, layer_slices, note, to_dev
from paper_2606_00946_amd import lodestar, synth

pytestmark = pytest.mark.gpu


def workload(dtype):
    cfg = dataclasses.replace(synth.CONFIGS["homogeneous"], dtype=dtype, R=384, update_batch=600)
    return synth.generate(cfg)


def score_on(run, stream):
    """Enqueue two scoring calls on `stream`: one that asks for the score matrix
    (canonical scores of every pair) and one that does not (on a bf16 context,
    the matrix-core path with canonical rescoring of the band).  Returns the
    first call's decisions and scores, and the second's decisions and minima."""
    import torch
    R, N = run.w.cfg.R, run.w.cfg.N
    chosen = torch.full((R,), -7, dtype=torch.int32, device="cuda")
    scores = torch.zeros(R * N, dtype=torch.float32, device="cuda")
    run.ctx.ls_score_batch(run.req_off, run.req_hashes, run.prompt_len, run.inst_feat, chosen, scores=scores,
                           stream=stream)
    chosen_f = torch.full((R,), -7, dtype=torch.int32, device="cuda")
    min_f = torch.zeros(R, dtype=torch.float32, device="cuda")
    run.ctx.ls_score_batch(run.req_off, run.req_hashes, run.prompt_len, run.inst_feat, chosen_f, min_ttft=min_f,
                           stream=stream)
    return chosen, scores, chosen_f, min_f


def check_fast_call(out, N):
    """The call without the score matrix decides exactly as the canonical one."""
    chosen, scores, chosen_f, min_f = (host(t) for t in out)
    np.testing.assert_array_equal(chosen_f, chosen)
    best = scores.reshape(-1, N)[np.arange(chosen.size), chosen]
    np.testing.assert_array_equal(min_f.view(np.uint32), best.view(np.uint32))


def host(t):
    return t.cpu().numpy()


def assert_close_to(got, ref, base, d, hidden, rtol, tag):
    for lname, a, b in layer_slices(d, hidden):
        dg = got[a:b].astype(np.float64) - base[a:b]
        dr = ref[a:b].astype(np.float64) - base[a:b]
        assert np.linalg.norm(dg - dr) <= rtol * np.linalg.norm(dr) + 1e-12, f"{tag}: {lname}"


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_shadow_training_and_swap(dtype):
    import torch
    w = workload(dtype)
    cfg = w.cfg
    mode = "bf16" if dtype == "bf16" else "fp32"
    F, P = 64, 32
    note(f"swap {dtype}: live scores")
    run = GpuRun(w)
    ctx = run.ctx
    serve = torch.cuda.current_stream()
    train = torch.cuda.Stream()
    out0 = score_on(run, serve)
    c0, s0 = out0[:2]
    before = (host(c0), host(s0))
    check_fast_call(out0, cfg.N)
    xa, ya = w.upd_feats[:160], w.upd_ttft[:160]
    xb, yb = w.upd_feats[160:260], w.upd_ttft[160:260]
    dev = [to_dev(np.asarray(a, np.float32)) for a in (xa, ya, xb, yb)]
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()

    ctx.ls_set_shadow_training(True, stream=train)
    ctx.ls_buffer_init(F, P)
    ob = oracle.Buffer(cfg.d, F, P)
    note(f"swap {dtype}: push and retrain the shadow on the training stream")
    ctx.ls_buffer_push(dev[0], dev[1], stream=train)
    oracle.buffer_push(mode, cfg.hidden, w.params, w.mu, w.inv_sigma, ob, xa, ya)
    n = int(ob.fifo_count[0]) + int(ob.rep_count[0])
    perm1 = np.concatenate([np.random.default_rng(e).permutation(n) for e in range(2)]).astype(np.int32)
    ctx.ls_train_round(2, 16, w.lr, perm1, loss, stream=train)
    out1 = score_on(run, serve)                   # may overlap the training
    c1, s1 = out1[:2]
    torch.cuda.synchronize()
    check_fast_call(out1, cfg.N)
    np.testing.assert_array_equal(host(c1), before[0])
    np.testing.assert_array_equal(host(s1).view(np.uint32), before[1].view(np.uint32))
    np.testing.assert_array_equal(ctx.ls_get_model()[0], w.params.astype(np.float32))

    note(f"swap {dtype}: push on the shadow, swap without a host wait")
    ctx.ls_buffer_push(dev[2], dev[3], stream=train)
    ctx.ls_swap_model(serve_stream=serve, train_stream=train)
    out2 = score_on(run, serve)
    c2, s2 = out2[:2]
    torch.cuda.synchronize()
    check_fast_call(out2, cfg.N)
    p1 = ctx.ls_get_model()[0]
    want1, _ = oracle.train_round(mode, cfg.hidden, w.params, w.mu, w.inv_sigma, ob, 2, 16, w.lr, perm1)
    assert_close_to(p1, want1, w.params, cfg.d, cfg.hidden, 1e-4, "first round")
    ref = GpuRun(w, params=p1)
    r = ref.score()
    np.testing.assert_array_equal(host(c2), r["chosen"])
    np.testing.assert_array_equal(host(s2).view(np.uint32), r["scores"].reshape(-1).view(np.uint32))
    assert not np.array_equal(host(s2), before[1])
    ref.ctx.close()
    # the second push embedded its samples with the shadow (the weights now serving)
    oracle.buffer_push(mode, cfg.hidden, p1, w.mu, w.inv_sigma, ob, xb, yb)
    assert tuple(ctx.ls_buffer_state()) == (int(ob.fifo_count[0]), int(ob.fifo_head[0]), int(ob.rep_count[0]))
    fx, fy, rx, ry = (host(t) for t in ctx.ls_buffer_read())
    wfx, wfy = ob.fifo_rows()
    wrx, wry = ob.replay_rows()
    np.testing.assert_array_equal(fx, wfx)
    np.testing.assert_array_equal(fy, wfy)
    np.testing.assert_array_equal(rx, wrx)
    np.testing.assert_array_equal(ry, wry)

    note(f"swap {dtype}: training continues from the serving model")
    n = int(ob.fifo_count[0]) + int(ob.rep_count[0])
    perm2 = np.random.default_rng(9).permutation(n).astype(np.int32)
    ctx.ls_train_round(1, 16, w.lr, perm2, loss, stream=train)
    ctx.ls_swap_model(serve_stream=serve, train_stream=train)
    torch.cuda.synchronize()
    p2 = ctx.ls_get_model()[0]
    want2, _ = oracle.train_round(mode, cfg.hidden, p1, w.mu, w.inv_sigma, ob, 1, 16, w.lr, perm2)
    assert_close_to(p2, want2, p1, cfg.d, cfg.hidden, 1e-4, "second round")

    note(f"swap {dtype}: shadow off, updates act on the live model")
    ctx.ls_set_shadow_training(False)
    got = run.update(w.upd_feats[:300], w.upd_ttft[:300])
    want = oracle.update(mode, cfg.d, cfg.hidden, p2, w.mu, w.inv_sigma, w.upd_feats[:300], w.upd_ttft[:300], w.lr)
    assert_close_to(got["params"], want["params"], p2, cfg.d, cfg.hidden, 1e-4, "live update")
    with pytest.raises(lodestar.LodestarError) as e:
        ctx.ls_swap_model()
    assert e.value.code == lodestar.LS_ERR_STATE
    torch.cuda.synchronize()
    del dev, loss
    ctx.close()


def test_set_model_writes_both_slots():
    """ls_set_model while the shadow is on: the shadow takes the new weights too,
    so a swap right after it serves them unchanged."""
    import torch
    w = workload("fp32")
    note("swap: set_model with the shadow on")
    run = GpuRun(w)
    ctx = run.ctx
    with pytest.raises(lodestar.LodestarError) as e:
        ctx.ls_swap_model()
    assert e.value.code == lodestar.LS_ERR_STATE
    ctx.ls_set_shadow_training(True)
    p = (w.params * 0.5).astype(np.float32)
    ctx.ls_set_model(p, w.mu, w.inv_sigma)
    ctx.ls_swap_model()
    torch.cuda.synchronize()
    np.testing.assert_array_equal(ctx.ls_get_model()[0], p)
    ref = GpuRun(w, params=p)
    a, b = run.score(), ref.score()
    np.testing.assert_array_equal(a["scores"].view(np.uint32), b["scores"].view(np.uint32))
    ref.ctx.close()
    ctx.close()
