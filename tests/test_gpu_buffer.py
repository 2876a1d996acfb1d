"""Online-learning data path through the C ABI against the oracle: the FIFO and
the gradient-coreset replay pool hold exactly the oracle's rows after every
push, and a retraining round gives the oracle's weights."""
import numpy as np
import pytest

import oracle
from gpu_helpers import layer_slices, note, rel_ok, to_dev
from paper_2606_00946_amd import lodestar, synth

pytestmark = pytest.mark.gpu


def _stream(w, n):
    x = w.upd_feats[:n].copy(); y = w.upd_ttft[:n].copy()
    for k in range(5, n, 5):                  # exact duplicates: ties in the coreset rule
        x[k] = x[k // 2]; y[k] = y[k // 2]
    return x, y


def _ctx(w):
    ctx = lodestar.Context(w.cfg.d, w.cfg.hidden, w.cfg.dtype)
    ctx.ls_set_model(w.params, w.mu, w.inv_sigma)
    return ctx


@pytest.mark.parametrize("name,F,P,n", [("tiny", 12, 6, 120), ("homogeneous", 64, 48, 400),
                                        ("large_batch", 200, 150, 700)])
def test_buffer_matches_oracle(name, F, P, n):
    import torch
    w = synth.generate(name)
    cfg = w.cfg
    mode = "bf16" if cfg.dtype == "bf16" else "fp32"
    x, y = _stream(w, n)
    ctx = _ctx(w)
    ctx.ls_buffer_init(F, P)
    ob = oracle.Buffer(cfg.d, F, P)
    rng = np.random.default_rng(3)
    s = 0
    pushes = 0
    while s < n:
        k = int(rng.integers(1, max(2, F // 2)))
        xs, ys = x[s:s + k], y[s:s + k]
        note(f"buffer {name} push {pushes} rows {s}..{s + len(ys)}")
        adm = torch.zeros(1, dtype=torch.int32, device="cuda")
        ctx.ls_buffer_push(to_dev(xs), to_dev(ys), adm)
        want_adm = oracle.buffer_push(mode, cfg.hidden, w.params, w.mu, w.inv_sigma, ob, xs, ys)
        torch.cuda.synchronize()
        fc, fh, rc = ctx.ls_buffer_state()
        assert (fc, fh, rc) == (int(ob.fifo_count[0]), int(ob.fifo_head[0]), int(ob.rep_count[0]))
        fx, fy, rx, ry = (t.cpu().numpy() for t in ctx.ls_buffer_read())
        wfx, wfy = ob.fifo_rows(); wrx, wry = ob.replay_rows()
        np.testing.assert_array_equal(fx, wfx); np.testing.assert_array_equal(fy, wfy)
        np.testing.assert_array_equal(rx, wrx); np.testing.assert_array_equal(ry, wry)
        assert int(adm.item()) == want_adm
        s += len(ys); pushes += 1
    print(f"{name}: {pushes} pushes, pool {rc}/{P}", flush=True)
    # a retraining round over both pools, in a permuted order
    nall = int(ob.fifo_count[0]) + int(ob.rep_count[0])
    perm = np.concatenate([np.random.default_rng(e).permutation(nall) for e in range(2)]).astype(np.int32)
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    note(f"train round {name} n={nall}")
    ctx.ls_train_round(2, 32, w.lr, perm, loss)
    got = ctx.ls_get_model()[0]
    want, want_loss = oracle.train_round(mode, cfg.hidden, w.params, w.mu, w.inv_sigma, ob, 2, 32, w.lr, perm)
    assert abs(loss.item() - want_loss) <= 1e-5 * abs(want_loss), (loss.item(), want_loss)
    for lname, a, b in layer_slices(cfg.d, cfg.hidden):
        dg = got[a:b].astype(np.float64) - w.params[a:b]
        dw = want[a:b].astype(np.float64) - w.params[a:b]
        assert np.linalg.norm(dg - dw) <= 1e-4 * np.linalg.norm(dw) + 1e-12, lname
    ctx.close()


@pytest.mark.parametrize("name,F,P,first,second", [("homogeneous", 64, 300, 1200, 700), ("large_batch", 40, 520, 900, 900),
                                                   ("large_batch", 16, 6200, 6300, 600)])
def test_buffer_large_pushes(name, F, P, first, second):
    """Pushes whose FIFO evictions exceed one admission chunk (256 candidates):
    the pool fills and starts replacing members within one push, and later
    chunks see slots taken by earlier ones; a pool of 6,200 slots is above what
    the per-slot state in LDS holds (6,144), so its decisions keep that state in
    global memory.  Pool and FIFO exactly the oracle's."""
    import torch
    w = synth.generate(name)
    cfg = w.cfg
    mode = "bf16" if cfg.dtype == "bf16" else "fp32"
    x, y = _stream(w, first + second)
    ctx = _ctx(w)
    ctx.ls_buffer_init(F, P)
    ob = oracle.Buffer(cfg.d, F, P)
    for a, b in ((0, first), (first, first + second)):
        note(f"buffer {name} large push rows {a}..{b}")
        adm = torch.zeros(1, dtype=torch.int32, device="cuda")
        ctx.ls_buffer_push(to_dev(x[a:b]), to_dev(y[a:b]), adm)
        want_adm = oracle.buffer_push(mode, cfg.hidden, w.params, w.mu, w.inv_sigma, ob, x[a:b], y[a:b])
        torch.cuda.synchronize()
        assert tuple(ctx.ls_buffer_state()) == (int(ob.fifo_count[0]), int(ob.fifo_head[0]), int(ob.rep_count[0]))
        fx, fy, rx, ry = (t.cpu().numpy() for t in ctx.ls_buffer_read())
        wfx, wfy = ob.fifo_rows()
        wrx, wry = ob.replay_rows()
        np.testing.assert_array_equal(fx, wfx)
        np.testing.assert_array_equal(fy, wfy)
        np.testing.assert_array_equal(rx, wrx)
        np.testing.assert_array_equal(ry, wry)
        assert int(adm.item()) == want_adm
        print(f"{name}: push of {b - a}, admitted {want_adm}, pool {int(ob.rep_count[0])}/{P}", flush=True)
    ctx.close()


def test_buffer_errors():
    import torch
    w = synth.generate("tiny")
    ctx = _ctx(w)
    x = to_dev(w.upd_feats[:4]); y = to_dev(w.upd_ttft[:4])
    with pytest.raises(lodestar.LodestarError) as e:
        ctx.ls_buffer_push(x, y)
    assert e.value.code == lodestar.LS_ERR_STATE
    with pytest.raises(lodestar.LodestarError) as e:
        ctx.ls_buffer_init(0, 4)
    assert e.value.code == lodestar.LS_ERR_INVALID
    ctx.ls_buffer_init(8, 4)
    with pytest.raises(lodestar.LodestarError) as e:
        ctx.ls_train_round(1, 4, 0.01)
    assert e.value.code == lodestar.LS_ERR_STATE
    ctx.ls_buffer_push(x, y)
    with pytest.raises(lodestar.LodestarError) as e:
        ctx.ls_train_round(1, 4, 0.01, perm=np.array([0, 0, 1, 2], np.int32))
    assert e.value.code == lodestar.LS_ERR_INVALID
    torch.cuda.synchronize()
    ctx.close()
