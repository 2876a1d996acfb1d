"""ls_score_batch_noalloc, the scoring entry point that allocates nothing (its
scratch is one array per GPU inside the library), against ls_score_batch on the
same context: two calls in a row, the second with a smaller batch, every output
bitwise equal; and the host-side rejection of a batch larger than the array."""
import numpy as np
import pytest

from gpu_helpers import note, to_dev
from paper_2606_00946_amd import lodestar, synth

pytestmark = pytest.mark.gpu


def _outputs(ctx, fn, R, N, d, inputs, with_scores):
    import torch
    out = {
        "chosen": torch.full((R,), -7, dtype=torch.int32, device="cuda"),
        "min_ttft": torch.full((R,), -7.0, dtype=torch.float32, device="cuda"),
        "scores": torch.full((R * N,), -7.0, dtype=torch.float32, device="cuda") if with_scores else None,
        "overlap": torch.full((R * N,), -7, dtype=torch.int32, device="cuda"),
        "feat": torch.full((R * d,), -7.0, dtype=torch.float32, device="cuda"),
    }
    getattr(ctx, fn)(*inputs, out["chosen"], out["min_ttft"], out["scores"], out["overlap"], out["feat"])
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items() if v is not None}


def _inputs(w, R):
    """The first R requests of the workload, as device arrays."""
    off = w.req_off[:R + 1]
    return (to_dev(off), to_dev(w.req_hashes[:off[-1]]), to_dev(w.prompt_len[:R].astype(np.int32)),
            to_dev(w.inst_feat.astype(np.float32)))


@pytest.mark.parametrize("name,R1,R2", [("large_batch", 4096, 1000), ("homogeneous", 4096, 77)])
def test_noalloc_matches_score_batch(name, R1, R2):
    w = synth.generate(name, R=R1)
    cfg = w.cfg
    ctx = lodestar.Context(cfg.d, cfg.hidden, cfg.dtype)
    ctx.ls_set_model(w.params, w.mu, w.inv_sigma)
    inst_h = to_dev(w.inst_hashes)
    ctx.ls_load_cache_state(w.inst_off, inst_h)
    for with_scores in (False, True):
        for R in (R1, R2):               # the second call is smaller: stale scratch must not leak into it
            note(f"no-alloc scoring {name} R={R} N={cfg.N} scores={with_scores}")
            inputs = _inputs(w, R)
            a = _outputs(ctx, "ls_score_batch_noalloc", R, cfg.N, cfg.d, inputs, with_scores)
            b = _outputs(ctx, "ls_score_batch", R, cfg.N, cfg.d, inputs, with_scores)
            for k in a:
                np.testing.assert_array_equal(a[k].view(np.uint8), b[k].view(np.uint8), err_msg=k)
            assert np.all((a["chosen"] >= 0) & (a["chosen"] < cfg.N))
    ctx.close()


def test_noalloc_rejects_a_batch_beyond_its_scratch():
    """The full Large batch needs far more scratch than the array holds: the call
    fails on the host with LS_ERR_INVALID and enqueues nothing; the context then
    still scores a batch that fits."""
    import torch
    w = synth.generate("large_batch")
    cfg = w.cfg
    ctx = lodestar.Context(cfg.d, cfg.hidden, cfg.dtype)
    ctx.ls_set_model(w.params, w.mu, w.inv_sigma)
    ctx.ls_load_cache_state(w.inst_off, to_dev(w.inst_hashes))
    note("no-alloc scoring: oversized batch rejected on the host")
    inputs = _inputs(w, cfg.R)
    chosen = torch.full((cfg.R,), -7, dtype=torch.int32, device="cuda")
    with pytest.raises(lodestar.LodestarError) as e:
        ctx.ls_score_batch_noalloc(*inputs, chosen)
    assert e.value.code == lodestar.LS_ERR_INVALID and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert np.all(chosen.cpu().numpy() == -7)
    note("no-alloc scoring: a batch that fits after the rejection")
    small = _inputs(w, 512)
    a = _outputs(ctx, "ls_score_batch_noalloc", 512, cfg.N, cfg.d, small, False)
    b = _outputs(ctx, "ls_score_batch", 512, cfg.N, cfg.d, small, False)
    for k in a:
        np.testing.assert_array_equal(a[k].view(np.uint8), b[k].view(np.uint8), err_msg=k)
    ctx.close()
