"""Per-kernel timing through the C ABI (ls_profile_enable, ls_profile_read).

While timing is on, each launch group of a call is bracketed by HIP events on
the call's stream. Timing must change no result, and it must report launches
and a positive device time for every group that ran: the table build, the
index load under capacities, K1, the instance partials, the scorer, the band
and its rescoring, K3 and the update."""
import numpy as np
import pytest

from gpu_helpers import GpuRun, note, to_dev
from paper_2606_00946_amd import lodestar, synth

pytestmark = pytest.mark.gpu


def _bits(a):
    a = np.asarray(a)
    return a.view(np.uint32) if a.dtype in (np.float32, np.int32) else a


@pytest.mark.parametrize("name,R", [("homogeneous", 512), ("large_batch", 1024)])
def test_profiling_changes_nothing_and_times_every_group(name, R):
    w = synth.generate(name, R=R)
    note(f"profiling {name} R={R}")
    runs = []
    for profile in (False, True):
        run = GpuRun(w, profile=profile)
        sc = run.score(with_scores=False)
        up = run.update()
        prof = run.ctx.ls_profile_read() if profile else None
        runs.append((sc, up, prof))
        run.ctx.close()
    (s0, u0, _), (s1, u1, prof) = runs
    for k in ("chosen", "min_ttft", "overlap", "feat"):
        assert np.array_equal(_bits(s0[k]), _bits(s1[k])), k
    assert np.float32(u0["loss"]).view(np.uint32) == np.float32(u1["loss"]).view(np.uint32)
    assert np.array_equal(u0["params"].view(np.uint32), u1["params"].view(np.uint32))
    want = ["table_build", "prefix_match", "instance_partial", "argmin", "update"]
    want += ["score_pairs_mfma", "band_select", "rescore"] if w.cfg.dtype == "bf16" else ["score_pairs"]
    for kind in want:
        assert kind in prof, (kind, sorted(prof))
        launches, ms = prof[kind]
        assert launches >= 1 and 0.0 < ms < 1e3, (kind, launches, ms)


def test_profiling_times_the_index_load():
    """Capacities make the load rebuild the instance lists (the index group)."""
    w = synth.generate("homogeneous", R=64)
    ctx = lodestar.Context(w.cfg.d, w.cfg.hidden, w.cfg.dtype)
    ctx.ls_profile_enable(True)
    ctx.ls_set_model(w.params, w.mu, w.inv_sigma)
    ctx.ls_set_cache_capacity(np.diff(w.inst_off))
    ctx.ls_load_cache_state(w.inst_off, to_dev(w.inst_hashes))
    prof = ctx.ls_profile_read()
    ctx.ls_profile_enable(False)
    ctx.close()
    for kind in ("table_build", "index"):
        assert kind in prof, (kind, sorted(prof))
        launches, ms = prof[kind]
        assert launches >= 1 and 0.0 < ms < 1e3, (kind, launches, ms)
