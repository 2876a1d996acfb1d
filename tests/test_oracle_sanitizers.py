"""The oracle built with AddressSanitizer and UndefinedBehaviorSanitizer (CPU
only): every pin, and whole workloads through scoring, routing, the update, the
data path and index maintenance, in a child process that preloads both
runtimes; any finding aborts it."""
import os
import subprocess
import sys
import textwrap

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = textwrap.dedent("""
    import sys
    sys.path[:0] = [{root!r}, {tests!r}]
    import numpy as np
    import oracle
    oracle.use_library({lib!r})
    import oracle_pins
    for pin in oracle_pins.ALL_PINS:
        pin()
    from paper_2606_00946_amd import synth
    for name, R in (("tiny", None), ("homogeneous", 512), ("large_batch", 64)):
        w = synth.generate(name, R=R)
        c = w.cfg
        mode = "bf16" if c.dtype == "bf16" else "fp32"
        args = (c.d, c.hidden, w.params, w.mu, w.inv_sigma, w.req_off, w.req_hashes, w.prompt_len, w.inst_feat,
                w.inst_off, w.inst_hashes)
        res = oracle.score(mode, *args, threads=4)
        pol = oracle.policy(heuristic=1, count_cols=(0, 1), theta_imbal=4.0, overload_k=0.5, n_samples=10,
                            n_min=1, epsilon=0.2, kv_col=4, tau_sat=0.0, tau_ben=0.0, k_filter=2, delta=0.05)
        rnd = np.random.default_rng(1).integers(0, 1 << 32, (c.R, 3), dtype=np.uint64).astype(np.uint32)
        oracle.route(mode, *args, pol, rnd, sel=np.arange(c.R, dtype=np.int32))
        B = min(300, w.upd_feats.shape[0])
        oracle.update(mode, c.d, c.hidden, w.params, w.mu, w.inv_sigma, w.upd_feats[:B], w.upd_ttft[:B], w.lr,
                      dropout=(0.1, 7, 0))
        buf = oracle.Buffer(c.d, 40, 16)
        oracle.buffer_push(mode, c.hidden, w.params, w.mu, w.inv_sigma, buf, w.upd_feats[:B], w.upd_ttft[:B])
    print("SANITIZED OK", flush=True)
""")


def _runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.slow
def test_oracle_under_asan_and_ubsan(tmp_path):
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not asan or not ubsan:
        pytest.skip("gcc has no sanitizer runtimes here")
    lib = str(tmp_path / "liblsoracle_san.so")
    oracle.compile_c(os.path.join(ROOT, "oracle", "lodestar_oracle.c"), lib, extra=oracle.SANITIZE_FLAGS)
    env = dict(os.environ, LD_PRELOAD=f"{asan}:{ubsan}", ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="4")
    code = CHILD.format(root=ROOT, tests=os.path.join(ROOT, "tests"), lib=lib)
    proc = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=600)
    assert proc.returncode == 0 and "SANITIZED OK" in proc.stdout, (proc.stdout[-2000:], proc.stderr[-4000:])
