"""Parity at the full sizes of the benchmark workloads: every session's whole
trajectory, step by step, through the C ABI against the oracle.

The oracle sessions run in worker processes (oracle.pool), one BLAS thread
each, so that a step of all sessions takes about as long as one session.
Inputs of the two largest workloads are drawn on the device (torch's
counter-based generator) and copied to the host for the oracle.  Tolerances
as in tests/harness.py.
"""
import os
import sys
import time

import numpy as np
import pytest
import torch

from oracle.pool import host_cores
from synth import configs as C
from synth import generator as g

from harness import Pair

pytestmark = pytest.mark.gpu
WORKERS = min(16, host_cores())


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a ROCm device")
    from paper_2607_10582_amd import binding
    binding.load_library()


def run_full(p: Pair, steps: int, label: str):
    t0 = time.time()
    say(f"[{label}] S={p.w.S} L={p.w.L} Hq={p.w.Hq} P={p.w.P} steps={steps}, oracle sessions "
        f"{len(p.oracle_sessions)} on {WORKERS} workers")
    for k in range(steps):
        st = p.step()
        if k == 0 or (k + 1) % 16 == 0:
            say(f"[{label}] step {k + 1}: {st.tokens} token-steps compared, evicted pages {st.evicted_pages}, "
                f"max rel {max(st.max_rel.values()):.2e}, {time.time() - t0:.0f} s")
    status = p.device_status()
    assert status == 0, f"device status {status:#x}"
    assert p.free_pages_consistent()
    say(f"[{label}] ok: {st.steps} steps, {st.tokens} token-steps, max rel {st.max_rel}, "
        f"tau-excused {st.tau_excused}, tie-excused {st.tie_excused}, evicted pages {st.evicted_pages}")
    p.close()
    return st


def test_qwen3_batch_all_sessions_all_steps():
    # 32 sessions x 1,700 tokens (3B shape), all 256 decode steps
    w = C.get("qwen3_32x1700")
    st = run_full(Pair(w, pool=WORKERS, fused=None), w.steps, "qwen3_32x1700-full")
    assert st.evicted_pages > 32 * 60


def test_long32k_all_sessions_all_steps():
    # 16 sessions x 32,768 tokens (1.5B shape), all 128 steps, as the
    # benchmark runs them (fused kernel, selection and compaction in one
    # call): the bulk eviction at step 1, page openings every 16 steps, and
    # the late steady state.  The one call applies the device's selection
    # at once, so it must equal the oracle's at every step (no tie band is
    # met on this trajectory).
    w = C.get("long32k")
    p = Pair(w, backend="torch", pool=WORKERS, fused=None, select_compact=True)
    cfg = p.md.kernel_config()
    assert cfg["first_fused"] and cfg["steady_fused"] and not cfg["spill"]
    st = run_full(p, w.steps, "long32k-full")
    assert st.evicted_pages > 16 * (32768 - 8192) // 16


@pytest.mark.parametrize("name", ["ragged_p16", "ragged_p64"])
def test_ragged_batch_all_sessions_all_steps(name):
    # 64 sessions of U[2,048, 65,536] tokens (3B shape), all 64 steps, on the
    # fused kernel; sessions below 5,120 tokens have more pinned tokens than
    # budget (the infeasible path).  Pages of 16 as the benchmark runs them
    # (selection and compaction in one call), pages of 64 with the two calls.
    w = C.get(name)
    p = Pair(w, backend="torch", pool=WORKERS, fused=None, select_compact=name == "ragged_p16")
    cfg = p.md.kernel_config()
    assert cfg["first_fused"] and cfg["steady_fused"]
    st = run_full(p, w.steps, f"{name}-full")
    assert p.warned
