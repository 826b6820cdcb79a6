"""md_init_static, the entry point that allocates nothing, against md_init.

The same workload runs once on a handle from md_init and once on a handle
from md_init_static (scratch in the library's static device array), each
checked step by step against the oracle by the harness; the two runs must
agree bit for bit in every output and every caller buffer.  Two
md_init_static handles in a row, the second on a smaller input, use the same
static array.
"""
import ctypes
import sys

import numpy as np
import pytest
import torch

from paper_2607_10582_amd import binding as B
from paper_2607_10582_amd.cache import PagedCache
from synth import configs as C

from harness import Pair

pytestmark = pytest.mark.gpu

STATE = ("page_table", "page_serial", "n_pages", "n_tokens", "importance", "t_ref", "t_ins", "region",
         "free_list", "free_count", "clock", "next_serial")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a ROCm device")
    B.load_library()


def trajectory(w, static: bool, steps: int, **kw):
    p = Pair(w, static=static, **kw)
    cfg = p.md.kernel_config()
    out = []
    for _ in range(steps):
        p.step()
        c = p.cache
        rec = {n: getattr(c, n).cpu().numpy().copy() for n in STATE}
        rec["abar"] = p.abar.cpu().numpy().copy()
        rec["token_score"] = p.tscore.cpu().numpy().copy()
        rec["page_score"] = p.md.page_score.cpu().numpy().copy()
        rec["evict_serial"] = p.md.evict_serial.cpu().numpy().copy()
        rec["evict_count"] = p.md.evict_count.cpu().numpy().copy()
        rec["infeasible"] = p.md.infeasible.cpu().numpy().copy()
        out.append(rec)
    assert p.device_status() == 0
    assert p.free_pages_consistent()
    p.close()
    return out, cfg


def same_bits(a: np.ndarray, b: np.ndarray) -> bool:
    return a.shape == b.shape and np.array_equal(a.view(np.uint8), b.view(np.uint8))


@pytest.mark.parametrize("fused", [True, False])
def test_static_handles_match_md_init_twice(fused):
    # first two sessions of eight layers (on the fused kernel: two row
    # groups, whose partial masses sit in the static scratch too), then a
    # batch of three sessions (one over the budget from the start, one
    # infeasible), then one smaller session: each md_init_static handle
    # reuses the static array the previous one left behind
    rows = C.with_overrides(C.get("small"), L=8, S=2, n0=None, n0_range=(1, 2), steps=6)
    big = C.with_overrides(C.get("small"), L=2, S=3, n0=None, n0_range=(1, 2), steps=10)
    small = C.with_overrides(C.get("small"), L=2, n0=200, steps=8)
    cases = [(rows, dict(n0s=[450, 700], budgets=[225, 300])),
             (big, dict(n0s=[450, 1200, 90], budgets=[225, 400, 50])), (small, dict())]
    for w, kw in cases:
        say(f"[no-alloc] S={w.S} steps={w.steps} fused={fused}")
        ref, cfg_ref = trajectory(w, False, w.steps, fused=fused, **kw)
        got, cfg_got = trajectory(w, True, w.steps, fused=fused, **kw)
        assert cfg_ref == cfg_got
        if w is rows and fused:
            assert cfg_got["first_row_groups"] == 2 and cfg_got["steady_row_groups"] == 2
        for k, (a, b) in enumerate(zip(ref, got)):
            for name in a:
                assert same_bits(a[name], b[name]), (k + 1, name)
        say(f"[no-alloc] S={w.S}: {len(ref)} steps identical to md_init's")


def test_static_handle_rejects_a_scratch_beyond_the_static_array():
    # the multi-kernel path keeps every slot's logits: 300,000 pages of 16
    # slots x 12 rows x 4 bytes = 230 MB > 128 MiB.  Nothing runs on the
    # device before the size is checked (no fused-kernel probe on this path).
    c = PagedCache(L=1, Hq=12, Hkv=2, d=128, P=16, S=1, max_pages=8, n_phys=8, device="cuda")
    b = torch.ones((1, 7), dtype=torch.float32, device="cuda")
    lam = torch.zeros((1, 7), dtype=torch.float32, device="cuda")
    cfg = B.md_config(n_layers=1, n_q_heads=12, n_kv_heads=2, head_dim=128, page_size=16, max_sessions=1,
                      max_pages=8, n_phys_pages=300000, n_regions=7, pinned_region_mask=1, rho=0.9,
                      alpha=1.0, tau_scale=2.0, flags=B.MD_FLAG_NO_FUSED, window=1)
    rp = B.md_region_params(base_priority=b.data_ptr(), decay_rate=lam.data_ptr())
    st, h = B.md_init_raw(cfg, rp, c.view(), torch.cuda.current_stream().cuda_stream, static=True)
    assert st == B.MD_E_TOO_LARGE and h is None
    assert "static" in B.md_status_str(st)
    # the same configuration within the array's size initialises
    cfg.n_phys_pages = 8
    st, h = B.md_init_raw(cfg, rp, c.view(), torch.cuda.current_stream().cuda_stream, static=True)
    assert st == B.MD_OK and h is not None
    B.md_destroy(h)
