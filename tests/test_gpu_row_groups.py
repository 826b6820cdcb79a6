"""Row groups of the fused observation kernel, through the C ABI on the
device.

When a step's units would fill less than half of the fused grid, each unit
covers one range of the (layer, KV head) rows and the groups' partial masses
(sums over disjoint rows of the mean of Sec. III-C) meet in the unit of the
first group, which finishes the tokens (EWMA, refresh, Eq. 4, Eq. 5).
Checked here: parity with the oracle on even and uneven splits, agreement
with units that walk every row, the library's choice of the split, and void
steps when the non-finite query row belongs to any group.
"""
import sys

import numpy as np
import pytest
import torch

from paper_2607_10582_amd import binding as B
from synth import configs as C

from harness import Pair, REL

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a ROCm device")
    B.load_library()


def run_pair(p: Pair, steps: int, label: str):
    say(f"[{label}] S={p.w.S} L={p.w.L} Hq={p.w.Hq} Hkv={p.w.Hkv} P={p.w.P} steps={steps} "
        f"config {p.md.kernel_config()}")
    for _ in range(steps):
        st = p.step()
    status = p.device_status()
    assert status == 0, f"device status {status:#x}"
    assert p.free_pages_consistent()
    say(f"[{label}] ok: {st.steps} steps, {st.tokens} token-steps, max rel {st.max_rel}, "
        f"tau-excused {st.tau_excused}, tie-excused {st.tie_excused}, evicted pages {st.evicted_pages}")
    p.close()
    return st


def test_library_splits_rows_for_a_small_batch():
    # 32 sessions of 1,700 tokens (3B shape, 72 rows): 224 units at the first
    # observation and 64 later, against 512 workgroups; the library picks the
    # fused kernel with two row groups for the first and eight (of nine rows)
    # for the later ones.  With 8 sessions (16 units, 144 with nine groups)
    # row groups still fill a quarter of the grid and take both; with 4 (8
    # units, 72) the later observes take the multi-kernel path.
    w = C.with_overrides(C.get("qwen3_32x1700"), steps=16)
    p = Pair(w, fused=None, select_compact=True, oracle_sessions=[0, 13, 31])
    cfg = p.md.kernel_config()
    assert cfg["first_fused"] and cfg["steady_fused"]
    assert cfg["first_row_groups"] == 2 and cfg["steady_row_groups"] == 8
    st = run_pair(p, 16, "rows-auto-qwen3-32")
    assert st.evicted_pages > 3 * 60
    p8 = Pair(C.with_overrides(w, S=8), fused=None, oracle_sessions=[0, 7])
    cfg8 = p8.md.kernel_config()
    assert cfg8["first_fused"] and cfg8["first_row_groups"] == 9
    assert cfg8["steady_fused"] and cfg8["steady_row_groups"] == 9
    run_pair(p8, 16, "rows-auto-qwen3-8")
    p4 = Pair(C.with_overrides(w, S=4), fused=None, oracle_sessions=[])
    cfg4 = p4.md.kernel_config()
    assert cfg4["first_fused"] and not cfg4["steady_fused"]
    p4.close()


@pytest.mark.parametrize("L,Hq,Hkv,groups", [(13, 16, 2, 3), (8, 16, 2, 2), (28, 8, 1, 3), (36, 16, 2, 9)])
def test_row_groups_even_and_uneven_splits(L, Hq, Hkv, groups):
    # L * Hkv rows in `groups` ranges of floor / ceil (L * Hkv / groups) rows:
    # 26 rows as 8, 9, 9; 16 as 8, 8; 28 as 9, 9, 10; 72 as nine of 8
    w = C.with_overrides(C.get("qwen3_32x1700"), L=L, Hq=Hq, Hkv=Hkv, S=4, steps=12)
    p = Pair(w, fused=True)
    cfg = p.md.kernel_config()
    assert cfg["first_row_groups"] == groups and cfg["steady_row_groups"] == groups
    run_pair(p, 12, f"rows-L{L}-Hkv{Hkv}-g{groups}")


def test_row_groups_agree_with_units_on_every_row():
    # The same steps with and without row groups: attention masses and page
    # scores agree to rounding (the groups add their partial sums in another
    # order); the budget holds every token so that the slots line up.
    w = C.with_overrides(C.get("qwen3_32x1700"), S=6, steps=3, budget_frac=1.0)
    outs = []
    for rows in (True, False):
        p = Pair(w, oracle_sessions=[], fused=True, row_groups=rows)
        assert (p.md.kernel_config()["steady_row_groups"] > 1) == rows
        res = []
        for _ in range(3):
            p.step(compare=False)
            res.append((p.abar.cpu().numpy().copy(), p.md.page_score.cpu().numpy().copy()))
        assert p.device_status() == 0
        outs.append(res)
        p.close()
    for (a1, s1), (a2, s2) in zip(*outs):
        np.testing.assert_allclose(a1, a2, rtol=REL, atol=1e-30)
        fin = np.isfinite(s1)
        assert np.array_equal(fin, np.isfinite(s2))
        np.testing.assert_allclose(s1[fin], s2[fin], rtol=REL, atol=1e-30)


@pytest.mark.parametrize("layer", [0, 5, 7])
def test_nonfinite_query_voids_the_session_in_any_group(layer):
    # 8 layers x 2 KV heads = 16 rows in two groups (layers 0-3 and 4-7): a
    # NaN in session 0's query at the given layer voids session 0's step
    # whichever group reads it; session 1 evicts as usual.
    w = C.with_overrides(C.get("small"), L=8, S=2, n0=None, n0_range=(1, 2), steps=4)
    p = Pair(w, n0s=[450, 450], budgets=[225, 225], oracle_sessions=[], fused=True)
    assert p.md.kernel_config()["first_row_groups"] == 2
    c = p.cache
    np0, ptab0 = int(c.n_pages[0]), c.page_table[0].clone()
    slots0 = (c.page_table[0, :np0].long().view(-1, 1) * 16 +
              torch.arange(16, device=c.page_table.device).view(1, -1)).view(-1)[:450]
    imp0 = c.importance.view(-1)[slots0].clone()
    q, nk, reg, *_ = p.inputs(1)
    q[0, 0, layer, 3, 17] = float("nan")      # [S][W][L][Hq][d]
    p.md.observe(1, q, nk, reg)
    p.md.score()
    p.md.select_compact()
    torch.cuda.synchronize()
    assert p.md.device_status() == B.MD_DEV_NONFINITE
    cnt = p.md.evict_count.cpu().tolist()
    assert cnt[0] == 0 and cnt[1] > 0
    assert int(c.n_pages[0]) == np0 and torch.equal(c.page_table[0], ptab0)
    assert torch.equal(c.importance.view(-1)[slots0].view(torch.int32), imp0.view(torch.int32))
    q, nk, reg, *_ = p.inputs(2)
    p.md.observe(2, q, nk, reg)
    p.md.score()
    p.md.select_compact()
    torch.cuda.synchronize()
    assert p.md.device_status() == 0
    assert p.md.evict_count.cpu().tolist()[0] > 0
    p.close()


def test_row_groups_cooperative_launch():
    # the row-group instantiation as a cooperative launch
    w = C.with_overrides(C.get("qwen3_32x1700"), S=6, steps=10)
    p = Pair(w, fused=True, cooperative=True, oracle_sessions=[0, 5])
    assert p.md.kernel_config()["steady_row_groups"] > 1
    run_pair(p, 10, "rows-cooperative")


@pytest.mark.parametrize("P", [16, 64])
def test_row_groups_on_empty_and_short_sessions(P):
    # empty, single-token, exact-page, page+1, partial-tail and longer
    # sessions in one batch with row groups (16 layers x 2 KV heads = 32
    # rows in four groups); budgets below, at and above the pinned span
    w = C.with_overrides(C.get("small"), L=16, Hq=8, Hkv=2, S=7, n0=None, P=P,
                         n0_range=(1, 2), steps=24, system_len=20)
    n0s = [0, 1, 15, 16, 17, 130, 700]
    budgets = [0, 0, 5, 16, 10, 100, 200]
    p = Pair(w, n0s=n0s, budgets=budgets, fused=True)
    cfg = p.md.kernel_config()
    assert cfg["first_row_groups"] == 4 and cfg["steady_row_groups"] == 4
    run_pair(p, 24, f"rows-edges-P{P}")


def test_row_groups_with_the_offload_tier():
    # The offload tier observes its host-memory pages with the rows'
    # normalisers of the step, which the leaders of every row group publish:
    # three sessions of eight layers (16 rows, two groups), keys planted so
    # that pages leave for host memory and come back; every step compared
    # with the oracle, host-memory state included.
    from test_gpu_parity import run_offload
    w = C.with_overrides(C.get("small"), L=8, S=3, n0=None, n0_range=(1, 2), steps=40, system_len=60)
    p = Pair(w, n0s=[450, 700, 300], budgets=[225, 300, 200], planted=24, planted_strength=2.5, query_gain=0.7,
             fused=True, offload_pages=8, drop_threshold=1e-3)
    cfg = p.md.kernel_config()
    assert cfg["first_row_groups"] == 2 and cfg["steady_row_groups"] == 2
    st = run_offload(p, 40, "rows-offload")
    assert st.offloaded > 20 and st.recalled > 10
