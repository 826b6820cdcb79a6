"""C-ABI behaviour on the device: call order, step numbering, device status
bits (capacity, non-finite queries), and re-binding a saved cache."""
import numpy as np
import pytest
import torch

from paper_2607_10582_amd import binding as B
from synth import configs as C

from harness import Pair

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a ROCm device")
    B.load_library()


def small_pair(**kw):
    return Pair(C.with_overrides(C.get("small"), steps=8), **kw)


def test_call_order_and_step_numbering():
    p = small_pair(oracle_sessions=[])
    md = p.md
    q, nk, reg, *_ = p.inputs(1)
    with pytest.raises(B.MemDecayError) as e:
        md.score()
    assert e.value.status == B.MD_E_STATE
    with pytest.raises(B.MemDecayError) as e:
        md.select()
    assert e.value.status == B.MD_E_STATE
    md.observe(5, q, nk, reg)
    with pytest.raises(B.MemDecayError) as e:
        md.observe(7, q, nk, reg)                 # must be 6
    assert e.value.status == B.MD_E_STEP
    with pytest.raises(B.MemDecayError) as e:
        md.select()                               # needs a score first
    assert e.value.status == B.MD_E_STATE
    md.score()
    md.select()
    md.select()                                   # idempotent
    md.compact()
    with pytest.raises(B.MemDecayError) as e:
        md.select()
    assert e.value.status == B.MD_E_STATE
    md.observe(6, q, nk, reg)
    torch.cuda.synchronize()
    assert md.device_status() == 0
    p.close()


def test_free_list_exhaustion_sets_capacity():
    # 448 prompt tokens fill 28 pages exactly, so the first append needs a
    # page from the (empty) free list: nothing is appended, the bit is set.
    p = small_pair(oracle_sessions=[], n0s=[448], budgets=[448])
    c = p.cache
    c.free_count.zero_()
    for k in range(1, 3):
        q, nk, reg, *_ = p.inputs(k)
        p.md.observe(k, q, nk, reg)
        p.md.score()
    torch.cuda.synchronize()
    assert int(c.n_tokens[0].item()) == 448 and int(c.n_pages[0].item()) == 28
    assert p.md.device_status() == B.MD_DEV_CAPACITY
    assert int(c.free_count.item()) == 0
    assert int(c.clock[0].item()) == 448 + 2
    p.close()


def test_nonfinite_query_sets_status():
    p = small_pair(oracle_sessions=[])
    q, nk, reg, *_ = p.inputs(1)
    q[0, 0, 0, 3, 17] = float("nan")      # [S][W][L][Hq][d]
    p.md.observe(1, q, nk, reg)
    torch.cuda.synchronize()
    assert p.md.device_status() & B.MD_DEV_NONFINITE
    assert p.md.device_status() == 0              # reading clears the word
    p.close()


@pytest.mark.parametrize("one_call", [False, True])
@pytest.mark.parametrize("fused", [True, False])
def test_nonfinite_query_voids_the_sessions_step(fused, one_call):
    # Two sessions of 450 tokens with a budget of 225: the first observation
    # would evict about half of each.  Session 0's query holds a NaN: its step
    # is void (nothing selected, compacted or quantised; importance and
    # refresh clocks as before; the append stands), while session 1 evicts as
    # usual.  The next step, with a finite query, evicts session 0 too.
    w = C.with_overrides(C.get("small"), S=2, n0=None, n0_range=(1, 2), steps=8)
    p = Pair(w, n0s=[450, 450], budgets=[225, 225], oracle_sessions=[], fused=fused)
    c = p.cache
    slots0 = (c.page_table[0, :int(c.n_pages[0])].long().view(-1, 1) * 16 +
              torch.arange(16, device=c.page_table.device).view(1, -1)).view(-1)[:450]
    imp0, tref0 = c.importance.view(-1)[slots0].clone(), c.t_ref.view(-1)[slots0].clone()
    np0, ptab0 = int(c.n_pages[0]), c.page_table[0].clone()
    q, nk, reg, *_ = p.inputs(1)
    q[0, 0, 0, 3, 17] = float("nan")
    p.md.observe(1, q, nk, reg)
    p.md.score()
    if one_call:
        p.md.select_compact()
    else:
        p.md.select()
        p.md.compact()
    torch.cuda.synchronize()
    assert p.md.device_status() == B.MD_DEV_NONFINITE
    cnt = p.md.evict_count.cpu().tolist()
    assert cnt[0] == 0 and cnt[1] > 0
    assert int(c.n_pages[0]) == np0 and torch.equal(c.page_table[0], ptab0)
    assert int(c.n_tokens[0]) == 451                      # the append stands
    assert torch.equal(c.importance.view(-1)[slots0].view(torch.int32), imp0.view(torch.int32))
    assert torch.equal(c.t_ref.view(-1)[slots0], tref0)
    assert int(c.n_tokens[1]) <= 225
    q, nk, reg, *_ = p.inputs(2)
    p.md.observe(2, q, nk, reg)
    p.md.score()
    if one_call:
        p.md.select_compact()
    else:
        p.md.select()
        p.md.compact()
    torch.cuda.synchronize()
    assert p.md.device_status() == 0
    assert p.md.evict_count.cpu().tolist()[0] > 0 and int(c.n_tokens[0]) <= 225
    p.close()


def test_select_compact_order_of_calls():
    # md_select_compact needs md_score_pages since the observation, and
    # applies the selection: md_compact without lists then has nothing to
    # apply.  Its launch is timed under its own kernel id.
    p = small_pair(oracle_sessions=[], n0s=[450], budgets=[225])
    md = p.md
    md.profile(("evict",))
    q, nk, reg, *_ = p.inputs(1)
    md.observe(1, q, nk, reg)
    with pytest.raises(B.MemDecayError) as e:
        md.select_compact()
    assert e.value.status == B.MD_E_STATE
    md.score()
    md.select_compact()
    with pytest.raises(B.MemDecayError) as e:
        md.compact()
    assert e.value.status == B.MD_E_STATE
    with pytest.raises(B.MemDecayError) as e:
        md.select_compact()
    assert e.value.status == B.MD_E_STATE
    torch.cuda.synchronize()
    cnt = int(md.evict_count[0])
    assert cnt > 0 and 225 - 16 < int(p.cache.n_tokens[0]) <= 225
    assert int(p.cache.n_pages[0]) == 29 - cnt           # 451 tokens in 29 pages before
    ms, launches = md.profile_read("evict")
    assert launches == 1 and ms > 0
    assert md.device_status() == 0
    p.close()


def test_compact_applies_this_steps_selection():
    # md_compact with NULL lists applies the lists of this step's
    # md_select_evict; without a selection since the observation it is out
    # of order, and one list without the other is invalid.
    p = small_pair(oracle_sessions=[], n0s=[450], budgets=[225])
    md = p.md
    q, nk, reg, *_ = p.inputs(1)
    md.observe(1, q, nk, reg)
    md.score()
    with pytest.raises(B.MemDecayError) as e:
        md.compact()
    assert e.value.status == B.MD_E_STATE
    with pytest.raises(B.MemDecayError) as e:
        B.md_compact(md.handle, md.evict_serial.data_ptr(), None)
    assert e.value.status == B.MD_E_INVALID
    md.select()
    md.compact()
    torch.cuda.synchronize()
    n_after = int(p.cache.n_tokens[0])
    cnt = int(md.evict_count[0])
    assert cnt > 0 and 225 - 16 < n_after <= 225
    q, nk, reg, *_ = p.inputs(2)
    md.observe(2, q, nk, reg)
    md.score()
    md.select()
    with pytest.raises(B.MemDecayError) as e:
        B.md_compact(md.handle, md.evict_serial.data_ptr(), None)
    md.compact(md.evict_serial, md.evict_count)         # explicit lists still work
    with pytest.raises(B.MemDecayError) as e:
        md.compact()                                      # the selection was applied
    assert e.value.status == B.MD_E_STATE
    torch.cuda.synchronize()
    assert md.device_status() == 0
    p.close()


def test_bad_eviction_serial_sets_status():
    p = small_pair(oracle_sessions=[])
    q, nk, reg, *_ = p.inputs(1)
    p.md.observe(1, q, nk, reg)
    p.md.score()
    ev = torch.zeros_like(p.md.evict_serial)
    ev[0, 0] = 9999
    cnt = torch.ones_like(p.md.evict_count)
    n_before = int(p.cache.n_pages[0].item())
    p.md.compact(ev, cnt)
    torch.cuda.synchronize()
    assert p.md.device_status() == B.MD_DEV_BAD_EVICT
    assert int(p.cache.n_pages[0].item()) == n_before
    p.close()


def test_state_lives_in_caller_buffers():
    # Snapshot every caller-owned buffer mid-run, run on, restore into a new
    # handle, run the same steps again: identical results.
    w = C.with_overrides(C.get("small"), steps=12)
    p = Pair(w, oracle_sessions=[])
    for _ in range(4):
        p.step(compare=False)
    names = ("k_pool", "region", "t_ins", "t_ref", "importance", "page_table", "page_serial",
             "n_pages", "n_tokens", "clock", "next_serial", "budget", "free_list", "free_count")
    snap = {n: getattr(p.cache, n).clone() for n in names}
    first = []
    for _ in range(4):
        p.step(compare=False)
        m = int(p.cache.n_pages[0].item())
        first.append(p.md.page_score[0, :m].clone())
    for n in names:
        getattr(p.cache, n).copy_(snap[n])
    p.md.close()
    from paper_2607_10582_amd.cache import MemDecay
    p.md = MemDecay(p.cache, torch.from_numpy(p.b), torch.from_numpy(p.lam), rho=0.9,
                    alpha=1.0, tau_scale=2.0, pinned_mask=1, fused=True)   # the Pair's path
    p.k = 4
    for i in range(4):
        p.step(compare=False)
        m = int(p.cache.n_pages[0].item())
        assert torch.equal(p.md.page_score[0, :m].view(torch.int32), first[i].view(torch.int32))
    p.close()


@pytest.mark.parametrize("cooperative", [False, True])
def test_kernel_timing(cooperative):
    # md_profile_enable / md_profile_read: every launch of a timed kernel is
    # counted once with a positive, finite duration (the fused kernel's
    # events come with its own dispatch on an ordinary launch, around it on
    # a cooperative one); a read resets the counts, and timing off stops them
    p = small_pair(oracle_sessions=[], fused=True, cooperative=cooperative)
    md = p.md
    md.profile(("append", "attend", "select", "compact"))
    for k in range(1, 5):
        p.step(compare=False)
    torch.cuda.synchronize()
    for name in ("append", "attend", "select", "compact"):
        ms, n = md.profile_read(name)
        assert n == 4, (name, n)
        assert np.isfinite(ms) and 0.0 < ms < 4 * 1000.0, (name, ms)
        assert md.profile_read(name) == (0.0, 0)
    md.profile(())
    p.step(compare=False)
    assert md.profile_read("attend") == (0.0, 0)
    assert md.device_status() == 0
    p.close()
