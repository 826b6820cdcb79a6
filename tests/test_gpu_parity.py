"""Device path vs. the CPU oracle, through the C ABI, on seeded workloads.

Tolerances (see tests/harness.py): priorities within 1e-5 relative; refresh
decisions and evicted serials exact except inside the 1e-5 bands around tau
and around the eviction threshold, where either answer is correct.
"""
import sys

import numpy as np
import pytest
import torch

from synth import configs as C
from synth import generator as g

from harness import Pair, REL

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a ROCm device")
    from paper_2607_10582_amd import binding
    binding.load_library()          # fails loudly when the library is missing


def run_pair(p: Pair, steps: int, label: str):
    say(f"[{label}] S={p.w.S} L={p.w.L} Hq={p.w.Hq} Hkv={p.w.Hkv} P={p.w.P} steps={steps}")
    for _ in range(steps):
        st = p.step()
    status = p.device_status()
    assert status == 0, f"device status {status:#x}"
    assert p.free_pages_consistent()
    say(f"[{label}] ok: {st.steps} steps, {st.tokens} token-steps, max rel {st.max_rel}, "
        f"tau-excused {st.tau_excused}, tie-excused {st.tie_excused}, evicted pages {st.evicted_pages}")
    p.close()
    return st


@pytest.mark.parametrize("fused", [True, False])
def test_small_workload_free_run(fused):
    w = C.get("small")
    p = Pair(w, fused=fused)
    assert p.md.kernel_config()["fused"] == fused
    st = run_pair(p, w.steps, f"small-fused{int(fused)}")
    assert st.evicted_pages > 10


@pytest.mark.parametrize("name", ["small", "qwen3_32x1700"])
def test_cooperative_launch(name):
    # MD_FLAG_COOPERATIVE: the fused kernel as a cooperative launch (the
    # default is an ordinary one); same results
    w = C.get(name)
    if name != "small":
        w = C.with_overrides(w, S=8, steps=12)
    p = Pair(w, fused=True, cooperative=True, oracle_sessions=[0, w.S - 1])
    assert p.md.kernel_config()["fused"]
    st = run_pair(p, w.steps, f"cooperative-{name}")
    assert st.evicted_pages > 10


def test_small_workload_planted_refresh():
    # Planted keys along a per-(layer, KV head) direction and queries that
    # lean on it: those tokens take mass >= tau and refresh their clocks.
    w = C.get("small")
    p = Pair(w, planted=48, planted_strength=3.0, query_gain=1.0)
    refreshed = 0
    for _ in range(w.steps):
        st = p.step()
        o = p.oracles[0]
        refreshed += int(np.sum(o.t_ref[:o.n_slots] == o.t))
    assert refreshed > 200
    p.close()


def test_small_workload_near_tau():
    # Planted strengths spread so that many masses land close to tau.
    w = C.get("small")
    strengths = np.linspace(1.6, 3.6, 120)
    p = Pair(w, planted=120, planted_strength=strengths, query_gain=0.5)
    run_pair(p, w.steps, "small-near-tau")


@pytest.mark.parametrize("fused", [True, False])
@pytest.mark.parametrize("P", [16, 64])
def test_ragged_edge_sessions(P, fused):
    # empty, single-token, exact-page, page+1, partial-tail and longer
    # sessions in one batch; budgets below, at and above the pinned span.
    w = C.with_overrides(C.get("small"), L=3, Hq=4, Hkv=2, S=7, n0=None, P=P,
                         n0_range=(1, 2), steps=40, system_len=20)
    n0s = [0, 1, 15, 16, 17, 130, 700]
    budgets = [0, 0, 5, 16, 10, 100, 200]
    run_pair(Pair(w, n0s=n0s, budgets=budgets, fused=fused), 40, f"ragged-edges-P{P}-fused{int(fused)}")


@pytest.mark.parametrize("Hq,Hkv", [(16, 2), (16, 1), (4, 4), (2, 1), (12, 12)])
def test_group_sizes(Hq, Hkv):
    w = C.with_overrides(C.get("small"), L=2, Hq=Hq, Hkv=Hkv, steps=12)
    run_pair(Pair(w), 12, f"G={Hq // Hkv}")


def test_no_pinning_zero_alpha():
    w = C.with_overrides(C.get("small"), steps=20)
    p = Pair(w, pinned_mask=0, alpha=0.0)
    run_pair(p, 20, "unpinned-alpha0")
    assert not p.warned


def test_infeasible_budget():
    w = C.with_overrides(C.get("small"), S=3, n0=None, n0_range=(1, 2), system_len=300, steps=10)
    p = Pair(w, n0s=[450, 320, 900], budgets=[100, 400, 50])
    p.step()
    inf = p.md.infeasible.cpu().numpy()
    assert inf.tolist() == [1, 0, 1]
    assert p.warned          # md_read_device_status returned MD_W_BUDGET_INFEASIBLE
    run_pair(p, 9, "infeasible")


def test_qwen15_single_session_full_run():
    w = C.get("qwen15_1700")
    st = run_pair(Pair(w), w.steps, "qwen15_1700")
    assert st.evicted_pages > 60


@pytest.mark.parametrize("one_call", [False, True])
def test_max_pages_per_session(one_call):
    # 8191 pages of 16 tokens in one session: every select thread holds 8
    # pages (with md_select_compact, the compaction's threads too).
    w = C.with_overrides(C.get("small"), L=1, n0=131050, steps=4, system_len=1024,
                         mean_span=512.0, budget_frac=0.25)
    kw = {}
    if one_call:
        # scores exact on both sides (every unpinned page 0.5), so the
        # device's selection is the oracle's and can be applied at once
        b, lam = flat_priors(w, {r: 0.5 for r in range(1, 7)} | {0: 1.0})
        kw = dict(priors=(b, lam), alpha=0.0, strict_ties=True)
    p = Pair(w, max_pages=8192, select_compact=one_call, check_free_list=one_call, **kw)
    assert p.cache.max_pages == 8192
    run_pair(p, 4, f"max-pages-one-call{int(one_call)}")


@pytest.mark.parametrize("fused,one_call", [(True, False), (False, False), (True, True)])
def test_max_sessions(fused, one_call):
    # 1,024 sessions (the most a handle takes) of 1 to 400 tokens: the work
    # lists, lane claims and passes at their largest; a sample of sessions
    # checked token by token, among them the first and the last.  With
    # md_select_compact, 1,024 blocks find their free-list places by the
    # look-back (more blocks than are resident at once) and the pushes are
    # checked in (session, serial) order.
    w = C.with_overrides(C.get("small"), S=1024, n0=None, n0_range=(1, 400), steps=4, system_len=30)
    kw = {}
    if one_call:   # exact scores on both sides, as in test_max_pages_per_session
        b, lam = flat_priors(w, {r: 0.5 for r in range(1, 7)} | {0: 1.0})
        kw = dict(priors=(b, lam), alpha=0.0, strict_ties=True)
    p = Pair(w, oracle_sessions=[0, 1, 255, 256, 511, 700, 1022, 1023], fused=fused,
             select_compact=one_call, check_free_list=one_call, **kw)
    run_pair(p, 4, f"max-sessions-fused{int(fused)}-one-call{int(one_call)}")


def test_long32k_sampled_sessions_multikernel_path():
    # The 16 x 32,768-token workload on the multi-kernel path (the fused
    # path's full trajectories are in test_gpu_full_size.py); two sessions
    # checked token by token through the bulk eviction and two more steps.
    w = C.get("long32k")
    p = Pair(w, backend="torch", oracle_sessions=[0, 11], steps=6, fused=False)
    run_pair(p, 3, "long32k-multikernel")


def test_hybrid_fused_and_spill_sessions():
    # One session longer than a whole pass of the fused kernel (it takes the
    # multi-kernel path) next to short ones (fused) in the same steps.
    w = C.with_overrides(C.get("small"), L=1, Hq=16, Hkv=2, S=3, n0=None, P=64,
                         n0_range=(1, 2), steps=3, system_len=1024, mean_span=512.0)
    probe = Pair(C.with_overrides(w, S=1), n0s=[64], budgets=[64], max_pages=8192,
                 oracle_sessions=[])
    cfg = probe.md.kernel_config()
    probe.close()
    big = cfg["unit_max"] * cfg["workgroups"] + 1000
    assert big <= 8190 * 64
    say(f"[hybrid] kernel config {cfg}, long session {big} tokens")
    p = Pair(w, n0s=[900, big, 3000], budgets=[300, big // 4, 3000], max_pages=8192)
    assert p.md.kernel_config()["spill"]
    run_pair(p, 3, "hybrid")


def test_fused_matches_multikernel_path():
    # Both device paths on the same inputs: attention masses and page scores
    # agree to rounding.  The budget holds every token and no step opens a
    # page (1700 + 3 tokens stay within 107 pages), so the slots line up.
    w = C.with_overrides(C.get("qwen3_32x1700"), S=6, steps=3, budget_frac=1.0)
    outs = []
    for fused in (True, False):
        p = Pair(w, oracle_sessions=[], fused=fused)
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


def test_determinism_two_runs():
    w = C.with_overrides(C.get("qwen15_1700"), L=4, steps=16)
    outs = []
    for _ in range(2):
        p = Pair(w, oracle_sessions=[])
        scores = []
        for _ in range(16):
            p.step(compare=False)
            scores.append(p.md.page_score.cpu().numpy().copy())
            scores.append(p.abar.cpu().numpy().copy())
        outs.append(scores)
        p.close()
    for a, b in zip(*outs):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_selection_on_scores_of_the_fused_kernel():
    # md_score_pages with both outputs NULL enqueues nothing: the selection
    # then runs on the page scores the fused observation kernel wrote.  The
    # same steps with the scoring kernel refilling them (outputs requested)
    # must evict exactly the same pages, from the bulk eviction on.
    w = C.with_overrides(C.get("qwen3_32x1700"), S=8, steps=8)
    runs = []
    for outputs in (True, False):
        p = Pair(w, oracle_sessions=[])
        assert p.md.kernel_config()["fused"] and not p.md.kernel_config()["spill"]
        ev = []
        for k in range(1, 9):
            q, nk, reg, *_ = p.inputs(k)
            p.md.observe(k, q, nk, reg)
            p.md.score(page_score=outputs)
            p.md.select()
            cnt = p.md.evict_count.cpu().numpy().copy()
            ser = p.md.evict_serial.cpu().numpy()
            ev.append([ser[s, :cnt[s]].copy() for s in range(w.S)])
            p.md.compact()
        torch.cuda.synchronize()
        assert p.device_status() == 0
        c = p.cache
        np_ = c.n_pages.cpu().numpy().copy()
        runs.append((ev, c.n_tokens.cpu().numpy().copy(), np_,
                     [c.page_serial.cpu().numpy()[s, :np_[s]].copy() for s in range(w.S)]))
        p.close()
    (ev1, nt1, np1, ser1), (ev2, nt2, np2, ser2) = runs
    assert sum(len(x) for x in ev1[0]) > 0
    for a, b in zip(ev1, ev2):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)
    assert np.array_equal(nt1, nt2) and np.array_equal(np1, np2)
    for x, y in zip(ser1, ser2):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("name,steady_fused", [("qwen15_1700", False), ("long32k", True), ("qwen3_32x1700", True)])
def test_library_picks_the_path(name, steady_fused):
    # Without a path flag the library runs the multi-kernel path for small
    # caches and the fused kernel for large ones (for a batch of small ones
    # with row groups); either way the steps match the oracle.
    w = C.get(name)
    big = w.name == "long32k"
    p = Pair(w, fused=None, backend="torch" if big else "numpy",
             oracle_sessions=[3] if big else None, steps=4 if big else 12)
    cfg = p.md.kernel_config()
    say(f"[{name}] kernel config {cfg}")
    assert cfg["steady_fused"] == steady_fused
    run_pair(p, 3 if big else 12, f"{name}-auto")


@pytest.mark.parametrize("fused", [True, False])
def test_normalised_attention_term(fused):
    # The score's attention term measured against the uniform attention level
    # (alpha * |K_t| * a_i, Sec. IV-D), on both observation paths; planted
    # keys give some tokens attention well above uniform.
    w = C.with_overrides(C.get("small"), attention_norm=True)
    p = Pair(w, planted=48, planted_strength=3.0, query_gain=1.0, fused=fused)
    st = run_pair(p, w.steps, f"norm-attention-fused{int(fused)}")
    assert st.evicted_pages > 10


def test_normalised_attention_term_batch():
    w = C.with_overrides(C.get("qwen3_32x1700"), S=8, attention_norm=True)
    run_pair(Pair(w, steps=10), 10, "norm-attention-qwen3x8")


@pytest.mark.parametrize("fused", [True, False])
@pytest.mark.parametrize("shape,W,k", [("g6", 2, 2), ("g4", 4, 4), ("g6", 1, 3), ("g6p64", 2, 3)])
def test_window_and_observation_interval(shape, W, k, fused):
    # Attention sampled every k-th decode step with a window of the W latest
    # decode queries (Sec. III-C); the steps in between only append.  A
    # causal mask keeps each window query to the tokens of its own step; on
    # the fused kernel the window's queries are extra MFMA columns.
    base = C.get("small")
    if shape == "g4":
        base = C.with_overrides(base, L=2, Hq=8, Hkv=2)
    if shape == "g6p64":
        base = C.with_overrides(base, L=2, P=64, n0=700, budget_frac=0.3)
    w = C.with_overrides(base, window=W, obs_interval=k, steps=24)
    p = Pair(w, fused=fused, planted=24, planted_strength=2.5, query_gain=0.7)
    assert p.md.kernel_config()["steady_fused"] == fused
    st = run_pair(p, 24, f"window{W}-every{k}-{shape}-fused{int(fused)}")
    assert st.evicted_pages > 5


@pytest.mark.parametrize("fused", [True, False])
def test_window_on_a_batch_with_empty_and_short_sessions(fused):
    w = C.with_overrides(C.get("small"), L=3, Hq=4, Hkv=2, S=5, n0=None, n0_range=(1, 2),
                         window=3, obs_interval=3, steps=30, system_len=20)
    p = Pair(w, n0s=[0, 1, 17, 130, 700], budgets=[0, 5, 10, 100, 200], fused=fused)
    run_pair(p, 30, f"window3-edges-fused{int(fused)}")


def test_window_long32k_sampled_sessions():
    # the 32k batch observed every other step with a window of two, on the
    # fused kernel (G W = 12 columns)
    w = C.get("long32k_w2k2")
    p = Pair(w, backend="torch", oracle_sessions=[0, 11], steps=6, fused=True)
    assert p.md.kernel_config()["steady_fused"]
    run_pair(p, 6, "window2-long32k-fused")


@pytest.mark.parametrize("aligned", [False, True])
def test_lifetime_statistics_and_decay_fit(aligned):
    # Region-lifetime calibration (Sec. IV-B): after every observation the
    # device adds each cached token's attention mass to its (region, age
    # bucket) bin; the oracle does the same in float64.  The budget holds
    # every token, as in a measurement pass.  Counts and age sums are exact
    # integers; mass sums agree within 1e-5 relative plus the fixed-point
    # rounding; the Eq. 6 fits of the two agree closely.
    from oracle.calibration import LifetimeStats, fit_decay
    from paper_2607_10582_amd import binding as B
    w = C.with_overrides(C.get("qwen15_1700"), L=4, steps=24, region_aligned=aligned, append_run=4)
    p = Pair(w, planted=64, planted_strength=2.0, query_gain=0.5, budgets=[10**6])
    bucket, nb, nr = 64, 32, 7
    dev = [torch.zeros((w.S, nr, nb), dtype=torch.int64, device="cuda") for _ in range(3)]
    ost = LifetimeStats(nr, bucket, nb)
    for _ in range(24):
        p.step()
        p.md.calib_accumulate(p.abar, bucket, dev)
        o, rec = p.oracles[0], p.last_rec[0]
        live = o.live()
        ost.add(rec.t, o.t_ins[live], o.region[live], rec.abar)
    torch.cuda.synchronize()
    assert p.device_status() == 0
    mass, count, age = [x.cpu().numpy().view(np.uint64)[0] for x in dev]
    assert np.array_equal(count.astype(np.int64), ost.count)
    assert np.array_equal(age.astype(np.int64), ost.age_sum)
    got = mass.astype(np.float64) / 2.0**40
    np.testing.assert_allclose(got, ost.mass, rtol=1e-5, atol=ost.count.max() * 2.0**-40)
    lam, logc = B.md_calib_fit(mass[None], count[None], age[None])
    olam, ologc = fit_decay(ost.mass, ost.count, ost.age_sum)
    assert np.array_equal(np.isnan(lam), np.isnan(olam)) and np.count_nonzero(~np.isnan(olam)) >= 5
    ok = ~np.isnan(olam)
    np.testing.assert_allclose(lam[ok], olam[ok], rtol=1e-3, atol=1e-7)
    say(f"[calibration] fitted half-lives {np.round(np.log(2) / lam, 1)}")
    p.close()


# ---------------------------------------------------------------- region-aligned pages

def check_aligned_layout(p: Pair):
    """On the device: every page of every session holds one region, its holes
    come after its last token, and only pages closed at a region boundary
    have holes."""
    from paper_2607_10582_amd import binding as B
    c, P = p.cache, p.w.P
    reg = c.region.cpu().numpy()
    npg = c.n_pages.cpu().numpy()
    npos = c.n_tokens.cpu().numpy()
    nlive = c.n_live.cpu().numpy()
    ptab = c.page_table.cpu().numpy()
    for s in range(p.w.S):
        live = 0
        for i in range(int(npg[s])):
            used = P if i < npg[s] - 1 else int(npos[s]) - (int(npg[s]) - 1) * P
            r = reg[ptab[s, i], :used]
            hole = r == B.MD_REGION_HOLE
            k = int(np.count_nonzero(~hole))
            assert k >= 1 and not hole[:k].any() and hole[k:].all(), (s, i, r)
            assert np.all(r[:k] == r[0]), (s, i, r)
            live += k
        assert live == int(nlive[s]), (s, live, int(nlive[s]))


@pytest.mark.parametrize("fused", [True, False])
def test_region_aligned_small(fused):
    # Region-aligned pages (the allocator variant of Sec. III-D): a fresh page
    # at every region boundary, in the prompt and in the decode stream (turns
    # of 5 tokens per region).  Parity step by step, then the layout.
    w = C.get("small_aligned")
    p = Pair(w, fused=fused, planted=24, planted_strength=2.5, query_gain=0.7)
    say(f"[aligned-small] pages {int(p.cache.n_pages[0])}, slots {int(p.cache.n_tokens[0])}, "
        f"tokens {int(p.cache.n_live[0])}")
    check_aligned_layout(p)
    for _ in range(w.steps):
        st = p.step()
        check_aligned_layout(p)
    assert p.device_status() == 0 and p.free_pages_consistent()
    say(f"[aligned-small-fused{int(fused)}] ok: {st.steps} steps, max rel {st.max_rel}, "
        f"evicted pages {st.evicted_pages}")
    p.close()
    assert st.evicted_pages > 10


@pytest.mark.parametrize("fused", [True, False])
def test_region_aligned_long32k_sampled_sessions(fused):
    # The 16 x 32,768-token batch with region-aligned pages, inputs drawn on
    # the device, two sessions checked token by token.
    w = C.get("long32k_aligned")
    p = Pair(w, backend="torch", oracle_sessions=[0, 11], steps=6, fused=fused)
    check_aligned_layout(p)
    run_pair(p, 3, f"aligned-long32k-fused{int(fused)}")


@pytest.mark.parametrize("P", [16, 64])
def test_region_aligned_ragged_batch(P):
    # Short spans (mean 40) so that most pages of P = 64 close early, empty
    # and one-token sessions, and the fused kernel with its lanes.
    w = C.with_overrides(C.get("small"), L=2, Hq=16, Hkv=2, S=6, n0=None, n0_range=(1, 2), P=P,
                         append_cycle=C.APPEND_CYCLE, region_aligned=True, append_run=3, steps=12,
                         system_len=30)
    p = Pair(w, n0s=[0, 1, 40, 333, 1200, 3000], budgets=[0, 1, 20, 150, 500, 1000], fused=True)
    check_aligned_layout(p)
    run_pair(p, 12, f"aligned-ragged-P{P}")


@pytest.mark.parametrize("fused", [True, False])
def test_region_aligned_window(fused):
    # W = 2 window queries every other step on both paths: the causal mask
    # and the hole mask together.
    w = C.with_overrides(C.get("small_aligned"), window=2, obs_interval=2, steps=24)
    p = Pair(w, fused=fused, planted=24, planted_strength=2.5, query_gain=0.7)
    assert p.md.kernel_config()["fused"] == fused
    run_pair(p, 24, f"aligned-window2-fused{int(fused)}")


# ---------------------------------------------------------------- quantised tier

def run_quant(p: Pair, steps: int, label: str):
    say(f"[{label}] S={p.w.S} L={p.w.L} Hq={p.w.Hq} P={p.w.P} thr={p.w.quant_threshold} steps={steps}")
    for _ in range(steps):
        st = p.step()
    assert p.device_status() == 0 and p.free_pages_consistent()
    nq = sum(int(pg.quant) for o in p.oracles.values() for pg in o.pages)
    say(f"[{label}] ok: {st.steps} steps, max rel {st.max_rel}, evicted pages {st.evicted_pages}, "
        f"quantised pages now {nq}")
    p.close()
    return nq


@pytest.mark.parametrize("fused", [True, False])
@pytest.mark.parametrize("thr", [0.35, float("inf")])
def test_quantised_tier_small(thr, fused):
    # The quantised tier (Sec. III-E): pages scoring below the threshold keep
    # 8-bit codes; the codes and scales written on the device equal the
    # oracle's bit for bit (checked in the harness after every step), and the
    # attention over them matches within the usual tolerance.
    w = C.with_overrides(C.get("small"), quant_threshold=thr)
    p = Pair(w, fused=fused, planted=24, planted_strength=2.5, query_gain=0.7)
    assert run_quant(p, w.steps, f"quant-small-{thr}-fused{int(fused)}") > 2


@pytest.mark.parametrize("fused", [True, False])
def test_quantised_tier_3b_shape_pages_of_64_region_aligned(fused):
    w = C.with_overrides(C.get("small"), L=2, Hq=16, Hkv=2, P=64, n0=900, budget_frac=0.6,
                         append_cycle=C.APPEND_CYCLE, region_aligned=True, append_run=4,
                         quant_threshold=0.4, steps=20)
    p = Pair(w, fused=fused)
    assert run_quant(p, 20, f"quant-3b-p64-aligned-fused{int(fused)}") > 0


@pytest.mark.parametrize("aligned", [False, True])
@pytest.mark.parametrize("fused", [True, False])
def test_quantised_tier_with_a_window(fused, aligned):
    # quantised tiles under a window of two queries, on plain and on
    # region-aligned pages, on both observation paths
    w = C.with_overrides(C.get("small_aligned" if aligned else "small"), L=2, window=2, obs_interval=2,
                         quant_threshold=0.35, steps=24)
    p = Pair(w, fused=fused, planted=24, planted_strength=2.5, query_gain=0.7)
    assert p.md.kernel_config()["fused"] == fused
    assert run_quant(p, 24, f"quant-window2-aligned{int(aligned)}-fused{int(fused)}") > 0


def test_quantised_tier_long32k_sampled_sessions():
    w = C.with_overrides(C.get("long32k"), quant_threshold=0.3)
    p = Pair(w, backend="torch", oracle_sessions=[0, 11], steps=6, fused=True)
    assert run_quant(p, 3, "quant-long32k") > 0


# ---------------------------------------------------------------- exact ties

def flat_priors(w, b_of_region):
    """Region tables with lambda = 0 (no decay): a token scores b of its
    region exactly when alpha = 0."""
    b = np.zeros((w.S, 7), np.float32)
    for r, v in b_of_region.items():
        b[:, r] = v
    return b, np.zeros((w.S, 7), np.float32)


@pytest.mark.parametrize("fused", [True, False])
@pytest.mark.parametrize("P", [16, 64])
def test_exact_ties_go_to_the_older_page(P, fused):
    # lambda = 0, alpha = 0 and b = 0.5 for every movable region: every
    # unpinned page scores exactly 0.5 on both sides (sums of 0.5 and their
    # quotients by the member count are exact in float32), so the eviction
    # is decided by serial alone, the older page first (the min-heap order
    # read as ascending (S_p, serial)).  With 20,000 tokens at P = 16 a
    # session holds 1,250 pages, more than the selection's 1,024 threads, so
    # the walk over the pages of the threshold key crosses thread runs.  The
    # evicted serials must equal the oracle's exactly.
    w = C.with_overrides(C.get("small"), S=3, n0=None, n0_range=(1, 2), P=P, system_len=64,
                         mean_span=512.0, steps=6, append_cycle=C.APPEND_CYCLE)
    b, lam = flat_priors(w, {r: 0.5 for r in range(1, 7)} | {0: 1.0})
    p = Pair(w, n0s=[20000, 17001, 3000], budgets=[10000, 4000, 2999], priors=(b, lam), alpha=0.0,
             strict_ties=True, fused=fused)
    st = run_pair(p, 6, f"exact-ties-P{P}-fused{int(fused)}")
    assert st.evicted_pages > 500 // (P // 16) and st.tie_excused == 0


@pytest.mark.parametrize("fused", [True, False])
def test_exact_ties_on_region_aligned_pages_below_and_at_the_threshold(fused):
    # Region-aligned pages hold one region each, so a page scores its
    # region's b exactly: 0.25 for plan, tool_in and retrieval, 0.5 for the
    # others.  The bulk eviction takes every 0.25 page, then 0.5 pages in
    # serial order until the budget holds.
    w = C.with_overrides(C.get("small"), S=2, n0=None, n0_range=(1, 2), system_len=64, mean_span=300.0,
                         steps=6, append_cycle=C.APPEND_CYCLE, region_aligned=True, append_run=2)
    b, lam = flat_priors(w, {0: 1.0, 1: 0.25, 2: 0.5, 3: 0.25, 4: 0.5, 5: 0.25, 6: 0.5})
    p = Pair(w, n0s=[18000, 9000], budgets=[5000, 4500], priors=(b, lam), alpha=0.0, strict_ties=True,
             fused=fused)
    st = run_pair(p, 6, f"exact-ties-aligned-fused{int(fused)}")
    assert st.evicted_pages > 500 and st.tie_excused == 0


@pytest.mark.parametrize("fused", [True, False])
def test_region_aligned_closed_page_stays_closed(fused):
    # 16 system and 5 plan tokens.  Step 1 appends a user token (b = 0): it
    # closes the plan page, opens its own page and is evicted at once.  Step 2
    # appends a plan token: the plan page is the last page again but stays
    # closed, so the token opens a fresh page (serial 3); the tie between the
    # two plan pages (both score 1) then evicts the older one.
    from synth.configs import PLAN, USER
    w = C.with_overrides(C.get("small"), n0=21, system_len=16, region_aligned=True, append_cycle=(USER, PLAN),
                         append_run=1, steps=4)
    b, lam = flat_priors(w, {0: 1.0, PLAN: 1.0, USER: 0.0, 3: 1.0, 4: 1.0, 5: 1.0, 6: 1.0})
    p = Pair(w, regions=[np.array([0] * 16 + [PLAN] * 5, np.uint8)], budgets=[21], priors=(b, lam),
             alpha=0.0, strict_ties=True, fused=fused)
    p.step()
    assert p.cache.page_serial[0, :int(p.cache.n_pages[0])].tolist() == [0, 1]
    p.step()
    assert p.cache.page_serial[0, :int(p.cache.n_pages[0])].tolist() == [0, 3]
    run_pair(p, 2, f"aligned-closed-page-fused{int(fused)}")


# ---------------------------------------------------------------- free list

@pytest.mark.parametrize("fused", [True, False])
@pytest.mark.parametrize("explicit", [False, True])
def test_free_list_order(fused, explicit):
    # 12 sessions: each append takes pages off the top of the free list in
    # session order, and each compaction pushes the freed ids in (session,
    # serial) order; the harness checks both at every step, for md_compact
    # without lists (this step's selection) and with the same lists given
    w = C.with_overrides(C.get("qwen3_32x1700"), L=2, S=12, steps=24)
    p = Pair(w, oracle_sessions=[0, 7], check_free_list=True, fused=fused, explicit_lists=explicit)
    run_pair(p, 24, f"free-list-order-fused{int(fused)}-explicit{int(explicit)}")


# ---------------------------------------------------------------- one-call selection and compaction

@pytest.mark.parametrize("fused", [True, False])
def test_select_compact_free_list_order(fused):
    # md_select_compact (one launch: each session's block selects and
    # compacts, the blocks find their free-list places by a look-back over
    # tagged counts): the same pops and (session, serial) pushes as the two
    # calls, and the oracle's selection at every step
    w = C.with_overrides(C.get("qwen3_32x1700"), L=2, S=12, steps=24)
    p = Pair(w, oracle_sessions=[0, 7], check_free_list=True, fused=fused, select_compact=True)
    run_pair(p, 24, f"select-compact-free-list-fused{int(fused)}")


@pytest.mark.parametrize("P", [16, 64])
def test_select_compact_exact_ties(P):
    # the exact-tie batch (every unpinned page scores 0.5; more pages than
    # the block's threads), selected and compacted in one launch
    w = C.with_overrides(C.get("small"), S=3, n0=None, n0_range=(1, 2), P=P, system_len=64,
                         mean_span=512.0, steps=6, append_cycle=C.APPEND_CYCLE)
    b, lam = flat_priors(w, {r: 0.5 for r in range(1, 7)} | {0: 1.0})
    p = Pair(w, n0s=[20000, 17001, 3000], budgets=[10000, 4000, 2999], priors=(b, lam), alpha=0.0,
             strict_ties=True, check_free_list=True, select_compact=True)
    st = run_pair(p, 6, f"select-compact-exact-ties-P{P}")
    assert st.evicted_pages > 500 // (P // 16) and st.tie_excused == 0


def test_select_compact_region_aligned_and_infeasible():
    # region-aligned pages (live counts from the region codes) with exact
    # ties, and a session whose pinned tokens exceed its budget
    w = C.with_overrides(C.get("small"), S=3, n0=None, n0_range=(1, 2), system_len=64, mean_span=300.0,
                         steps=6, append_cycle=C.APPEND_CYCLE, region_aligned=True, append_run=2)
    b, lam = flat_priors(w, {0: 1.0, 1: 0.25, 2: 0.5, 3: 0.25, 4: 0.5, 5: 0.25, 6: 0.5})
    p = Pair(w, n0s=[18000, 9000, 500], budgets=[5000, 4500, 32], priors=(b, lam), alpha=0.0,
             strict_ties=True, check_free_list=True, select_compact=True)
    st = run_pair(p, 6, "select-compact-aligned")
    assert st.evicted_pages > 500 and st.tie_excused == 0 and p.warned


def test_select_compact_with_the_quantised_tier():
    # with a tier the call makes the two calls' launches (the tier runs
    # between the selection and the compaction)
    w = C.with_overrides(C.get("small"), quant_threshold=0.35, steps=12)
    p = Pair(w, select_compact=True)
    run_pair(p, 12, "select-compact-quant")


def test_select_compact_long32k_sampled_sessions():
    # the 32k batch as the benchmark runs it (fused observation, one-call
    # selection and compaction): the bulk eviction, then steady steps
    w = C.with_overrides(C.get("long32k"), steps=20)
    p = Pair(w, backend="torch", oracle_sessions=[0, 11], fused=None, check_free_list=True,
             select_compact=True)
    st = run_pair(p, 20, "select-compact-long32k")
    assert st.evicted_pages > 2 * (32768 - 8192) // 16


def test_physical_pages_are_reproducible():
    # Two runs of the same batch hand out the same physical pages.
    w = C.with_overrides(C.get("qwen3_32x1700"), L=2, S=10, steps=20)
    runs = []
    for _ in range(2):
        p = Pair(w, oracle_sessions=[])
        tabs = []
        for _ in range(20):
            p.step(compare=False)
            c = p.cache
            tabs.append((c.page_table.cpu().numpy().copy(), c.free_list.cpu().numpy().copy(),
                         int(c.free_count.item())))
        assert p.device_status() == 0
        runs.append(tabs)
        p.close()
    for (t1, f1, c1), (t2, f2, c2) in zip(*runs):
        assert np.array_equal(t1, t2) and c1 == c2 and np.array_equal(f1[:c1], f2[:c2])


# ---------------------------------------------------------------- offload tier

def run_offload(p: Pair, steps: int, label: str):
    say(f"[{label}] S={p.w.S} L={p.w.L} Hq={p.w.Hq} P={p.w.P} host pages {p.offload_pages} steps={steps}")
    for _ in range(steps):
        st = p.step()
    assert p.device_status() == 0 and p.free_pages_consistent()
    c = p.md.counters()
    say(f"[{label}] ok: {st.steps} steps, max rel {st.max_rel}, evicted {st.evicted_pages}, offloaded "
        f"{st.offloaded}, recalled {st.recalled}, dropped {st.dropped}; device counters {c}")
    if len(p.oracle_sessions) == p.w.S:   # the counters cover every session
        assert c[4] == st.offloaded and c[5] == st.recalled and c[6] == st.dropped
    p.close()
    return st


@pytest.mark.parametrize("fused", [True, False])
def test_offload_tier_small_batch(fused):
    # The offload tier (Sec. III-E's second tier): three sessions, keys
    # planted so that attention moves between tokens; pages leaving the
    # cache go to host memory (8 per session) and come back when a token's
    # mass next to the cached tokens reaches tau.  Everything is compared
    # with the oracle at every step, the host-memory list, its tokens'
    # state and scores and the copied keys included.
    w = C.with_overrides(C.get("small"), S=3, n0=None, n0_range=(1, 2), steps=48, system_len=60)
    p = Pair(w, n0s=[450, 700, 300], budgets=[225, 300, 200], planted=24, planted_strength=2.5, query_gain=0.7,
             fused=fused, offload_pages=8, drop_threshold=1e-3)
    st = run_offload(p, 48, f"offload-small-fused{int(fused)}")
    assert st.offloaded > 30 and st.recalled > 20


@pytest.mark.parametrize("fused", [True, False])
def test_offload_tier_drops_pages_below_the_threshold(fused):
    # a larger refresh scale (tau = 8 / |K_t|) keeps most host-memory pages
    # from coming back, so they age below the drop threshold and are dropped
    w = C.with_overrides(C.get("small"), S=2, n0=None, n0_range=(1, 2), steps=48, tau_scale=8.0)
    p = Pair(w, n0s=[450, 600], budgets=[225, 240], planted=24, planted_strength=2.5, query_gain=0.7,
             fused=fused, offload_pages=4, drop_threshold=0.05)
    st = run_offload(p, 48, f"offload-drops-fused{int(fused)}")
    assert st.offloaded > 5 and st.dropped > 0


@pytest.mark.parametrize("fused", [True, False])
def test_offload_tier_with_quantised_pages_of_64(fused):
    # 3B shape, pages of 64, the quantised tier on: quantised pages move to
    # host memory as codes and scales and come back unchanged
    w = C.with_overrides(C.get("small"), L=2, Hq=16, Hkv=2, P=64, n0=900, budget_frac=0.6,
                         append_cycle=C.APPEND_CYCLE, quant_threshold=0.4, steps=20)
    p = Pair(w, planted=24, planted_strength=2.5, query_gain=0.7, fused=fused, offload_pages=8, drop_threshold=1e-3)
    st = run_offload(p, 20, f"offload-quant-p64-fused{int(fused)}")
    assert st.offloaded > 10 and st.recalled > 5


def test_offload_tier_long32k_sampled_sessions():
    # the 16 x 32,768-token batch with 16 host-memory pages per session and
    # no drop threshold: the bulk eviction fills host memory with the best
    # of the 1,536 pages each session evicts, later steps observe them
    w = C.get("long32k")
    p = Pair(w, backend="torch", oracle_sessions=[0, 11], steps=6, fused=True, offload_pages=16,
             drop_threshold=0.0)
    st = run_offload(p, 4, "offload-long32k")
    assert st.offloaded >= 32
