"""Drive the device path (through the C ABI) and the CPU oracle on the same
seeded inputs, one decode step at a time, and compare them.

Comparison rules
----------------
* Attention mass, importance, token scores and page scores: within
  REL = 1e-5 relative (float32 accumulation on the device, float64 in the
  oracle), with an absolute floor ABS for values that underflow in float32.
* Refresh clocks: equal, except for tokens whose oracle mass lies within
  REL * tau of tau: either decision is correct there (excused, counted).
* Evicted page serials: equal, except for pages whose oracle page score lies
  within REL of the oracle's eviction threshold (the largest evicted score),
  or pages holding an excused token: there several answers are correct.  The
  device's own selection must in any case be the ascending-(score, serial)
  prefix of its own scores that meets the budget (checked here, in the test).
* With strict_ties=True (inputs built so that page scores tie exactly on
  both sides) the evicted serials must be identical: no tie band.
* With check_free_list=True the free list is checked at every step: an
  append takes its pages in session order off the top of the stack, and a
  compaction pushes the freed physical ids in (session, serial) order.
* After a comparison the oracle's discrete decisions are carried to the
  device when an excusal let them differ: the oracle's refresh clock is
  written over the device's for excused tokens, and md_compact applies the
  oracle's eviction list.  Data only flows from the oracle to the device.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np
import torch

import oracle
from oracle.pool import SessionPool
from paper_2607_10582_amd import binding as B
from paper_2607_10582_amd.cache import MemDecay, PagedCache
from synth import configs as C
from synth import generator as g

REL = 1e-5
ABS = 1e-30


def f32(x) -> float:
    return float(np.float32(x))


def bits_to_torch(bits: np.ndarray, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(device).view(torch.bfloat16)


def torch_to_bits(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def rel_err(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return np.abs(got - ref) / np.maximum(np.abs(ref), ABS / REL)


def check_selection_prefix(scores, serials, sizes, pinned, n, budget, P, evicted, infeasible):
    """Selection invariants on one side's own scores (no oracle involved)."""
    ev = set(int(x) for x in evicted)
    cand = [i for i in range(len(serials)) if not pinned[i]]
    assert all(int(serials[i]) in ev for i in cand) if infeasible else True
    assert not any(int(serials[i]) in ev for i in range(len(serials)) if pinned[i])
    removed = sum(int(sizes[i]) for i in range(len(serials)) if int(serials[i]) in ev)
    if not infeasible:
        assert n - removed <= budget
        if ev:
            assert n - removed > budget - P
            order = sorted(cand, key=lambda i: (float(scores[i]), int(serials[i])))
            k = len(ev)
            assert set(int(serials[i]) for i in order[:k]) == ev
    else:
        assert n - removed > budget


@dataclass
class Stats:
    steps: int = 0
    tokens: int = 0
    max_rel: Dict[str, float] = field(default_factory=lambda: {"abar": 0.0, "a": 0.0, "score": 0.0,
                                                               "page": 0.0})
    tau_excused: int = 0
    tie_excused: int = 0
    evicted_pages: int = 0
    offloaded: int = 0        # offload tier: pages moved to host memory,
    recalled: int = 0         # recalled from it,
    dropped: int = 0          # dropped from it

    def bump(self, key, arr):
        if arr.size:
            self.max_rel[key] = max(self.max_rel[key], float(np.max(arr)))


class Pair:
    """One workload on the device and in the oracle (for ``oracle_sessions``)."""

    def __init__(self, w: C.Workload, *, device="cuda", backend="numpy",
                 oracle_sessions: Optional[List[int]] = None, n0s=None, budgets=None,
                 regions=None, planted: int = 0, planted_strength=3.0, query_gain=0.0,
                 pinned_mask=None, alpha=None, n_phys_extra: int = 0, max_pages=None,
                 steps=None, fused: Optional[bool] = True, priors=None, strict_ties: bool = False,
                 check_free_list: bool = False, static: bool = False, pool: int = 0,
                 offload_pages: int = 0, drop_threshold: float = 0.0, cooperative: bool = False,
                 explicit_lists: bool = False, select_compact: bool = False, row_groups: bool = True):
        # pool > 0: the oracle sessions run in that many worker processes
        # (oracle.pool), all sessions of a step at once
        self.w = w
        self.dev = torch.device(device)
        self.backend = backend
        self.steps = w.steps if steps is None else steps
        self.n0s = g.prefix_lengths(w) if n0s is None else np.asarray(n0s, np.int64)
        S = len(self.n0s)
        assert S == w.S
        self.B = g.budgets(w, self.n0s) if budgets is None else np.asarray(budgets, np.int64)
        self.b, self.lam = g.region_priors(w) if priors is None else \
            (np.asarray(priors[0], np.float32), np.asarray(priors[1], np.float32))
        self.strict_ties = strict_ties
        self.check_free_list = check_free_list
        # explicit_lists: md_compact always gets the lists (else without them
        # whenever the device's selection is the oracle's)
        self.explicit_lists = explicit_lists
        # select_compact: the selection and its application as one call
        # (md_select_compact); the device's selection must then equal the
        # oracle's at every step, since it is applied before the comparison
        self.select_compact = select_compact
        assert not (select_compact and explicit_lists)
        self.pinned_mask = w.pinned_mask if pinned_mask is None else pinned_mask
        self.alpha = w.alpha if alpha is None else alpha
        self.oracle_sessions = list(range(S)) if oracle_sessions is None else list(oracle_sessions)
        self.query_gain = query_gain
        self.planted = planted
        P = w.P
        al = w.region_aligned
        w_steps = C.with_overrides(w, steps=self.steps)
        n_phys = g.pages_needed(w_steps, self.n0s) + n_phys_extra
        regs = [g.region_spans(w, s, int(self.n0s[s])) if regions is None else np.asarray(regions[s], np.uint8)
                for s in range(S)]
        pages = [PagedCache.pages_for(regs[s], P, al) for s in range(S)]
        grow = self.steps if al else (self.steps + P - 1) // P
        mp = max(max(pages) + grow + 1, 1) if max_pages is None else max_pages
        self.cache = PagedCache(L=w.L, Hq=w.Hq, Hkv=w.Hkv, d=w.d, P=P, S=S, max_pages=mp,
                                n_phys=n_phys, device=self.dev, offload_pages=offload_pages)
        self.offload_pages = offload_pages
        perm = g.page_permutation(w, n_phys)
        pos = 0
        self.oracles: Dict[int, oracle.Session] = {}
        self.pool = SessionPool(pool) if pool else None
        for s in range(S):
            n0 = int(self.n0s[s])
            reg = regs[s]
            m = pages[s]
            ids = perm[pos:pos + m]
            pos += m
            if backend == "numpy":
                kb = g.k_prefix(w, s, n0)
                if planted:
                    toks = g.planted_tokens(w, s, n0, planted)
                    kb = g.planted_keys(w, s, kb, toks, planted_strength)
                kt = bits_to_torch(kb, self.dev)
            else:
                kt = g.torch_keys(w, s, n0, self.dev)
                kb = torch_to_bits(kt) if s in self.oracle_sessions else None
            if n0:
                self.cache.load_session(s, kt.view(n0, w.L, w.Hkv, w.d), reg, ids,
                                        budget=int(self.B[s]), clock=n0, region_aligned=al)
            else:
                self.cache.budget[s] = int(self.B[s])
                self.cache.clock[s] = 0
            del kt
            if s in self.oracle_sessions:
                kw = dict(L=w.L, Hq=w.Hq, Hkv=w.Hkv, d=w.d, P=P, b=self.b[s], lam=self.lam[s],
                          alpha=f32(self.alpha), rho=f32(w.rho), tau_scale=f32(w.tau_scale),
                          pinned_mask=self.pinned_mask, budget=int(self.B[s]), clock=n0, region=reg,
                          capacity=n0 + self.steps, attention_norm=w.attention_norm, region_aligned=al,
                          quant_threshold=w.quant_threshold, offload_pages=offload_pages,
                          drop_threshold=drop_threshold)
                kbs = kb if n0 else np.zeros((0, w.L, w.Hkv, w.d), np.uint16)
                if self.pool is not None:
                    self.pool.add(s, kw, kbs, n0)
                else:
                    self.oracles[s] = oracle.Session(keys_bits=kbs, **kw)
            del kb
        self.cache.set_free_pages(perm[pos:][::-1])
        self.md = MemDecay(self.cache, torch.from_numpy(self.b), torch.from_numpy(self.lam),
                           rho=f32(w.rho), alpha=f32(self.alpha), tau_scale=f32(w.tau_scale),
                           pinned_mask=self.pinned_mask, fused=fused, attention_norm=w.attention_norm,
                           window=w.window, region_aligned=al, quant_threshold=w.quant_threshold,
                           static=static, drop_threshold=f32(drop_threshold), cooperative=cooperative,
                           row_groups=row_groups)
        n_slots = n_phys * P
        self.abar = torch.zeros(n_slots, dtype=torch.float32, device=self.dev)
        self.tscore = torch.zeros(n_slots, dtype=torch.float32, device=self.dev)
        self.stats = Stats()
        self.last_rec = {}
        self.status_seen = 0
        self.warned = False        # md_read_device_status returned MD_W_BUDGET_INFEASIBLE
        self.k = 0

    # -------------------------------------------------------------- inputs
    def inputs(self, k: int):
        w, S = self.w, self.w.S
        reg = np.full(S, g.append_region(w, k), dtype=np.uint8)
        obs = g.observes(w, k)       # queries exist only at observation steps
        if self.backend == "numpy":
            q = np.stack([g.q_window(w, s, k) if obs else np.zeros((w.window, w.L, w.Hq, w.d), np.float32)
                          for s in range(S)])                            # [S][W][L][Hq][d]
            if self.query_gain:
                q = np.stack([np.stack([g.planted_query(w, s, qw, self.query_gain) for qw in q[s]])
                              for s in range(S)])
            nk = np.stack([g.k_append(w, s, k) for s in range(S)])
            qt = torch.from_numpy(q).to(self.dev)
            nkt = bits_to_torch(nk, self.dev)
            qo = {s: q[s] for s in self.oracle_sessions}
            nko = {s: nk[s] for s in self.oracle_sessions}
        else:
            qt = torch.stack([g.torch_queries(w, k - w.window + 1 + j, self.dev) if obs else
                              torch.zeros((S, w.L, w.Hq, w.d), device=self.dev)
                              for j in range(w.window)], dim=1).contiguous()
            nkt = g.torch_append_keys(w, k, self.dev)
            qh = qt.cpu().numpy()
            qo = {s: qh[s] for s in self.oracle_sessions}
            nb = torch_to_bits(nkt)
            nko = {s: nb[s] for s in self.oracle_sessions}
        return qt, nkt, torch.from_numpy(reg).to(self.dev), qo, nko, reg

    # -------------------------------------------------------------- one step
    def step(self, compare: bool = True):
        self.k += 1
        k = self.k
        w, P, S = self.w, self.w.P, self.w.S
        qt, nkt, regt, qo, nko, reg = self.inputs(k)
        md = self.md
        if self.check_free_list:
            torch.cuda.synchronize(self.dev)
            before = self.free_list_state()
        if not g.observes(w, k):
            # a decode step without an observation: append only, on both sides
            md.observe(k, None, nkt, regt)
            torch.cuda.synchronize(self.dev)
            nt_dev = self.live_counts()
            recs = self.oracle_step({s: (None, nko[s], int(reg[s])) for s in self.oracle_sessions})
            for s in self.oracle_sessions:
                rec = recs[s]
                if compare:
                    assert int(nt_dev[s]) == rec.n, (k, s, "append-only n")
            self.stats.steps += 1
            return self.stats
        md.observe(k, qt, nkt, regt, abar_out=self.abar)
        if self.check_free_list:
            torch.cuda.synchronize(self.dev)
            self.check_pops(before, self.free_list_state())
        md.score(token_score=self.tscore)
        c = self.cache

        def snapshot():
            h = {name: getattr(c, name).cpu().numpy() for name in
                 ("page_table", "page_serial", "n_pages", "n_tokens", "importance", "t_ref", "region")}
            h["n_live"] = self.live_counts()
            return h

        if self.select_compact:
            # the tables as the selection sees them, then both in one call
            torch.cuda.synchronize(self.dev)
            host = snapshot()
            if self.check_free_list:
                pre_compact = self.free_list_state()
            md.select_compact()
        else:
            md.select()
        torch.cuda.synchronize(self.dev)
        rc, dev_status = md.device_status(with_warning=True)
        self.warned |= rc == B.MD_W_BUDGET_INFEASIBLE
        self.status_seen |= dev_status
        assert dev_status == 0, f"step {k}: device status {dev_status:#x}"
        if not self.select_compact:
            host = snapshot()
        abar = self.abar.cpu().numpy()
        tsc = self.tscore.cpu().numpy()
        psc = md.page_score.cpu().numpy()
        ev_ser = md.evict_serial.cpu().numpy()
        ev_cnt = md.evict_count.cpu().numpy()
        infeas = md.infeasible.cpu().numpy()
        final_ser = ev_ser.copy()
        final_cnt = ev_cnt.copy()
        same_selection = True   # every compared session's selection equals the oracle's
        tref_fix = []
        quant_before = {s: {p.serial for p in self.oracles[s].pages if p.quant}
                        for s in self.oracle_sessions} if w.quant_threshold > 0 else {}
        recs = self.oracle_step({s: (qo[s], nko[s], int(reg[s])) for s in self.oracle_sessions})
        for s in self.oracle_sessions:
            rec = recs[s]
            self.last_rec[s] = rec
            if not compare:
                continue
            npg, nt = int(host["n_pages"][s]), int(host["n_live"][s])
            assert nt == rec.n_select, (k, s, nt, rec.n_select)
            ptab = host["page_table"][s, :npg].astype(np.int64)
            pser = host["page_serial"][s, :npg]
            assert pser.tolist() == rec.page_serial.tolist(), (k, s)
            slots = self.token_slots(host, s)
            assert slots.size == nt, (k, s, "tokens in the page tables", slots.size, nt)
            dev_sizes = np.bincount(slots // P, minlength=c.n_phys)[ptab] if npg else np.zeros(0, np.int64)
            assert dev_sizes.tolist() == rec.page_size.tolist(), (k, s, "tokens per page")
            st = self.stats
            st.tokens += nt
            # attention mass and importance
            e = rel_err(abar[slots], rec.abar)
            st.bump("abar", e)
            assert np.all(e <= REL), (k, s, "abar", float(e.max()), int(np.argmax(e)))
            e = rel_err(host["importance"].reshape(-1)[slots], rec.a)
            st.bump("a", e)
            assert np.all(e <= REL), (k, s, "a", float(e.max()))
            # refresh decisions
            band = np.abs(rec.abar - rec.tau) <= REL * rec.tau
            tref_g = host["t_ref"].reshape(-1)[slots]
            mism = tref_g != rec.t_ref
            assert not np.any(mism & ~band), (k, s, "t_ref", np.flatnonzero(mism & ~band)[:5])
            exc = mism & band
            st.tau_excused += int(exc.sum())
            if exc.any():
                tref_fix.append((slots[exc], rec.t_ref[exc]))
            # token scores
            gs = tsc[slots]
            pin = np.isinf(rec.score)
            assert np.array_equal(np.isinf(gs), pin), (k, s, "pinned tokens")
            ok = ~pin & ~exc
            e = rel_err(gs[ok], rec.score[ok])
            st.bump("score", e)
            assert np.all(e <= REL), (k, s, "score", float(e.max()) if e.size else 0)
            # page scores
            gp = psc[s, :npg]
            assert np.array_equal(np.isinf(gp), rec.page_pinned), (k, s, "pinned pages")
            page_of = np.repeat(np.arange(npg), rec.page_size)
            exc_pages = np.zeros(npg, bool)
            exc_pages[page_of[exc]] = True
            okp = ~rec.page_pinned & ~exc_pages
            e = rel_err(gp[okp], rec.page_score[okp])
            st.bump("page", e)
            assert np.all(e <= REL), (k, s, "page score", float(e.max()) if e.size else 0)
            # eviction
            g_ev = ev_ser[s, :ev_cnt[s]]
            assert np.all(np.diff(g_ev) > 0), (k, s, "evicted serials ascend")
            assert bool(infeas[s]) == rec.infeasible, (k, s, "infeasible")
            check_selection_prefix(gp, pser, rec.page_size, np.isinf(gp), nt, int(self.B[s]), P,
                                   g_ev, bool(infeas[s]))
            if self.strict_ties:
                assert g_ev.tolist() == rec.evicted.tolist(), (k, s, "evicted serials (exact ties)")
            if g_ev.tolist() != rec.evicted.tolist():
                same_selection = False
                diff = set(g_ev.tolist()) ^ set(rec.evicted.tolist())
                thr = max((rec.page_score[i] for i in range(npg)
                           if rec.page_serial[i] in set(rec.evicted.tolist())), default=0.0)
                for ser_ in diff:
                    i = int(np.flatnonzero(rec.page_serial == ser_)[0])
                    near = abs(rec.page_score[i] - thr) <= REL * max(thr, ABS)
                    assert near or exc_pages[i], (k, s, "eviction differs outside the tie band",
                                                  ser_, rec.page_score[i], thr)
                st.tie_excused += len(diff)
            st.evicted_pages += len(rec.evicted)
            if self.offload_pages:
                self.check_offloaded_observation(s, rec)
            final_ser[s, :] = 0
            final_ser[s, :len(rec.evicted)] = rec.evicted
            final_cnt[s] = len(rec.evicted)
        for slots_, vals in tref_fix:
            c.t_ref.view(-1)[torch.from_numpy(slots_).to(self.dev)] = \
                torch.from_numpy(vals.astype(np.int32)).to(self.dev)
        if self.select_compact:
            assert same_selection, (k, "the one-call form applied a selection other than the oracle's")
        elif self.check_free_list:
            pre_compact = self.free_list_state()
        if self.select_compact:
            pass   # applied already
        elif same_selection and not self.explicit_lists:
            # the device's own selection: md_compact without lists (the path
            # a caller takes)
            md.compact()
        else:
            md.compact(torch.from_numpy(final_ser).to(self.dev), torch.from_numpy(final_cnt).to(self.dev))
        torch.cuda.synchronize(self.dev)
        if self.check_free_list:
            self.check_pushes(pre_compact, final_ser, final_cnt, self.free_list_state())
        if compare:
            n_pages = c.n_pages.cpu().numpy()
            n_tokens = self.live_counts()
            pser = c.page_serial.cpu().numpy()
            for s in self.oracle_sessions:
                rec = recs[s]
                gone = set(rec.evicted.tolist())
                assert int(n_tokens[s]) == rec.n_after, (k, s, "n after compaction")
                assert pser[s, :n_pages[s]].tolist() == [x for x in rec.page_serial.tolist() if x not in gone], (k, s)
                if w.quant_threshold > 0:
                    self.check_quantised(s, quant_before[s])
                if self.offload_pages:
                    self.check_offloaded_after(s, rec)
        self.stats.steps += 1
        return self.stats

    # -------------------------------------------------------------- offload tier
    def off_list(self, s: int):
        c = self.cache
        n = int(c.off_count[s].item())
        return c.off_serial[s, :n].cpu().numpy(), c.off_slot[s, :n].cpu().numpy()

    def check_offloaded_observation(self, s: int, rec):
        """After the observation: the pages in host memory (recalled ones
        gone), their tokens' mass, importance and refresh clock, and their
        page scores, against the oracle's."""
        c, P, k = self.cache, self.w.P, self.k
        ser, slot = self.off_list(s)
        assert ser.tolist() == rec.off_serial.tolist(), (k, s, "pages in host memory", ser, rec.off_serial)
        if not ser.size:
            return
        st = self.stats
        abar = c.off_abar[s].cpu().numpy()[slot].reshape(-1)
        e = rel_err(abar, rec.off_abar)
        st.bump("abar", e)
        assert np.all(e <= REL), (k, s, "host-memory abar", float(e.max()))
        a = c.off_importance[s].cpu().numpy()[slot].reshape(-1)
        e = rel_err(a, rec.off_a)
        st.bump("a", e)
        assert np.all(e <= REL), (k, s, "host-memory importance", float(e.max()))
        tref = c.off_t_ref[s].cpu().numpy()[slot].reshape(-1)
        assert np.array_equal(tref, rec.off_t_ref), (k, s, "host-memory refresh clocks")
        ps = c.off_score[s, :ser.size].cpu().numpy()
        e = rel_err(ps, rec.off_page_score)
        st.bump("page", e)
        assert np.all(e <= REL), (k, s, "host-memory page scores", float(e.max()))

    def check_offloaded_after(self, s: int, rec):
        """After the compaction: the pages in host memory, and the keys of
        those moved there this step, bit for bit."""
        c, w = self.cache, self.w
        ser, slot = self.off_list(s)
        assert ser.tolist() == rec.off_after.tolist(), (self.k, s, "host memory after", ser, rec.off_after)
        self.stats.offloaded += len(rec.offloaded_now)
        self.stats.recalled += len(rec.recalled)
        self.stats.dropped += len(rec.dropped)
        o = self.oracles.get(s)
        if o is None or not rec.offloaded_now.size:
            return
        pages = {p.serial: p for p in o.offloaded}
        for x in rec.offloaded_now.tolist():
            p = pages[x]
            if p.quant:
                continue
            j = int(slot[int(np.flatnonzero(ser == x)[0])])
            keys = np.asarray(o.keys[:, :, p.slots, :]).transpose(2, 0, 1, 3)          # [P][L][Hkv][d]
            want = PagedCache.to_pool_layout(torch.from_numpy(keys.astype(np.int16)).view(1, w.P, w.L, w.Hkv, w.d))
            got = c.host_keys[s, j].view(torch.int16)
            assert torch.equal(got, want.reshape(-1)), (self.k, s, x, "keys in host memory")

    def check_quantised(self, s: int, before):
        """Quantised tier: the device's page formats equal the oracle's, and
        the codes and scales of the pages quantised this step are bit-exact
        (decoded from the pool with the byte layout memdecay.h gives)."""
        c, o, P, w = self.cache, self.oracles[s], self.w.P, self.w
        npg = int(c.n_pages[s].item())
        ptab = c.page_table[s, :npg].cpu().numpy().astype(np.int64)
        fmt = c.page_format.cpu().numpy()[ptab]
        assert fmt.tolist() == [int(p.quant) for p in o.pages], (self.k, s, "page formats")
        t_ = np.arange(16)[:, None]
        e_ = np.arange(w.d)[None, :]
        off = 1024 * (e_ // 64) + 16 * (t_ + 16 * ((e_ // 8) % 4)) + 8 * ((e_ // 32) % 2) + e_ % 8   # [16][d]
        for i, p in enumerate(o.pages):
            if not p.quant or p.serial in before:
                continue
            raw = c.k_pool[int(ptab[i])].contiguous().view(torch.uint8).view(w.L, w.Hkv, P // 16, 4096).cpu().numpy()
            slots = np.asarray(p.slots, np.int64)
            for g0 in range(0, slots.size, 16):
                grp = slots[g0:g0 + 16]
                blk = raw[:, :, g0 // 16]                                        # [L][Hkv][4096]
                codes = blk[:, :, off].view(np.int8)[:, :, :grp.size]            # [L][Hkv][tokens][d]
                scale = blk[:, :, 2048:2052].copy().view(np.float32)[:, :, 0]    # [L][Hkv]
                want_c = o.codes[:, :, grp].astype(np.int8)                      # [L][Hkv][tokens][d]
                want_s = o.qscale[:, :, grp[0]]
                assert np.array_equal(codes, want_c), (self.k, s, p.serial, "codes")
                assert np.array_equal(scale.view(np.uint32), want_s.astype(np.float32).view(np.uint32)), \
                    (self.k, s, p.serial, "scales")

    def oracle_step(self, inputs):
        """One oracle step of the given sessions: {s: (q, new_key_bits,
        new_region)} -> {s: StepRecord}."""
        if self.pool is not None:
            return self.pool.step(inputs)
        return {s: self.oracles[s].step(*inp) for s, inp in inputs.items()}

    def free_list_state(self):
        c = self.cache
        return {"fc": int(c.free_count.item()), "free": c.free_list.cpu().numpy().copy(),
                "np": c.n_pages.cpu().numpy().copy(), "ptab": c.page_table.cpu().numpy().copy(),
                "pser": c.page_serial.cpu().numpy().copy()}

    def check_pops(self, a, b):
        """An append takes pages off the top of the free-list stack in
        session order: the first session that opens a page gets the top
        entry, the next one the entry below, and so on."""
        fc, rank = a["fc"], 0
        for s in range(self.w.S):
            if b["np"][s] == a["np"][s] + 1:
                assert b["ptab"][s, b["np"][s] - 1] == a["free"][fc - 1 - rank], (self.k, s, "pop order")
                rank += 1
            else:
                assert b["np"][s] == a["np"][s], (self.k, s)
        assert b["fc"] == fc - rank, (self.k, "free count after the append", b["fc"], fc, rank)

    def check_pushes(self, a, ev_ser, ev_cnt, b):
        """A compaction pushes the freed physical ids in (session, serial)
        order on top of the free-list stack."""
        want = []
        for s in range(self.w.S):
            ser = a["pser"][s, :a["np"][s]]
            for x in ev_ser[s, :ev_cnt[s]]:
                i = np.flatnonzero(ser == x)
                assert i.size == 1, (self.k, s, int(x))
                want.append(int(a["ptab"][s, i[0]]))
        fc = a["fc"]
        assert b["fc"] == fc + len(want), (self.k, "free count after the compaction")
        assert b["free"][fc:fc + len(want)].tolist() == want, (self.k, "push order")
        assert np.array_equal(b["free"][:fc], a["free"][:fc]), (self.k, "entries below untouched")

    def live_counts(self) -> np.ndarray:
        """|K_t| per session on the device: n_live with region-aligned pages."""
        c = self.cache
        return (c.n_live if self.w.region_aligned else c.n_tokens).cpu().numpy()

    def token_slots(self, host, s: int) -> np.ndarray:
        """Slots of session s's tokens in logical order, read from the device's
        page table, counters and region codes (holes left out)."""
        P = self.w.P
        npg, npos = int(host["n_pages"][s]), int(host["n_tokens"][s])
        ptab = host["page_table"][s, :npg].astype(np.int64)
        slots = (ptab[:, None] * P + np.arange(P)[None, :]).reshape(-1)[:npos]
        if self.w.region_aligned:
            slots = slots[host["region"].reshape(-1)[slots] != B.MD_REGION_HOLE]
        return slots

    def device_status(self) -> int:
        return self.md.device_status() | self.status_seen

    def free_pages_consistent(self) -> bool:
        """Live pages plus free pages account for every physical page."""
        c = self.cache
        npg = c.n_pages.cpu().numpy()
        live = np.concatenate([c.page_table[s, :npg[s]].cpu().numpy() for s in range(c.S)] +
                              [np.zeros(0, np.int32)])
        fc = int(c.free_count.item())
        free = c.free_list[:fc].cpu().numpy()
        allp = np.concatenate([live, free])
        return allp.size == c.n_phys and np.unique(allp).size == c.n_phys

    def close(self):
        self.md.close()
        if self.pool is not None:
            self.pool.close()
            self.pool = None
