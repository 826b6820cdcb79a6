"""The C ABI on the host (no GPU needed): the library loads, exports every
entry point include/memdecay.h declares, its ctypes mirror matches the
header's struct layout, and argument validation rejects bad calls before
any HIP call or launch."""
import ctypes
import os
import re
import subprocess
import tempfile

import numpy as np
import pytest

from paper_2607_10582_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "memdecay.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        from paper_2607_10582_amd.build import build
        build()
    return B.load_library()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:md_status|int32_t|const char\*)\s+(md_[a-z_]+)\s*\(",
                                 text, flags=re.M)))


def test_header_declares_the_entry_points():
    assert declared_functions() == sorted(B.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    nm = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True, text=True)
    syms = set(l.split()[-1] for l in nm.stdout.splitlines() if l.strip())
    for f in declared_functions():
        assert f in syms, f
        assert hasattr(lib, f)


def test_abi_version_and_status_strings(lib):
    assert B.md_abi_version() == 10
    for st in (0, -1, -2, -3, -4, -5, -6):
        assert B.md_status_str(st)
    assert B.md_status_str(12345) == "unknown status"


def test_struct_layout_matches_the_header(lib):
    src = r'''
    #include <stdio.h>
    #include <stddef.h>
    #include "memdecay.h"
    int main(void) {
      printf("%zu %zu %zu %zu %zu %zu %zu\n", sizeof(md_config), offsetof(md_config, rho),
             offsetof(md_config, flags), offsetof(md_config, window),
             offsetof(md_config, quant_threshold), sizeof(md_region_params), sizeof(md_cache_view));
      printf("%zu %zu %zu %zu %zu %zu %zu\n", offsetof(md_cache_view, importance), offsetof(md_cache_view, free_count),
             offsetof(md_cache_view, n_live), offsetof(md_cache_view, page_format),
             offsetof(md_cache_view, host_keys), offsetof(md_cache_view, off_abar),
             offsetof(md_config, drop_threshold));
      return 0; }
    '''
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "layout.c")
        exe = os.path.join(d, "layout")
        open(c, "w").write(src)
        subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), c, "-o", exe], check=True)
        out = subprocess.run([exe], capture_output=True, text=True, check=True).stdout.split()
    got = [ctypes.sizeof(B.md_config), B.md_config.rho.offset, B.md_config.flags.offset,
           B.md_config.window.offset, B.md_config.quant_threshold.offset,
           ctypes.sizeof(B.md_region_params), ctypes.sizeof(B.md_cache_view),
           B.md_cache_view.importance.offset, B.md_cache_view.free_count.offset,
           B.md_cache_view.n_live.offset, B.md_cache_view.page_format.offset,
           B.md_cache_view.host_keys.offset, B.md_cache_view.off_abar.offset, B.md_config.drop_threshold.offset]
    assert [int(x) for x in out] == got


def good_config(**kw):
    c = dict(n_layers=28, n_q_heads=12, n_kv_heads=2, head_dim=128, page_size=16,
             max_sessions=16, max_pages=2100, n_phys_pages=40000, n_regions=7,
             pinned_region_mask=1, rho=0.9, alpha=1.0, tau_scale=2.0, flags=0, window=1)
    c.update(kw)
    return B.md_config(**c)


def fake_view(**kw):
    v = B.md_cache_view()
    for i, (name, _) in enumerate(B.md_cache_view._fields_):
        setattr(v, name, 0x10000 * (i + 1))
    for k, val in kw.items():
        setattr(v, k, val)
    return v


def fake_rp():
    return B.md_region_params(base_priority=0x900000, decay_rate=0x910000)


@pytest.mark.parametrize("kw,expect", [
    (dict(head_dim=64), B.MD_E_UNSUPPORTED),
    (dict(page_size=32), B.MD_E_UNSUPPORTED),
    (dict(page_size=0), B.MD_E_UNSUPPORTED),
    (dict(n_q_heads=13), B.MD_E_INVALID),
    (dict(n_q_heads=34, n_kv_heads=2), B.MD_E_UNSUPPORTED),
    (dict(n_layers=100, n_q_heads=12), B.MD_E_UNSUPPORTED),
    (dict(max_sessions=0), B.MD_E_INVALID),
    (dict(max_sessions=1025), B.MD_E_UNSUPPORTED),
    (dict(max_pages=8193), B.MD_E_UNSUPPORTED),
    (dict(n_phys_pages=0), B.MD_E_INVALID),
    (dict(n_regions=0), B.MD_E_INVALID),
    (dict(n_regions=33), B.MD_E_INVALID),
    (dict(pinned_region_mask=1 << 7), B.MD_E_INVALID),
    (dict(rho=1.0), B.MD_E_INVALID),
    (dict(rho=-0.1), B.MD_E_INVALID),
    (dict(rho=float("nan")), B.MD_E_INVALID),
    (dict(alpha=-1.0), B.MD_E_INVALID),
    (dict(alpha=float("inf")), B.MD_E_INVALID),
    (dict(tau_scale=-2.0), B.MD_E_INVALID),
    (dict(flags=64), B.MD_E_INVALID),
    (dict(window=0), B.MD_E_INVALID),
    (dict(quant_threshold=-1.0), B.MD_E_INVALID),
    (dict(quant_threshold=float("nan")), B.MD_E_INVALID),
    (dict(window=3), B.MD_E_UNSUPPORTED),            # G = 6: 18 MFMA columns
    (dict(flags=3), B.MD_E_INVALID),
    (dict(offload_pages=-1), B.MD_E_INVALID),
    (dict(offload_pages=65), B.MD_E_INVALID),
    (dict(offload_pages=4, drop_threshold=-0.5), B.MD_E_INVALID),
    (dict(offload_pages=4, drop_threshold=float("nan")), B.MD_E_INVALID),
    (dict(offload_pages=4, window=2), B.MD_E_UNSUPPORTED),          # the tier takes one query per observation
    (dict(offload_pages=4, flags=8), B.MD_E_UNSUPPORTED),           # and plain pages
])
def test_init_rejects_bad_configs_on_the_host(lib, kw, expect):
    st, h = B.md_init_raw(good_config(**kw), fake_rp(), fake_view(), 0)
    assert st == expect and h is None


OPTIONAL = ("n_live", "page_format", "host_keys", "off_count", "off_serial", "off_slot", "off_region", "off_t_ins",
            "off_t_ref", "off_importance", "off_format", "off_score", "off_abar")


@pytest.mark.parametrize("field", [f for f, _ in B.md_cache_view._fields_ if f not in OPTIONAL])
def test_init_rejects_null_buffers(lib, field):
    st, h = B.md_init_raw(good_config(), fake_rp(), fake_view(**{field: 0}), 0)
    assert st == B.MD_E_INVALID


@pytest.mark.parametrize("field", ["host_keys", "off_count", "off_serial", "off_slot", "off_region", "off_t_ins",
                                   "off_t_ref", "off_importance", "off_format", "off_score", "off_abar"])
def test_offload_tier_needs_its_buffers(lib, field):
    st, h = B.md_init_raw(good_config(offload_pages=4), fake_rp(), fake_view(**{field: 0}), 0)
    assert st == B.MD_E_INVALID and h is None


def test_quantised_tier_needs_the_page_formats(lib):
    st, h = B.md_init_raw(good_config(quant_threshold=0.5), fake_rp(), fake_view(page_format=0), 0)
    assert st == B.MD_E_INVALID and h is None


@pytest.mark.parametrize("kw", [dict(n_live=0), dict(n_live=0x10002), dict(region=0x10001)])
def test_region_aligned_pages_need_the_token_counts(lib, kw):
    # n_live is required (and word-aligned) with region-aligned pages, and the
    # region codes are read four at a time
    st, h = B.md_init_raw(good_config(flags=B.MD_FLAG_REGION_ALIGNED), fake_rp(), fake_view(**kw), 0)
    assert st == B.MD_E_INVALID and h is None


def test_init_rejects_misaligned_buffers(lib):
    assert B.md_init_raw(good_config(), fake_rp(), fake_view(k_pool=0x10008), 0)[0] == B.MD_E_INVALID
    assert B.md_init_raw(good_config(), fake_rp(), fake_view(t_ref=0x10002), 0)[0] == B.MD_E_INVALID
    rp = B.md_region_params(base_priority=0, decay_rate=0x910000)
    assert B.md_init_raw(good_config(), rp, fake_view(), 0)[0] == B.MD_E_INVALID


def test_calls_reject_a_null_handle(lib):
    L = lib
    assert L.md_observe_step(None, 1, 0x1000, None, None, None) == B.MD_E_INVALID
    assert L.md_score_pages(None, None, None) == B.MD_E_INVALID
    assert L.md_select_evict(None, 0x1000, 0x1000, 0x1000) == B.MD_E_INVALID
    assert L.md_compact(None, 0x1000, 0x1000) == B.MD_E_INVALID
    assert L.md_select_compact(None, 0x1000, 0x1000, 0x1000) == B.MD_E_INVALID
    assert L.md_destroy(None) == B.MD_E_INVALID
    out = ctypes.c_int32()
    assert L.md_read_device_status(None, ctypes.byref(out)) == B.MD_E_INVALID
    assert L.md_init(None, None, None, None, None) == B.MD_E_INVALID


def test_calib_fit_matches_the_oracle_fit(lib):
    # md_calib_fit is host code: count-weighted least squares of Eq. 6 on
    # sums added over sessions, against the oracle's fit of the same sums.
    from oracle.calibration import fit_decay
    rng = np.random.default_rng(5)
    S, nr, nb = 3, 7, 20
    count = rng.integers(0, 60, (S, nr, nb)).astype(np.uint64)
    count[:, 6, 1:] = 0                          # region 6: a single bucket, no fit
    count[:, 6, 0] = 5
    ages = (np.arange(nb) * 8 + 3.5)[None, None, :]
    mean = 0.01 * np.exp(-rng.uniform(0.01, 0.1, (1, nr, 1)) * ages) * np.exp(rng.normal(0, 0.2, (S, nr, nb)))
    mass_fx = np.round(count * mean * 2.0**40).astype(np.uint64)
    age_sum = (count * np.round(ages)).astype(np.uint64)
    lam, logc = B.md_calib_fit(mass_fx, count, age_sum)
    olam, ologc = fit_decay(mass_fx.sum(0).astype(np.float64) / 2.0**40, count.sum(0).astype(np.float64),
                            age_sum.sum(0).astype(np.float64))
    assert np.array_equal(np.isnan(lam), np.isnan(olam)) and np.isnan(lam[6])
    ok = ~np.isnan(olam)
    np.testing.assert_allclose(lam[ok], olam[ok], rtol=1e-9)
    np.testing.assert_allclose(logc[ok], ologc[ok], rtol=1e-9)


def test_pool_layout_matches_the_header():
    # memdecay.h: element (t, e) of a (page, layer, KV head) tile sits at
    # (t & ~15) d + (e / 8) 128 + (t % 16) 8 + e % 8; the caller-side helpers
    # place keys there and read them back
    import torch
    from paper_2607_10582_amd.cache import PagedCache
    m, P, L, Hkv, d = 2, 64, 3, 2, 128
    k = torch.arange(m * P * L * Hkv * d, dtype=torch.float64).view(m, P, L, Hkv, d)
    pool = PagedCache.to_pool_layout(k)
    flat = pool.reshape(m, L, Hkv, P * d)
    for (pg, t, l, kv, e) in [(0, 0, 0, 0, 0), (1, 17, 2, 1, 9), (0, 63, 1, 0, 127), (1, 40, 0, 1, 64)]:
        off = (t & ~15) * d + (e // 8) * 128 + (t % 16) * 8 + e % 8
        assert flat[pg, l, kv, off] == k[pg, t, l, kv, e]
    assert torch.equal(PagedCache.from_pool_layout(pool), k)
