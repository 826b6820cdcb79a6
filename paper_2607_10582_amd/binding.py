"""ctypes binding of libmemdecay.so: the C ABI's entry points under the same
names, argument marshalling only.  Every step of the retention path runs in
the library's HIP kernels; there is no fallback.  If the library is missing
the first call raises.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libmemdecay.so")

MD_OK = 0
MD_E_INVALID = -1
MD_E_UNSUPPORTED = -2
MD_E_STEP = -3
MD_E_HIP = -4
MD_E_STATE = -5
MD_E_NOMEM = -6
MD_E_TOO_LARGE = -7
MD_W_BUDGET_INFEASIBLE = 1

MD_DEV_CAPACITY = 0x1
MD_DEV_NONFINITE = 0x2
MD_DEV_BAD_EVICT = 0x4
MD_DEV_CORRUPT = 0x8
MD_DEV_TIMEOUT = 0x10

MD_FLAG_NO_FUSED = 0x1
MD_FLAG_FUSED = 0x2
MD_FLAG_NORM_ATTENTION = 0x4
MD_FLAG_REGION_ALIGNED = 0x8
MD_FLAG_COOPERATIVE = 0x10
MD_FLAG_NO_ROW_GROUPS = 0x20
MD_REGION_HOLE = 0xFF

EXPORTS = ("md_abi_version", "md_status_str", "md_init", "md_init_static", "md_observe_step",
           "md_score_pages", "md_select_evict", "md_compact", "md_select_compact", "md_read_device_status",
           "md_profile_enable", "md_profile_read", "md_read_counters", "md_kernel_config",
           "md_calib_accumulate", "md_calib_fit",
           "md_destroy")

# kernel ids of md_profile_enable / md_profile_read
KERNELS = ("append", "logits", "rowstats", "mass", "score", "select", "compact", "attend", "evict")
(MD_K_APPEND, MD_K_LOGITS, MD_K_ROWSTATS, MD_K_MASS, MD_K_SCORE, MD_K_SELECT, MD_K_COMPACT,
 MD_K_ATTEND, MD_K_EVICT) = range(9)


class md_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("max_sessions", ctypes.c_int32),
                ("max_pages", ctypes.c_int32), ("n_phys_pages", ctypes.c_int32),
                ("n_regions", ctypes.c_int32), ("pinned_region_mask", ctypes.c_uint32),
                ("rho", ctypes.c_float), ("alpha", ctypes.c_float),
                ("tau_scale", ctypes.c_float), ("flags", ctypes.c_int32), ("window", ctypes.c_int32),
                ("quant_threshold", ctypes.c_float), ("offload_pages", ctypes.c_int32),
                ("drop_threshold", ctypes.c_float)]


class md_region_params(ctypes.Structure):
    _fields_ = [("base_priority", ctypes.c_void_p), ("decay_rate", ctypes.c_void_p)]


class md_cache_view(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "k_pool", "region", "t_ins", "t_ref", "importance", "page_table", "page_serial",
        "n_pages", "n_tokens", "clock", "next_serial", "budget", "free_list", "free_count", "n_live",
        "page_format", "host_keys", "off_count", "off_serial", "off_slot", "off_region", "off_t_ins",
        "off_t_ref", "off_importance", "off_format", "off_score", "off_abar")]


class MemDecayError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed: {status} ({md_status_str(status)})")


_lib = None


def _start_hip_runtime() -> None:
    """Start the HIP runtime before the library is loaded.

    Loading libmemdecay.so registers its GPU code object, and with it an
    exit handler that unregisters the code object through the HIP runtime.
    Exit handlers run in the reverse order of their registration, so when
    the runtime (and any tool attached to it, such as a profiler, which
    registers its own exit handler when the runtime starts) starts after the
    library is loaded, the runtime's shutdown runs first and the library's
    handler then calls into a runtime that is gone.  Starting the runtime
    first puts the library's handler ahead of the runtime's.  Without a
    device (a build host) the call fails and nothing else happens.
    """
    try:
        hip = ctypes.CDLL("libamdhip64.so", mode=ctypes.RTLD_GLOBAL)
        hip.hipInit.restype = ctypes.c_int
        hip.hipInit.argtypes = [ctypes.c_uint]
        hip.hipInit(0)
    except (OSError, AttributeError):
        pass


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libmemdecay.so (built by paper_2607_10582_amd.build), after
    starting the HIP runtime."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it first "
                           "(python -m paper_2607_10582_amd.build)")
    _start_hip_runtime()
    lib = ctypes.CDLL(path)
    vp, i32 = ctypes.c_void_p, ctypes.c_int32
    lib.md_abi_version.restype = i32
    lib.md_abi_version.argtypes = []
    lib.md_status_str.restype = ctypes.c_char_p
    lib.md_status_str.argtypes = [i32]
    lib.md_init.restype = i32
    lib.md_init.argtypes = [ctypes.POINTER(md_config), ctypes.POINTER(md_region_params),
                            ctypes.POINTER(md_cache_view), vp, ctypes.POINTER(vp)]
    lib.md_init_static.restype = i32
    lib.md_init_static.argtypes = [ctypes.POINTER(md_config), ctypes.POINTER(md_region_params),
                                   ctypes.POINTER(md_cache_view), vp, ctypes.POINTER(vp)]
    lib.md_observe_step.restype = i32
    lib.md_observe_step.argtypes = [vp, i32, vp, vp, vp, vp]
    lib.md_score_pages.restype = i32
    lib.md_score_pages.argtypes = [vp, vp, vp]
    lib.md_select_evict.restype = i32
    lib.md_select_evict.argtypes = [vp, vp, vp, vp]
    lib.md_compact.restype = i32
    lib.md_compact.argtypes = [vp, vp, vp]
    lib.md_select_compact.restype = i32
    lib.md_select_compact.argtypes = [vp, vp, vp, vp]
    lib.md_read_device_status.restype = i32
    lib.md_read_device_status.argtypes = [vp, ctypes.POINTER(i32)]
    lib.md_profile_enable.restype = i32
    lib.md_profile_enable.argtypes = [vp, ctypes.c_uint32]
    lib.md_profile_read.restype = i32
    lib.md_profile_read.argtypes = [vp, i32, ctypes.POINTER(ctypes.c_double),
                                    ctypes.POINTER(ctypes.c_int64)]
    lib.md_read_counters.restype = i32
    lib.md_read_counters.argtypes = [vp, ctypes.POINTER(ctypes.c_int64)]
    lib.md_calib_accumulate.restype = i32
    lib.md_calib_accumulate.argtypes = [vp, vp, i32, i32, vp, vp, vp]
    lib.md_calib_fit.restype = i32
    lib.md_calib_fit.argtypes = [vp, vp, vp, i32, i32, i32, vp, vp]
    lib.md_kernel_config.restype = i32
    lib.md_kernel_config.argtypes = [vp, ctypes.POINTER(i32)]
    lib.md_destroy.restype = i32
    lib.md_destroy.argtypes = [vp]
    _lib = lib
    return lib


def _check(fn: str, st: int) -> int:
    if st < 0:
        raise MemDecayError(fn, st)
    return st


def md_abi_version() -> int:
    return load_library().md_abi_version()


def md_status_str(status: int) -> str:
    return load_library().md_status_str(status).decode()


def md_init_raw(cfg: md_config, rp: md_region_params, cv: md_cache_view, stream: int,
                static: bool = False):
    """Returns (status, handle or None) without raising; static=True calls
    md_init_static."""
    h = ctypes.c_void_p()
    fn = load_library().md_init_static if static else load_library().md_init
    st = fn(ctypes.byref(cfg), ctypes.byref(rp), ctypes.byref(cv), ctypes.c_void_p(stream), ctypes.byref(h))
    return st, (h.value if st == MD_OK else None)


def md_init(cfg: md_config, rp: md_region_params, cv: md_cache_view, stream: int) -> int:
    st, h = md_init_raw(cfg, rp, cv, stream)
    _check("md_init", st)
    return h


def md_init_static(cfg: md_config, rp: md_region_params, cv: md_cache_view, stream: int) -> int:
    st, h = md_init_raw(cfg, rp, cv, stream, static=True)
    _check("md_init_static", st)
    return h


def md_observe_step(h: int, step: int, q: int, new_k: int | None, new_region: int | None,
                    abar_out: int | None = None) -> int:
    return _check("md_observe_step", load_library().md_observe_step(
        h, step, q, new_k or None, new_region or None, abar_out or None))


def md_score_pages(h: int, page_score: int | None, token_score: int | None = None) -> int:
    return _check("md_score_pages", load_library().md_score_pages(
        h, page_score or None, token_score or None))


def md_select_evict(h: int, evict_serial: int, evict_count: int, infeasible: int) -> int:
    return _check("md_select_evict", load_library().md_select_evict(
        h, evict_serial, evict_count, infeasible))


def md_compact(h: int, evict_serial: int | None = None, evict_count: int | None = None) -> int:
    """Both lists None: apply this step's selection."""
    return _check("md_compact", load_library().md_compact(h, evict_serial or None, evict_count or None))


def md_select_compact(h: int, evict_serial: int, evict_count: int, infeasible: int) -> int:
    return _check("md_select_compact", load_library().md_select_compact(
        h, evict_serial, evict_count, infeasible))


def md_read_device_status(h: int, with_warning: bool = False):
    """The device status word (cleared by the read); with_warning=True
    returns (return code, status word), the return code being
    MD_W_BUDGET_INFEASIBLE or MD_OK."""
    out = ctypes.c_int32(0)
    rc = _check("md_read_device_status", load_library().md_read_device_status(h, ctypes.byref(out)))
    return (rc, out.value) if with_warning else out.value


def md_profile_enable(h: int, kernel_mask: int) -> int:
    return _check("md_profile_enable", load_library().md_profile_enable(h, kernel_mask))


def md_profile_read(h: int, kernel: int):
    """(total milliseconds, launches) of ``kernel`` since the last read."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check("md_profile_read", load_library().md_profile_read(h, kernel, ctypes.byref(ms),
                                                             ctypes.byref(n)))
    return ms.value, n.value


def md_calib_accumulate(h: int, abar: int, bucket_steps: int, n_buckets: int, mass_fx: int, count: int,
                        age_sum: int) -> int:
    return _check("md_calib_accumulate", load_library().md_calib_accumulate(
        h, abar, bucket_steps, n_buckets, mass_fx, count, age_sum))


def md_calib_fit(mass_fx, count, age_sum):
    """Eq. 6 fit on host numpy uint64 arrays [S][n_regions][n_buckets];
    returns (lambda_hat, log_c) as float64 arrays [n_regions]."""
    import numpy as np
    arrs = [np.ascontiguousarray(x, dtype=np.uint64) for x in (mass_fx, count, age_sum)]
    S, nr, nb = arrs[0].shape
    lam = np.zeros(nr, np.float64)
    logc = np.zeros(nr, np.float64)
    _check("md_calib_fit", load_library().md_calib_fit(
        arrs[0].ctypes.data, arrs[1].ctypes.data, arrs[2].ctypes.data, S, nr, nb,
        lam.ctypes.data, logc.ctypes.data))
    return lam, logc


def md_read_counters(h: int):
    """(tokens scored, steps observed, pages evicted, tokens evicted, pages
    offloaded, recalled, dropped from host memory, host-memory pages
    observed) since md_init."""
    out = (ctypes.c_int64 * 8)()
    _check("md_read_counters", load_library().md_read_counters(h, out))
    return tuple(int(x) for x in out)


def md_kernel_config(h: int) -> dict:
    """How md_init laid out the observation step (fused kernel available,
    sessions that may outgrow it, largest fused unit in tokens, fused
    workgroups, path of the first and of the later observes, and their row
    groups)."""
    out = (ctypes.c_int32 * 8)()
    _check("md_kernel_config", load_library().md_kernel_config(h, out))
    return {"fused": bool(out[0]), "spill": bool(out[1]), "unit_max": int(out[2]), "workgroups": int(out[3]),
            "first_fused": bool(out[4]), "steady_fused": bool(out[5]), "first_row_groups": int(out[6]),
            "steady_row_groups": int(out[7])}


def md_destroy(h: int) -> int:
    return _check("md_destroy", load_library().md_destroy(h))
