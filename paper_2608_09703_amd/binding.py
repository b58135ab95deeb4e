"""ctypes binding of ``libmls.so`` (C ABI in ``include/mls.h``).

Argument marshalling only: every step of the loss runs in the library's HIP
kernels. PyTorch provides device memory and the current stream. The library
must have been built (``python -m paper_2608_09703_amd.build_lib``); loading
fails loudly otherwise.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

PKG = os.path.dirname(os.path.abspath(__file__))
# MLS_LIBRARY selects another build of the same library (e.g. the host-sanitized
# copy for CPU-only host tests); by default the in-tree libmls.so.
LIB_PATH = os.environ.get("MLS_LIBRARY") or os.path.join(PKG, "libmls.so")

MAX_MODELS = 8

MLS_OK = 0
MLS_INVALID_ARG = 1
MLS_UNSUPPORTED = 2
MLS_WORKSPACE_TOO_SMALL = 3
MLS_HIP_ERROR = 4

MLS_BF16 = 0
MLS_F32 = 1

MLS_MODE_PAPER = 0
MLS_MODE_ADDITIVE = 1

MLS_JUNCTION_PREV_FIRST = 0
MLS_JUNCTION_FRESH_FIRST = 1
MLS_JUNCTION_ACCUMULATE = 1

MLS_ACCUMULATE_GRAD_W = 1
MLS_ACCUMULATE_GRAD_H = 2
MLS_FWD_BWD_RECOMPUTE = 4

MLS_DEVFLAG_LABEL_RANGE = 1
MLS_DEVFLAG_NONFINITE = 2

EXPORTED = (
    "mls_query_sizes",
    "mls_distill_fwd",
    "mls_distill_bwd",
    "mls_query_fwd_bwd_workspace",
    "mls_distill_fwd_bwd",
    "mls_diagnostics",
    "mls_junction_fwd",
    "mls_junction_bwd",
    "mls_head_logits",
    "mls_sample",
    "mls_spec_verify_workspace",
    "mls_spec_verify",
    "mls_spec_verify_noalloc",
    "mls_coeffs",
    "mls_read_stats_header",
    "mls_device_error",
    "mls_status_string",
    "mls_last_error",
    "mls_version",
    "mls_device_info",
    "mls_profile_enable",
    "mls_profile_report",
    "mls_mfma_probe",
)


class MlsError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status} ({detail})")
        self.status = status


class KernelTime(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", ctypes.c_int32),
                ("total_ms", ctypes.c_double)]


class Problem(ctypes.Structure):
    _fields_ = [
        ("M", ctypes.c_int32),
        ("teacher", ctypes.c_int32),
        ("T", ctypes.c_int64),
        ("V", ctypes.c_int64),
        ("d", ctypes.c_int64 * MAX_MODELS),
        ("h", ctypes.c_void_p * MAX_MODELS),
        ("W", ctypes.c_void_p * MAX_MODELS),
        ("labels", ctypes.c_void_p),
        ("ignore_index", ctypes.c_int64),
        ("alpha", ctypes.c_float),
        ("tau", ctypes.c_float),
        ("in_dtype", ctypes.c_int32),
        ("grad_h_dtype", ctypes.c_int32),
        ("flags", ctypes.c_uint32),
        ("vocab_chunk", ctypes.c_int64),
    ]


class Sampling(ctypes.Structure):
    _fields_ = [
        ("V", ctypes.c_int64),
        ("temperature", ctypes.c_float),
        ("top_p", ctypes.c_float),
        ("greedy", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
    ]


class Junction(ctypes.Structure):
    _fields_ = [
        ("T", ctypes.c_int64),
        ("d_prev", ctypes.c_int64),
        ("d_fresh", ctypes.c_int64),
        ("act_dtype", ctypes.c_int32),
        ("grad_dtype", ctypes.c_int32),
        ("layout", ctypes.c_int32),
        ("flags", ctypes.c_uint32),
    ]


_lib = None


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2608_09703_amd.build_lib`")
        L = ctypes.CDLL(LIB_PATH)
        vp = ctypes.c_void_p
        P = ctypes.POINTER(Problem)
        fp = ctypes.POINTER(ctypes.c_float)
        L.mls_query_sizes.argtypes = [P, ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_size_t)]
        L.mls_distill_fwd.argtypes = [P, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
        L.mls_distill_bwd.argtypes = [P, vp, vp, vp, ctypes.POINTER(vp), ctypes.POINTER(vp), vp,
                                      ctypes.c_size_t, vp]
        L.mls_query_fwd_bwd_workspace.argtypes = [P, ctypes.POINTER(ctypes.c_size_t)]
        L.mls_distill_fwd_bwd.argtypes = [P, vp, vp, vp, vp, vp, vp, ctypes.POINTER(vp),
                                          ctypes.POINTER(vp), vp, ctypes.c_size_t, vp]
        L.mls_diagnostics.argtypes = [P, vp, vp, vp, vp, ctypes.c_size_t, vp]
        J = ctypes.POINTER(Junction)
        L.mls_junction_fwd.argtypes = [J, vp, vp, vp, vp]
        L.mls_junction_bwd.argtypes = [J, vp, vp, vp, vp, vp, vp]
        S = ctypes.POINTER(Sampling)
        L.mls_head_logits.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                      vp, vp, vp, vp]
        L.mls_sample.argtypes = [S, ctypes.c_int64, vp, vp, vp, vp, vp]
        L.mls_spec_verify_workspace.argtypes = [ctypes.c_int64, ctypes.c_int64,
                                                ctypes.POINTER(ctypes.c_size_t)]
        L.mls_spec_verify.argtypes = [S, ctypes.c_int64, ctypes.c_int64, vp, vp, vp, vp, vp, vp, vp,
                                      vp, vp, ctypes.c_size_t, vp]
        L.mls_spec_verify_noalloc.argtypes = [S, ctypes.c_int64, ctypes.c_int64, vp, vp, vp, vp,
                                              vp, vp, vp, vp, vp]
        L.mls_coeffs.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_float, ctypes.c_float,
                                 ctypes.c_int32, fp, fp, fp]
        L.mls_read_stats_header.argtypes = [P, vp, vp, ctypes.POINTER(ctypes.c_int32),
                                            ctypes.POINTER(ctypes.c_int32)]
        L.mls_device_error.argtypes = [P, vp, vp, ctypes.POINTER(ctypes.c_int32)]
        L.mls_status_string.argtypes = [ctypes.c_int]
        L.mls_status_string.restype = ctypes.c_char_p
        L.mls_last_error.argtypes = []
        L.mls_last_error.restype = ctypes.c_char_p
        L.mls_version.argtypes = []
        L.mls_version.restype = ctypes.c_char_p
        ip = ctypes.POINTER(ctypes.c_int32)
        L.mls_device_info.argtypes = [ip, ip, ip, ip]
        L.mls_mfma_probe.argtypes = [ctypes.c_int32, ctypes.c_int32, vp, ctypes.c_size_t,
                                     ctypes.POINTER(ctypes.c_double), vp]
        L.mls_profile_enable.argtypes = [ctypes.c_int32]
        L.mls_profile_report.argtypes = [ctypes.POINTER(KernelTime), ctypes.c_int32,
                                         ctypes.POINTER(ctypes.c_int32)]
        for name in ("mls_query_sizes", "mls_distill_fwd", "mls_distill_bwd", "mls_coeffs",
                     "mls_read_stats_header", "mls_device_error", "mls_profile_enable",
                     "mls_profile_report"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def check(status: int, where: str):
    if status != MLS_OK:
        L = lib()
        detail = L.mls_last_error().decode() or L.mls_status_string(status).decode()
        raise MlsError(status, where, detail)


def make_problem(M: int, T: int, V: int, dims: Sequence[int], h_ptrs: Sequence[int],
                 W_ptrs: Sequence[int], labels_ptr: int, *, dtype: int = MLS_BF16,
                 teacher: int = -1, ignore_index: int = -100, alpha: float = 0.0,
                 tau: float = 1.0, flags: int = 0, vocab_chunk: int = 0,
                 grad_h_dtype: int = MLS_F32) -> Problem:
    p = Problem()
    p.M = M
    p.teacher = teacher
    p.T = T
    p.V = V
    for i in range(M):
        p.d[i] = int(dims[i])
        p.h[i] = h_ptrs[i]
        p.W[i] = W_ptrs[i]
    p.labels = labels_ptr
    p.ignore_index = ignore_index
    p.alpha = alpha
    p.tau = tau
    p.in_dtype = dtype
    p.grad_h_dtype = grad_h_dtype
    p.flags = flags
    p.vocab_chunk = vocab_chunk
    return p


def query_sizes(p: Problem):
    ws = ctypes.c_size_t(0)
    st = ctypes.c_size_t(0)
    check(lib().mls_query_sizes(ctypes.byref(p), ctypes.byref(ws), ctypes.byref(st)),
          "mls_query_sizes")
    return ws.value, st.value


def distill_fwd(p: Problem, stats: int, ce: int, kl: int, entropy: Optional[int], ws: int,
                ws_bytes: int, stream: int):
    check(lib().mls_distill_fwd(ctypes.byref(p), stats, ce, kl, entropy, ws, ws_bytes, stream),
          "mls_distill_fwd")


def distill_bwd(p: Problem, stats: int, g_ce: Optional[int], g_kl: Optional[int],
                grad_h: Sequence[Optional[int]], grad_W: Sequence[Optional[int]], ws: int,
                ws_bytes: int, stream: int):
    arr_h = (ctypes.c_void_p * MAX_MODELS)(*[x or None for x in grad_h])
    arr_W = (ctypes.c_void_p * MAX_MODELS)(*[x or None for x in grad_W])
    check(lib().mls_distill_bwd(ctypes.byref(p), stats, g_ce, g_kl, arr_h, arr_W, ws, ws_bytes,
                                stream), "mls_distill_bwd")


def query_fwd_bwd_workspace(p: Problem) -> int:
    n = ctypes.c_size_t(0)
    check(lib().mls_query_fwd_bwd_workspace(ctypes.byref(p), ctypes.byref(n)),
          "mls_query_fwd_bwd_workspace")
    return n.value


def distill_fwd_bwd(p: Problem, stats: int, ce: int, kl: int, entropy: Optional[int],
                    g_ce: Optional[int], g_kl: Optional[int], grad_h: Sequence[Optional[int]],
                    grad_W: Sequence[Optional[int]], ws: int, ws_bytes: int, stream: int):
    arr_h = (ctypes.c_void_p * MAX_MODELS)(*[x or None for x in grad_h])
    arr_W = (ctypes.c_void_p * MAX_MODELS)(*[x or None for x in grad_W])
    check(lib().mls_distill_fwd_bwd(ctypes.byref(p), stats, ce, kl, entropy, g_ce, g_kl, arr_h,
                                    arr_W, ws, ws_bytes, stream), "mls_distill_fwd_bwd")


def diagnostics(p: Problem, kl_pair: int, agree: int, argmax: Optional[int], ws: int,
                ws_bytes: int, stream: int):
    check(lib().mls_diagnostics(ctypes.byref(p), kl_pair, agree, argmax, ws, ws_bytes, stream),
          "mls_diagnostics")


def make_junction(T: int, d_prev: int, d_fresh: int, act_dtype: int = MLS_BF16,
                  grad_dtype: int = MLS_F32, layout: int = MLS_JUNCTION_PREV_FIRST,
                  flags: int = 0) -> Junction:
    j = Junction()
    j.T, j.d_prev, j.d_fresh = T, d_prev, d_fresh
    j.act_dtype, j.grad_dtype, j.layout, j.flags = act_dtype, grad_dtype, layout, flags
    return j


def junction_fwd(j: Junction, o: int, e: int, x: int, stream: int):
    check(lib().mls_junction_fwd(ctypes.byref(j), o, e, x, stream), "mls_junction_fwd")


def junction_bwd(j: Junction, o: int, e: int, g_x: int, g_o: int, g_e: int, stream: int):
    check(lib().mls_junction_bwd(ctypes.byref(j), o, e, g_x, g_o, g_e, stream), "mls_junction_bwd")


def make_sampling(V: int, temperature: float = 1.0, top_p: float = 1.0,
                  greedy: bool = False) -> Sampling:
    s = Sampling()
    s.V, s.temperature, s.top_p, s.greedy, s.reserved = V, temperature, top_p, int(bool(greedy)), 0
    return s


def head_logits(T: int, V: int, d: int, dtype: int, o: int, W: int, logits: int, stream: int):
    check(lib().mls_head_logits(T, V, d, dtype, o, W, logits, stream), "mls_head_logits")


ROW_PARAMS_BYTES = 20  # MLS_ROW_PARAMS_BYTES


def sample(s: Sampling, rows: int, logits: int, u: Optional[int], tokens: int, stream: int,
           params: Optional[int] = None):
    check(lib().mls_sample(ctypes.byref(s), rows, logits, u, tokens, params, stream), "mls_sample")


def spec_verify_workspace(batch: int, gamma: int) -> int:
    n = ctypes.c_size_t(0)
    check(lib().mls_spec_verify_workspace(batch, gamma, ctypes.byref(n)), "mls_spec_verify_workspace")
    return n.value


def spec_verify(s: Sampling, batch: int, gamma: int, draft_logits: Optional[int],
                target_logits: int, draft_tokens: Optional[int], u_accept: Optional[int],
                u_sample: Optional[int], n_accepted: int, next_token: int, ws: Optional[int],
                ws_bytes: int, stream: int, draft_params: Optional[int] = None):
    check(lib().mls_spec_verify(ctypes.byref(s), batch, gamma, draft_logits, target_logits,
                                draft_tokens, u_accept, u_sample, draft_params, n_accepted,
                                next_token, ws, ws_bytes, stream), "mls_spec_verify")


SPEC_VERIFY_STATIC_BYTES = 2 << 20  # MLS_SPEC_VERIFY_STATIC_BYTES


def spec_verify_noalloc(s: Sampling, batch: int, gamma: int, draft_logits: Optional[int],
                        target_logits: int, draft_tokens: Optional[int], u_accept: Optional[int],
                        u_sample: Optional[int], n_accepted: int, next_token: int, stream: int,
                        draft_params: Optional[int] = None):
    """mls_spec_verify with the library's static per-device scratch (no workspace)."""
    check(lib().mls_spec_verify_noalloc(ctypes.byref(s), batch, gamma, draft_logits, target_logits,
                                        draft_tokens, u_accept, u_sample, draft_params,
                                        n_accepted, next_token, stream),
          "mls_spec_verify_noalloc")


def coeffs(M: int, teacher: int = -1, alpha: float = 0.0, tau: float = 1.0,
           mode: int = MLS_MODE_PAPER, w: Optional[Sequence[float]] = None):
    FA = ctypes.c_float * MAX_MODELS
    g_ce = FA()
    g_kl = FA()
    wa = FA(*w) if w is not None else None
    check(lib().mls_coeffs(M, teacher, alpha, tau, mode, wa, g_ce, g_kl), "mls_coeffs")
    return list(g_ce)[:M], list(g_kl)[:M]


def device_info():
    """``(compute_units, clock_khz, mem_clock_khz, mem_bus_bits)`` of the current device."""
    v = [ctypes.c_int32(0) for _ in range(4)]
    check(lib().mls_device_info(*[ctypes.byref(x) for x in v]), "mls_device_info")
    return tuple(x.value for x in v)


def read_stats_header(p: Problem, stats: int, stream: int):
    n = ctypes.c_int32(0)
    f = ctypes.c_int32(0)
    check(lib().mls_read_stats_header(ctypes.byref(p), stats, stream, ctypes.byref(n),
                                      ctypes.byref(f)), "mls_read_stats_header")
    return n.value, f.value


def device_error(p: Problem, stats: int, stream: int) -> int:
    """OR of the MLS_DEVFLAG_* bits the last forward on ``stats`` raised (waits for the stream)."""
    f = ctypes.c_int32(0)
    check(lib().mls_device_error(ctypes.byref(p), stats, stream, ctypes.byref(f)), "mls_device_error")
    return f.value


MFMA_PROBE_SINK_FLOATS = 524288


def mfma_probe(random_operands: bool, iters: int, sink: Optional[int], sink_floats: int,
               stream: Optional[int]) -> float:
    """Enqueues the MFMA ceiling probe (or, with sink None, only sizes it); returns its FLOPs."""
    f = ctypes.c_double(0.0)
    check(lib().mls_mfma_probe(1 if random_operands else 0, iters, sink, sink_floats,
                               ctypes.byref(f), stream), "mls_mfma_probe")
    return f.value


def profile_enable(on: bool = True):
    check(lib().mls_profile_enable(1 if on else 0), "mls_profile_enable")


def profile_report():
    """{kernel name: (launches, total_ms)} since the last report (waits for the events)."""
    arr = (KernelTime * 32)()
    n = ctypes.c_int32(0)
    check(lib().mls_profile_report(arr, 32, ctypes.byref(n)), "mls_profile_report")
    return {arr[k].name.decode(): (arr[k].launches, arr[k].total_ms) for k in range(min(n.value, 32))}


def version() -> str:
    return lib().mls_version().decode()
