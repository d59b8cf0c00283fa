"""ctypes binding of libflexattn.so (include/flexattn.h).

Argument marshalling only: every step of the attention path runs in the HIP
library. PyTorch supplies device memory and streams. Importing this module
raises if the library has not been built; there is no fallback.

Functions keep the C names (``flex_attn_plan``, ``flex_attn_decode``, ...);
``PagedAttention`` bundles a plan with its device copy and workspace for the
common case of running one batch.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libflexattn.so")

FLEX_OK = 0
FLEX_ERR_INVALID_ARG = -1
FLEX_ERR_UNSUPPORTED = -2
FLEX_ERR_WORKSPACE = -3
FLEX_ERR_HIP = -4
FLEX_ERR_INTERNAL = -5
FLEX_MODE_SERIAL = 0
FLEX_MODE_CORUN = 1
FLEX_MODE_FUSED = 2

EXPORTED = [
    "flex_attn_status_string", "flex_attn_last_error", "flex_attn_plan", "flex_attn_plan_info_get",
    "flex_attn_plan_export", "flex_attn_plan_upload", "flex_attn_plan_destroy", "flex_attn_decode",
    "flex_attn_prefill", "flex_attn_mixed", "flex_attn_corun_create", "flex_attn_corun_destroy",
    "flex_attn_corun_streams", "flex_attn_corun_set_timing", "flex_attn_corun_timing_read",
    "flex_attn_debug_gather", "flex_attn_workspace_init", "flex_attn_kv_append",
    "flex_attn_mixed_static", "flex_attn_static_scratch_bytes", "flex_attn_validate_host", "flex_attn_set_debug",
    "flex_ctl_create", "flex_ctl_destroy", "flex_ctl_set_profile", "flex_ctl_observe", "flex_ctl_decide",
    "flex_ctl_estimates", "flex_ts_create", "flex_ts_destroy", "flex_ts_next", "flex_ts_observe", "flex_ts_totals",
]
FLEX_CTL_ONE_PHASE = 0
FLEX_CTL_BEST = 1
FLEX_CTL_SERIAL_FASTER = 2
FLEX_CTL_BACKLOG = 3
FLEX_CTL_BW_SATURATED = 4
FLEX_CTL_EXPLORE = 5
FLEX_CTL_PREFILL_BACKLOG = 6
FLEX_CTL_FUSED_FASTER = 7
FLEX_TS_DECODE = 0
FLEX_TS_PREFILL = 1
FLEX_TIMING_RING = 1024


class Shape(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim_qk", ctypes.c_int32), ("head_dim_v", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("sm_scale", ctypes.c_float),
                ("v_aliases_k", ctypes.c_int32)]


class PlanOpts(ctypes.Structure):
    _fields_ = [("cus_total", ctypes.c_int32), ("cus_decode", ctypes.c_int32), ("bm", ctypes.c_int32),
                ("min_split_tokens", ctypes.c_int32),
                ("wg_per_cu", ctypes.c_int32), ("split_granule", ctypes.c_int32),
                ("hbm_gbps", ctypes.c_double), ("decode_gbps_per_cu", ctypes.c_double),
                ("prefill_tflops_per_cu", ctypes.c_double), ("decode_tail", ctypes.c_int32)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("n_decode_seqs", ctypes.c_int32),
                ("n_prefill_seqs", ctypes.c_int32), ("n_decode_items", ctypes.c_int32),
                ("n_prefill_items", ctypes.c_int32), ("n_split_seqs", ctypes.c_int32),
                ("decode_wg_width", ctypes.c_int32), ("n_decode_ranges", ctypes.c_int32),
                ("prefill_grid_y", ctypes.c_int32), ("pages_per_split", ctypes.c_int32),
                ("cus_decode", ctypes.c_int32), ("cus_prefill", ctypes.c_int32), ("bm", ctypes.c_int32),
                ("plan_words", ctypes.c_int32), ("device_plan_bytes", ctypes.c_size_t),
                ("workspace_bytes", ctypes.c_size_t), ("decode_bytes", ctypes.c_double),
                ("prefill_flops", ctypes.c_double), ("n_fused_wgs", ctypes.c_int32),
                ("n_decode_tail_ranges", ctypes.c_int32), ("decode_tail_bytes", ctypes.c_double)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class Args(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("k_cache", ctypes.c_void_p), ("v_cache", ctypes.c_void_p),
                ("k_stride", ctypes.c_int64 * 3), ("v_stride", ctypes.c_int64 * 3),
                ("num_pages", ctypes.c_int32), ("block_table", ctypes.c_void_p),
                ("block_table_stride", ctypes.c_int32), ("seq_lens", ctypes.c_void_p),
                ("query_start_loc", ctypes.c_void_p), ("out", ctypes.c_void_p), ("lse", ctypes.c_void_p),
                ("d_plan", ctypes.c_void_p), ("d_plan_bytes", ctypes.c_size_t),
                ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t)]


class AppendArgs(ctypes.Structure):
    _fields_ = [("k_new", ctypes.c_void_p), ("v_new", ctypes.c_void_p), ("k_new_stride", ctypes.c_int64),
                ("v_new_stride", ctypes.c_int64), ("slot_mapping", ctypes.c_void_p), ("n_tokens", ctypes.c_int64),
                ("k_cache", ctypes.c_void_p), ("k_stride", ctypes.c_int64 * 3), ("v_cache", ctypes.c_void_p),
                ("v_stride", ctypes.c_int64 * 3), ("num_pages", ctypes.c_int64), ("bad_count", ctypes.c_void_p)]


class CtlOpts(ctypes.Structure):
    _fields_ = [("cus_total", ctypes.c_int32), ("granule", ctypes.c_int32), ("explore_every", ctypes.c_int32),
                ("backlog_seqs", ctypes.c_int32), ("backlog_prefill_tokens", ctypes.c_int32),
                ("alpha", ctypes.c_double), ("tolerance", ctypes.c_double), ("sat_frac", ctypes.c_double),
                ("hbm_gbps", ctypes.c_double), ("corun_overhead_us", ctypes.c_double),
                ("decode_gbps_per_cu", ctypes.c_double), ("prefill_tflops_per_cu", ctypes.c_double),
                ("fused_prior", ctypes.c_double)]


class CtlSignals(ctypes.Structure):
    _fields_ = [("decode_bytes", ctypes.c_double), ("prefill_flops", ctypes.c_double),
                ("pending_prefill_tokens", ctypes.c_int32), ("pending_decode_seqs", ctypes.c_int32),
                ("active_decode_seqs", ctypes.c_int32), ("fused_available", ctypes.c_int32),
                ("decode_tail", ctypes.c_int32)]


class CtlObservation(ctypes.Structure):
    _fields_ = [("cus_decode", ctypes.c_int32), ("decode_bytes", ctypes.c_double),
                ("prefill_flops", ctypes.c_double), ("decode_ms", ctypes.c_double), ("prefill_ms", ctypes.c_double),
                ("fused", ctypes.c_int32), ("step_ms", ctypes.c_double)]


class CtlDecision(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("cus_decode", ctypes.c_int32), ("cus_prefill", ctypes.c_int32),
                ("reason", ctypes.c_int32), ("predicted_us", ctypes.c_double)]


class TsOpts(ctypes.Structure):
    _fields_ = [("decode_share", ctypes.c_double), ("decay", ctypes.c_double)]


class FlexAttnError(RuntimeError):
    def __init__(self, status: int, what: str, detail: str):
        super().__init__(f"{what}: status {status} ({detail})")
        self.status = status


_lib = None


def lib():
    """Load libflexattn.so (once). Raises if it is missing: there is no fallback."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing; build it with "
                           "`python -m paper_2606_04415_amd.build` (hipcc, gfx950)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    L.flex_attn_status_string.argtypes = [ctypes.c_int]
    L.flex_attn_status_string.restype = ctypes.c_char_p
    L.flex_attn_last_error.argtypes = []
    L.flex_attn_last_error.restype = ctypes.c_char_p
    L.flex_attn_plan.argtypes = [ctypes.POINTER(Shape), ctypes.POINTER(PlanOpts), i32,
                                 ctypes.POINTER(i32), ctypes.POINTER(i32), i32, ctypes.POINTER(vp)]
    L.flex_attn_plan_info_get.argtypes = [vp, ctypes.POINTER(PlanInfo)]
    L.flex_attn_plan_export.argtypes = [vp, ctypes.POINTER(i32), sz]
    L.flex_attn_plan_upload.argtypes = [vp, vp, sz, vp]
    L.flex_attn_plan_destroy.argtypes = [vp]
    L.flex_attn_plan_destroy.restype = None
    for f in ("flex_attn_decode", "flex_attn_prefill"):
        getattr(L, f).argtypes = [vp, ctypes.POINTER(Args), vp]
    L.flex_attn_mixed.argtypes = [vp, ctypes.POINTER(Args), ctypes.c_int, vp, vp]
    L.flex_attn_mixed_static.argtypes = [vp, ctypes.POINTER(Args), ctypes.c_int, vp, vp]
    L.flex_attn_static_scratch_bytes.argtypes = []
    L.flex_attn_static_scratch_bytes.restype = ctypes.c_size_t
    L.flex_attn_validate_host.argtypes = [vp, ctypes.POINTER(i32), i32, i32, ctypes.POINTER(i32), ctypes.POINTER(i32)]
    L.flex_attn_set_debug.argtypes = [ctypes.c_int]
    L.flex_attn_corun_create.argtypes = [i32, i32, ctypes.POINTER(vp)]
    L.flex_attn_corun_destroy.argtypes = [vp]
    L.flex_attn_corun_destroy.restype = None
    L.flex_attn_corun_streams.argtypes = [vp, ctypes.POINTER(vp), ctypes.POINTER(vp)]
    L.flex_attn_corun_set_timing.argtypes = [vp, ctypes.c_int]
    L.flex_attn_corun_timing_read.argtypes = [vp, ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_float),
                                              i32, ctypes.POINTER(i32)]
    L.flex_attn_debug_gather.argtypes = [vp, ctypes.POINTER(Args), i32, i32, vp, vp, vp]
    L.flex_attn_workspace_init.argtypes = [vp, sz, vp]
    L.flex_attn_kv_append.argtypes = [ctypes.POINTER(Shape), ctypes.POINTER(AppendArgs), vp]
    L.flex_ctl_create.argtypes = [ctypes.POINTER(CtlOpts), ctypes.POINTER(vp)]
    L.flex_ctl_destroy.argtypes = [vp]
    L.flex_ctl_destroy.restype = None
    L.flex_ctl_set_profile.argtypes = [vp, i32, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(ctypes.c_double)]
    L.flex_ctl_observe.argtypes = [vp, ctypes.POINTER(CtlObservation)]
    L.flex_ctl_decide.argtypes = [vp, ctypes.POINTER(CtlSignals), ctypes.POINTER(CtlDecision)]
    L.flex_ctl_estimates.argtypes = [vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double), i32]
    L.flex_ts_create.argtypes = [ctypes.POINTER(TsOpts), ctypes.POINTER(vp)]
    L.flex_ts_destroy.argtypes = [vp]
    L.flex_ts_destroy.restype = None
    L.flex_ts_next.argtypes = [vp, i32, i32, ctypes.POINTER(i32)]
    L.flex_ts_observe.argtypes = [vp, i32, ctypes.c_double]
    L.flex_ts_totals.argtypes = [vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
    for f in EXPORTED:
        if f not in ("flex_attn_status_string", "flex_attn_last_error", "flex_attn_plan_destroy",
                     "flex_attn_corun_destroy", "flex_ctl_destroy", "flex_ts_destroy",
                     "flex_attn_static_scratch_bytes"):
            getattr(L, f).restype = ctypes.c_int
    _lib = L
    return L


def status_string(status: int) -> str:
    return lib().flex_attn_status_string(status).decode()


def last_error() -> str:
    return lib().flex_attn_last_error().decode()


def check(status: int, what: str):
    if status != FLEX_OK:
        raise FlexAttnError(status, what, f"{status_string(status)}: {last_error()}")


def _i32_array(values):
    """An int32* argument over values (an int sequence, a numpy array or a CPU
    tensor): a view when they already are contiguous int32, else one
    vectorised conversion (no per-element Python loop). Values outside int32
    raise ValueError. The returned pointer keeps its array alive."""
    import numpy as np
    if hasattr(values, "detach"):   # torch tensor
        values = values.detach().cpu().numpy()
    a = np.asarray(values).reshape(-1)
    if a.dtype != np.int32:
        if a.size and (a.dtype.kind not in "iu" or int(a.min()) < -2 ** 31 or int(a.max()) > 2 ** 31 - 1):
            raise ValueError("expected integers that fit int32")
        a = a.astype(np.int32)
    a = np.ascontiguousarray(a) if a.size else np.zeros(1, dtype=np.int32)
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


class Plan:
    """Owning wrapper of a flex_attn_plan_t*."""

    def __init__(self, handle: int):
        self.handle = ctypes.c_void_p(handle)
        info = PlanInfo()
        check(lib().flex_attn_plan_info_get(self.handle, ctypes.byref(info)), "flex_attn_plan_info_get")
        self.info = info.as_dict()

    def export(self):
        n = self.info["plan_words"]
        buf = (ctypes.c_int32 * n)()
        check(lib().flex_attn_plan_export(self.handle, buf, n), "flex_attn_plan_export")
        return list(buf)

    def close(self):
        if self.handle and self.handle.value:
            lib().flex_attn_plan_destroy(self.handle)
            self.handle = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def make_shape(num_q_heads, num_kv_heads, head_dim_qk, head_dim_v, page_size, sm_scale, v_aliases_k=False):
    return Shape(num_q_heads, num_kv_heads, head_dim_qk, head_dim_v, page_size, float(sm_scale),
                 1 if v_aliases_k else 0)


def make_opts(**kw) -> PlanOpts:
    o = PlanOpts()
    for k, v in kw.items():
        setattr(o, k, v)
    return o


def flex_attn_plan(shape: Shape, opts: Optional[PlanOpts], query_start_loc: Sequence[int],
                   seq_lens: Sequence[int], max_pages_per_seq: int) -> Plan:
    """Host plan (no HIP call). query_start_loc and seq_lens: int sequences,
    numpy arrays or CPU tensors. Raises FlexAttnError with the library's
    status on failure."""
    out = ctypes.c_void_p()
    st = lib().flex_attn_plan(ctypes.byref(shape), ctypes.byref(opts) if opts is not None else None,
                              len(seq_lens), _i32_array(query_start_loc), _i32_array(seq_lens),
                              int(max_pages_per_seq), ctypes.byref(out))
    check(st, "flex_attn_plan")
    return Plan(out.value)


def plan_status(shape: Shape, opts: Optional[PlanOpts], query_start_loc, seq_lens, max_pages_per_seq) -> int:
    """Status code of flex_attn_plan for these inputs (the plan, if any, is freed)."""
    out = ctypes.c_void_p()
    st = lib().flex_attn_plan(ctypes.byref(shape), ctypes.byref(opts) if opts is not None else None,
                              len(seq_lens), _i32_array(query_start_loc), _i32_array(seq_lens),
                              int(max_pages_per_seq), ctypes.byref(out))
    if st == FLEX_OK:
        lib().flex_attn_plan_destroy(out)
    return st


# ------------------------------------------------------- torch adapters ---

def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def current_stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _require(cond, what):
    if not cond:
        raise ValueError(what)


def make_args(q, k_cache, v_cache, block_table, seq_lens, query_start_loc, out, lse=None,
              d_plan=None, workspace=None) -> Args:
    """Args from device tensors (bf16 caches [pages, P, Hkv, d] with unit inner stride).

    Checks what the C side cannot see: dtypes (bf16 q/caches/out, fp32 lse,
    int32 metadata), contiguity of q, out, lse and the metadata rows, a unit
    innermost cache stride, and that every tensor is on one device."""
    import torch
    for name, t in (("q", q), ("k_cache", k_cache), ("out", out)) + ((("v_cache", v_cache),) if v_cache is not None else ()):
        _require(t.dtype == torch.bfloat16, f"{name} must be bfloat16, not {t.dtype}")
    for name, t in (("block_table", block_table), ("seq_lens", seq_lens), ("query_start_loc", query_start_loc)):
        _require(t.dtype == torch.int32, f"{name} must be int32, not {t.dtype}")
    _require(lse is None or lse.dtype == torch.float32, "lse must be float32")
    for name, t in (("q", q), ("out", out), ("seq_lens", seq_lens), ("query_start_loc", query_start_loc)) + \
            ((("lse", lse),) if lse is not None else ()):
        _require(t.is_contiguous(), f"{name} must be contiguous")
    _require(block_table.dim() == 2 and block_table.stride(1) == 1, "block_table must be 2-D with unit column stride")
    for name, t in (("k_cache", k_cache),) + ((("v_cache", v_cache),) if v_cache is not None else ()):
        _require(t.dim() == 4 and t.stride(3) == 1, f"{name} must be [pages, P, Hkv, d] with a unit innermost stride")
    devs = {t.device for t in (q, k_cache, block_table, seq_lens, query_start_loc, out)
            if t is not None}
    _require(len(devs) == 1, f"tensors on several devices: {devs}")
    a = Args()
    a.q = q.data_ptr()
    a.k_cache = k_cache.data_ptr()
    a.v_cache = v_cache.data_ptr() if v_cache is not None else None
    ks = k_cache.stride()
    a.k_stride = (ctypes.c_int64 * 3)(ks[0], ks[1], ks[2])
    vsrc = v_cache if v_cache is not None else k_cache
    vs = vsrc.stride()
    a.v_stride = (ctypes.c_int64 * 3)(vs[0], vs[1], vs[2])
    a.num_pages = k_cache.shape[0]
    a.block_table = block_table.data_ptr()
    a.block_table_stride = block_table.stride(0)
    a.seq_lens = seq_lens.data_ptr()
    a.query_start_loc = query_start_loc.data_ptr()
    a.out = out.data_ptr()
    a.lse = lse.data_ptr() if lse is not None else None
    if d_plan is not None:
        a.d_plan = d_plan.data_ptr()
        a.d_plan_bytes = d_plan.numel() * d_plan.element_size()
    if workspace is not None:
        a.workspace = workspace.data_ptr()
        a.workspace_bytes = workspace.numel() * workspace.element_size()
    return a


def flex_attn_plan_upload(plan: Plan, d_plan, stream=None):
    s = stream if stream is not None else current_stream()
    check(lib().flex_attn_plan_upload(plan.handle, ctypes.c_void_p(d_plan.data_ptr()),
                                      d_plan.numel() * d_plan.element_size(), s), "flex_attn_plan_upload")


def flex_attn_decode(plan: Plan, args: Args, stream=None):
    s = stream if stream is not None else current_stream()
    check(lib().flex_attn_decode(plan.handle, ctypes.byref(args), s), "flex_attn_decode")


def flex_attn_prefill(plan: Plan, args: Args, stream=None):
    s = stream if stream is not None else current_stream()
    check(lib().flex_attn_prefill(plan.handle, ctypes.byref(args), s), "flex_attn_prefill")


def flex_attn_mixed(plan: Plan, args: Args, mode: int, stream=None, corun: "Corun" = None):
    s = stream if stream is not None else current_stream()
    check(lib().flex_attn_mixed(plan.handle, ctypes.byref(args), mode, s,
                                corun.handle if corun is not None else None), "flex_attn_mixed")


def flex_attn_validate_host(plan: Plan, block_table, num_pages: int, seq_lens, query_start_loc):
    """Host-side check of a run's metadata against the plan (torch CPU int32 tensors or int lists).
    Raises FlexAttnError (FLEX_ERR_INVALID_ARG) naming the first violation."""
    import torch
    bt = torch.as_tensor(block_table, dtype=torch.int32).contiguous()
    if bt.dim() != 2:
        raise ValueError("block_table must be 2-D")
    ptr = ctypes.cast(bt.data_ptr(), ctypes.POINTER(ctypes.c_int32))
    check(lib().flex_attn_validate_host(plan.handle, ptr, bt.stride(0), int(num_pages), _i32_array(seq_lens),
                                        _i32_array(query_start_loc)), "flex_attn_validate_host")


def set_debug(level: int) -> int:
    """Debug mode of the run calls (device check before launch); returns the previous level."""
    r = lib().flex_attn_set_debug(int(level))
    if r < 0:
        check(r, "flex_attn_set_debug")
    return r


def flex_attn_mixed_static(plan: Plan, args: Args, mode: int, stream=None, corun: "Corun" = None):
    """flex_attn_mixed with the split-K partials in the library's fixed scratch (allocates nothing)."""
    s = stream if stream is not None else current_stream()
    check(lib().flex_attn_mixed_static(plan.handle, ctypes.byref(args), mode, s,
                                       corun.handle if corun is not None else None), "flex_attn_mixed_static")


def static_scratch_bytes() -> int:
    return int(lib().flex_attn_static_scratch_bytes())


def flex_attn_debug_gather(plan: Plan, args: Args, seq: int, seq_len: int, k_out, v_out=None, stream=None):
    s = stream if stream is not None else current_stream()
    check(lib().flex_attn_debug_gather(plan.handle, ctypes.byref(args), seq, seq_len, _ptr(k_out),
                                       _ptr(v_out), s), "flex_attn_debug_gather")


def flex_attn_workspace_init(workspace, stream=None):
    s = stream if stream is not None else current_stream()
    check(lib().flex_attn_workspace_init(ctypes.c_void_p(workspace.data_ptr()),
                                         workspace.numel() * workspace.element_size(), s),
          "flex_attn_workspace_init")


def make_append_args(k_new, v_new, slot_mapping, k_cache, v_cache, bad_count=None) -> AppendArgs:
    """AppendArgs from device tensors: k_new [n, Hkv, d_qk] / v_new [n, Hkv, d_v] with
    contiguous rows, slot_mapping int32 [n], caches [pages, P, Hkv, d]."""
    a = AppendArgs()
    a.k_new = k_new.data_ptr()
    a.k_new_stride = k_new.stride(0)
    if v_new is not None:
        a.v_new = v_new.data_ptr()
        a.v_new_stride = v_new.stride(0)
    a.slot_mapping = slot_mapping.data_ptr()
    a.n_tokens = slot_mapping.numel()
    a.k_cache = k_cache.data_ptr()
    ks = k_cache.stride()
    a.k_stride = (ctypes.c_int64 * 3)(ks[0], ks[1], ks[2])
    vsrc = v_cache if v_cache is not None else k_cache
    a.v_cache = v_cache.data_ptr() if v_cache is not None else None
    vs = vsrc.stride()
    a.v_stride = (ctypes.c_int64 * 3)(vs[0], vs[1], vs[2])
    a.num_pages = k_cache.shape[0]
    a.bad_count = bad_count.data_ptr() if bad_count is not None else None
    return a


def flex_attn_kv_append(shape: Shape, args: AppendArgs, stream=None):
    s = stream if stream is not None else current_stream()
    check(lib().flex_attn_kv_append(ctypes.byref(shape), ctypes.byref(args), s), "flex_attn_kv_append")


class Controller:
    """The online co-location controller (flex_ctl_*): observe steps, decide splits."""

    def __init__(self, **opts):
        o = CtlOpts()
        for k, v in opts.items():
            setattr(o, k, v)
        h = ctypes.c_void_p()
        check(lib().flex_ctl_create(ctypes.byref(o), ctypes.byref(h)), "flex_ctl_create")
        self.handle = h
        self.K = (o.cus_total or 256) // (o.granule or 64)

    def close(self):
        if self.handle:
            lib().flex_ctl_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_profile(self, cus, decode_gbps, prefill_tflops):
        n = len(cus)
        check(lib().flex_ctl_set_profile(self.handle, n, (ctypes.c_int32 * n)(*cus),
                                         (ctypes.c_double * n)(*decode_gbps), (ctypes.c_double * n)(*prefill_tflops)),
              "flex_ctl_set_profile")

    def observe(self, cus_decode, decode_bytes, prefill_flops, decode_ms, prefill_ms, fused=False, step_ms=0.0):
        ob = CtlObservation(cus_decode, decode_bytes, prefill_flops, decode_ms, prefill_ms, 1 if fused else 0, step_ms)
        check(lib().flex_ctl_observe(self.handle, ctypes.byref(ob)), "flex_ctl_observe")

    def decide(self, decode_bytes, prefill_flops, pending_prefill_tokens=0, pending_decode_seqs=0,
               active_decode_seqs=1, fused_available=False, decode_tail=False) -> dict:
        sg = CtlSignals(decode_bytes, prefill_flops, pending_prefill_tokens, pending_decode_seqs, active_decode_seqs,
                        1 if fused_available else 0, 1 if decode_tail else 0)
        d = CtlDecision()
        check(lib().flex_ctl_decide(self.handle, ctypes.byref(sg), ctypes.byref(d)), "flex_ctl_decide")
        return {"mode": d.mode, "cus_decode": d.cus_decode, "cus_prefill": d.cus_prefill, "reason": d.reason,
                "predicted_us": d.predicted_us}

    def estimates(self):
        dg, pt = (ctypes.c_double * self.K)(), (ctypes.c_double * self.K)()
        check(lib().flex_ctl_estimates(self.handle, dg, pt, self.K), "flex_ctl_estimates")
        return list(dg), list(pt)


class TimeSlice:
    """The time-slice scheduler (flex_ts_*): one phase per step, decode's share
    of the device time held near decode_share."""

    def __init__(self, decode_share=0.5, decay=1.0):
        h = ctypes.c_void_p()
        check(lib().flex_ts_create(ctypes.byref(TsOpts(decode_share, decay)), ctypes.byref(h)), "flex_ts_create")
        self.handle = h

    def close(self):
        if self.handle:
            lib().flex_ts_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def next(self, decode_ready: bool, prefill_ready: bool) -> int:
        ph = ctypes.c_int32()
        check(lib().flex_ts_next(self.handle, int(bool(decode_ready)), int(bool(prefill_ready)), ctypes.byref(ph)),
              "flex_ts_next")
        return ph.value

    def observe(self, phase: int, ms: float):
        check(lib().flex_ts_observe(self.handle, int(phase), float(ms)), "flex_ts_observe")

    def totals(self):
        d, p = ctypes.c_double(), ctypes.c_double()
        check(lib().flex_ts_totals(self.handle, ctypes.byref(d), ctypes.byref(p)), "flex_ts_totals")
        return d.value, p.value


class Corun:
    """Owning wrapper of a co-run stream pair (two CU-masked streams)."""

    def __init__(self, cus_prefill: int, cus_decode: int):
        h = ctypes.c_void_p()
        check(lib().flex_attn_corun_create(cus_prefill, cus_decode, ctypes.byref(h)), "flex_attn_corun_create")
        self.handle = h
        self.cus_prefill = cus_prefill
        self.cus_decode = cus_decode

    def streams(self):
        p, d = ctypes.c_void_p(), ctypes.c_void_p()
        check(lib().flex_attn_corun_streams(self.handle, ctypes.byref(p), ctypes.byref(d)),
              "flex_attn_corun_streams")
        return p.value, d.value

    def set_timing(self, enable: bool = True):
        check(lib().flex_attn_corun_set_timing(self.handle, 1 if enable else 0), "flex_attn_corun_set_timing")

    def timing_read(self):
        """(prefill_ms, decode_ms) lists of the recorded steps, oldest first (waits for them)."""
        n = FLEX_TIMING_RING
        pre = (ctypes.c_float * n)()
        dec = (ctypes.c_float * n)()
        cnt = ctypes.c_int32()
        check(lib().flex_attn_corun_timing_read(self.handle, pre, dec, n, ctypes.byref(cnt)),
              "flex_attn_corun_timing_read")
        return list(pre[:cnt.value]), list(dec[:cnt.value])

    def close(self):
        if self.handle and self.handle.value:
            lib().flex_attn_corun_destroy(self.handle)
            self.handle = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class PagedAttention:
    """One batch's plan, its device copy and its workspace (torch-allocated).

    ``inputs`` holds the device tensors: q, k_cache, v_cache (or None when V
    aliases K), block_table, seq_lens, query_start_loc (int32). ``run`` calls
    the library on the current torch stream.
    """

    def __init__(self, shape: Shape, opts: Optional[PlanOpts], h_query_start_loc, h_seq_lens,
                 max_pages_per_seq: int, device="cuda"):
        import torch
        self.shape = shape
        self.plan = flex_attn_plan(shape, opts, h_query_start_loc, h_seq_lens, max_pages_per_seq)
        info = self.plan.info
        self.d_plan = torch.empty(max(256, info["device_plan_bytes"]), dtype=torch.uint8, device=device)
        self.workspace = torch.empty(max(256, info["workspace_bytes"]), dtype=torch.uint8, device=device)
        flex_attn_plan_upload(self.plan, self.d_plan)

    def args(self, q, k_cache, v_cache, block_table, seq_lens, query_start_loc, out, lse=None) -> Args:
        return make_args(q, k_cache, v_cache, block_table, seq_lens, query_start_loc, out, lse,
                         self.d_plan, self.workspace)

    def alloc_out(self, q, with_lse=False):
        import torch
        T, Hq = q.shape[0], q.shape[1]
        out = torch.empty((T, Hq, self.shape.head_dim_v), dtype=torch.bfloat16, device=q.device)
        lse = torch.empty((T, Hq), dtype=torch.float32, device=q.device) if with_lse else None
        return out, lse
