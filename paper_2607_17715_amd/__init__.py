"""Python binding of libc2kv.so, the C2KV compose-and-attend path on MI355X.

Argument marshalling only: torch tensors supply device memory and the current
HIP stream; every step of the path runs in the library's HIP kernels.  Names
follow the C ABI in include/c2kv.h (c2kv_compose, c2kv_attend,
c2kv_compose_attend, ...).  There is no fallback: if the library is missing,
importing the binding raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
# C2KV_LIBRARY selects another build of the same library (e.g. one with extra flags)
LIB_PATH = os.environ.get("C2KV_LIBRARY") or os.path.join(_PKG, "libc2kv.so")

C2KV_OK, C2KV_E_INVAL, C2KV_E_UNSUPPORTED, C2KV_E_WORKSPACE, C2KV_E_HIP, C2KV_E_NOMEM, \
    C2KV_E_STATE = 0, -1, -2, -3, -4, -5, -6
C2KV_F32, C2KV_BF16, C2KV_I8 = 0, 1, 2
C2KV_KEYS_ROPE_AT_ORIG, C2KV_KEYS_PRE_ROPE = 0, 1
C2KV_POOL_FULL, C2KV_POOL_COMPRESSED = 0, 1
_DTYPE_CODE = {"f32": C2KV_F32, "bf16": C2KV_BF16, "i8": C2KV_I8}

EXPORTED = [
    "c2kv_plan_create", "c2kv_plan_destroy", "c2kv_plan_get_info", "c2kv_plan_get_requests",
    "c2kv_plan_get_slots", "c2kv_plan_get_block_table", "c2kv_plan_upload", "c2kv_compose",
    "c2kv_attend", "c2kv_compose_attend", "c2kv_timing_enable", "c2kv_timing_reset",
    "c2kv_timing_read", "c2kv_last_error", "c2kv_version", "c2kv_host_alloc",
    "c2kv_host_free", "c2kv_load", "c2kv_sif_plan_create", "c2kv_compose_attend_static",
]
STATIC_SCRATCH_BYTES = 32 << 20   # C2KV_STATIC_SCRATCH_BYTES


class C2KVError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"c2kv status {status}: {msg}")
        self.status = status


class AttnCfg(ctypes.Structure):
    _fields_ = [("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("act_dtype", ctypes.c_int32),
                ("rope_base", ctypes.c_double), ("softmax_scale", ctypes.c_float)]


class ComposeDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_segments", ctypes.c_int32),
                ("req_seg_off", ctypes.c_void_p), ("seg_row0", ctypes.c_void_p),
                ("seg_span", ctypes.c_void_p), ("seg_orig_pos0", ctypes.c_void_p),
                ("seg_new_pos0", ctypes.c_void_p), ("seg_kept_off", ctypes.c_void_p),
                ("kept_idx", ctypes.c_void_p), ("key_encoding", ctypes.c_int32),
                ("pool_layout", ctypes.c_int32)]


class PlanOpts(ctypes.Structure):
    _fields_ = [("page_size", ctypes.c_int32), ("kv_splits", ctypes.c_int32),
                ("rows_per_block", ctypes.c_int32), ("num_cus", ctypes.c_int32),
                ("merge_mode", ctypes.c_int32)]


class PoolDesc(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("k_scale", ctypes.c_void_p), ("v_scale", ctypes.c_void_p),
                ("n_rows", ctypes.c_int64)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("suffix_len", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("n_pages", ctypes.c_int32),
                ("max_pages", ctypes.c_int32), ("n_segments", ctypes.c_int32),
                ("total_slots", ctypes.c_int64), ("max_src_row", ctypes.c_int64),
                ("workspace_bytes", ctypes.c_size_t), ("rows_per_block", ctypes.c_int32),
                ("n_work_items", ctypes.c_int32), ("n_merge_groups", ctypes.c_int32),
                ("max_splits", ctypes.c_int32)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python paper_2607_17715_amd/build.py`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    P = ctypes.POINTER
    sig = {
        "c2kv_plan_create": [P(AttnCfg), P(ComposeDesc), i32, P(PlanOpts), P(vp)],
        "c2kv_plan_destroy": [vp],
        "c2kv_plan_get_info": [vp, P(PlanInfo)],
        "c2kv_plan_get_requests": [vp, vp, vp],
        "c2kv_plan_get_slots": [vp, vp, vp, vp],
        "c2kv_plan_get_block_table": [vp, vp],
        "c2kv_plan_upload": [vp, vp, sz, vp],
        "c2kv_compose": [vp, P(PoolDesc), vp, vp, vp, vp, vp, vp],
        "c2kv_attend": [vp, vp, vp, vp, vp, vp, vp, vp, vp],
        "c2kv_compose_attend": [vp, P(PoolDesc), vp, vp, vp, vp, vp, vp],
        "c2kv_compose_attend_static": [vp, P(PoolDesc), vp, vp, vp, vp, vp, vp],
        "c2kv_timing_enable": [i32],
        "c2kv_timing_reset": [],
        "c2kv_timing_read": [ctypes.c_char_p, P(ctypes.c_double), P(i64)],
        "c2kv_last_error": [],
        "c2kv_version": [],
        "c2kv_host_alloc": [sz, P(vp), P(vp)],
        "c2kv_host_free": [vp],
        "c2kv_load": [vp, P(PoolDesc), P(PoolDesc), vp],
        "c2kv_sif_plan_create": [P(AttnCfg), i32, i32, i32, i32, P(PlanOpts), P(vp)],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = None if name == "c2kv_plan_destroy" else (
            ctypes.c_char_p if name in ("c2kv_last_error", "c2kv_version") else ctypes.c_int)
    return lib


_lib = _load()


def lib() -> ctypes.CDLL:
    return _lib


def _check(status: int):
    if status != C2KV_OK:
        raise C2KVError(status, _lib.c2kv_last_error().decode(errors="replace"))


def version() -> str:
    return _lib.c2kv_version().decode()


def _np_ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def _dev_ptr(t) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return t.data_ptr()


def _stream(stream=None):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


class Plan:
    """Host plan of one batch of compositions (c2kv_plan_create), shared by every layer."""

    def __init__(self, n_q_heads: int, n_kv_heads: int, head_dim: int, act_dtype: str,
                 rope_base: float, req_seg_off, seg_row0, seg_span, seg_orig_pos0,
                 seg_kept_off, kept_idx, suffix_len: int, seg_new_pos0=None,
                 softmax_scale: float = 0.0, page_size: int = 0, kv_splits: int = 0,
                 rows_per_block: int = 0, num_cus: int = 0, merge_mode: int = 0,
                 keys_pre_rope: bool = False, pool_compressed: bool = False):
        self._arrays = dict(
            req_seg_off=np.ascontiguousarray(req_seg_off, np.int32),
            seg_row0=np.ascontiguousarray(seg_row0, np.int64),
            seg_span=np.ascontiguousarray(seg_span, np.int32),
            seg_orig_pos0=np.ascontiguousarray(seg_orig_pos0, np.int32),
            seg_kept_off=np.ascontiguousarray(seg_kept_off, np.int32),
            kept_idx=np.ascontiguousarray(kept_idx, np.int32),
            seg_new_pos0=None if seg_new_pos0 is None else np.ascontiguousarray(seg_new_pos0, np.int32),
        )
        a = self._arrays
        self.cfg = AttnCfg(n_q_heads, n_kv_heads, head_dim, _DTYPE_CODE[act_dtype],
                           float(rope_base), float(softmax_scale))
        self.act_dtype = act_dtype
        desc = ComposeDesc(len(a["req_seg_off"]) - 1, len(a["seg_row0"]),
                           _np_ptr(a["req_seg_off"]), _np_ptr(a["seg_row0"]),
                           _np_ptr(a["seg_span"]), _np_ptr(a["seg_orig_pos0"]),
                           _np_ptr(a["seg_new_pos0"]), _np_ptr(a["seg_kept_off"]),
                           _np_ptr(a["kept_idx"]), C2KV_KEYS_PRE_ROPE if keys_pre_rope
                           else C2KV_KEYS_ROPE_AT_ORIG,
                           C2KV_POOL_COMPRESSED if pool_compressed else C2KV_POOL_FULL)
        opts = PlanOpts(page_size, kv_splits, rows_per_block, num_cus, merge_mode)
        h = ctypes.c_void_p()
        _check(_lib.c2kv_plan_create(ctypes.byref(self.cfg), ctypes.byref(desc),
                                     int(suffix_len), ctypes.byref(opts), ctypes.byref(h)))
        self._h = h
        self.suffix_len = int(suffix_len)
        self.workspace = None
        inf = PlanInfo()
        _check(_lib.c2kv_plan_get_info(self._h, ctypes.byref(inf)))
        self.info = inf.as_dict()

    @classmethod
    def sif(cls, n_q_heads: int, n_kv_heads: int, head_dim: int, act_dtype: str,
            rope_base: float, batch: int, n_tokens: int, block: int, sink: int,
            softmax_scale: float = 0.0, page_size: int = 0, kv_splits: int = 0,
            rows_per_block: int = 0, num_cus: int = 0, merge_mode: int = 0) -> "Plan":
        """Plan of extraction-time SIF attention (c2kv_sif_plan_create); run it with
        c2kv_attend(plan, None, None, q, k, v, out, lse)."""
        self = cls.__new__(cls)
        self._arrays = {}
        self.cfg = AttnCfg(n_q_heads, n_kv_heads, head_dim, _DTYPE_CODE[act_dtype],
                           float(rope_base), float(softmax_scale))
        self.act_dtype = act_dtype
        opts = PlanOpts(page_size, kv_splits, rows_per_block, num_cus, merge_mode)
        h = ctypes.c_void_p()
        _check(_lib.c2kv_sif_plan_create(ctypes.byref(self.cfg), int(batch), int(n_tokens),
                                         int(block), int(sink), ctypes.byref(opts),
                                         ctypes.byref(h)))
        self._h = h
        self.workspace = None
        inf = PlanInfo()
        _check(_lib.c2kv_plan_get_info(self._h, ctypes.byref(inf)))
        self.info = inf.as_dict()
        self.suffix_len = self.info["suffix_len"]
        return self

    @classmethod
    def for_sif(cls, w, **opts) -> "Plan":
        return cls.sif(w.n_q_heads, w.n_kv_heads, w.head_dim, w.act_dtype, w.rope_base,
                       w.batch, w.n_tokens, w.block, w.sink, **opts)

    @classmethod
    def for_workload(cls, w, **opts) -> "Plan":
        return cls(w.n_q_heads, w.n_kv_heads, w.head_dim, w.act_dtype, w.rope_base,
                   w.req_seg_off, w.seg_row0, w.seg_span, w.seg_orig_pos0, w.seg_kept_off,
                   w.kept_idx, w.suffix_len, seg_new_pos0=w.seg_new_pos0,
                   keys_pre_rope=getattr(w, "keys_pre_rope", False),
                   pool_compressed=getattr(w, "pool_compressed", False), **opts)

    def __del__(self):
        h = getattr(self, "_h", None)
        lib_ = _lib
        if h is not None and h.value and lib_ is not None:   # None at interpreter teardown
            lib_.c2kv_plan_destroy(h)
            self._h = None

    @property
    def handle(self):
        return self._h

    # ---- host copies of the layout --------------------------------------------
    def requests(self):
        B = self.info["batch"]
        n = np.zeros(B, np.int32)
        e = np.zeros(B, np.int32)
        _check(_lib.c2kv_plan_get_requests(self._h, _np_ptr(n), _np_ptr(e)))
        return n, e

    def slots(self):
        T = self.info["total_slots"]
        src = np.zeros(max(T, 1), np.int64)
        pos = np.zeros(max(T, 1), np.int32)
        dl = np.zeros(max(T, 1), np.int32)
        _check(_lib.c2kv_plan_get_slots(self._h, _np_ptr(src), _np_ptr(pos), _np_ptr(dl)))
        return src[:T], pos[:T], dl[:T]

    def block_table(self):
        bt = np.zeros((self.info["batch"], self.info["max_pages"]), np.int32)
        _check(_lib.c2kv_plan_get_block_table(self._h, _np_ptr(bt)))
        return bt

    # ---- device ---------------------------------------------------------------
    def upload(self, workspace=None, stream=None):
        """Bind the plan to a device workspace (allocated here if not given)."""
        import torch
        nbytes = int(self.info["workspace_bytes"])
        if workspace is None:
            workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device="cuda")
            off = (-workspace.data_ptr()) % 256
            workspace = workspace[off:off + nbytes]
        _check(_lib.c2kv_plan_upload(self._h, ctypes.c_void_p(workspace.data_ptr()),
                                     workspace.numel(), _stream(stream)))
        self.workspace = workspace
        return self


def pool_desc(k, v, k_scale=None, v_scale=None) -> PoolDesc:
    import torch
    code = {torch.float32: C2KV_F32, torch.bfloat16: C2KV_BF16, torch.int8: C2KV_I8}[k.dtype]
    if v.dtype != k.dtype or v.shape != k.shape:
        raise ValueError("pool K and V must have the same dtype and shape")
    return PoolDesc(code, _dev_ptr(k), _dev_ptr(v), _dev_ptr(k_scale), _dev_ptr(v_scale),
                    int(k.shape[0]))


def page_shapes(plan: Plan):
    """Shapes of k_pages and v_pages (v_pages holds each page transposed)."""
    i, c = plan.info, plan.cfg
    return ((i["n_pages"], c.n_kv_heads, i["page_size"], c.head_dim),
            (i["n_pages"], c.n_kv_heads, c.head_dim, i["page_size"]))


def c2kv_compose(plan: Plan, pool: PoolDesc, k_pages, v_pages, slot_src_row=None,
                 slot_pos=None, block_table=None, stream=None):
    _check(_lib.c2kv_compose(plan.handle, ctypes.byref(pool), _dev_ptr(k_pages),
                             _dev_ptr(v_pages), _dev_ptr(slot_src_row), _dev_ptr(slot_pos),
                             _dev_ptr(block_table), _stream(stream)))


def c2kv_attend(plan: Plan, k_pages, v_pages, q, k_suf, v_suf, out, lse=None, stream=None):
    _check(_lib.c2kv_attend(plan.handle, _dev_ptr(k_pages), _dev_ptr(v_pages), _dev_ptr(q),
                            _dev_ptr(k_suf), _dev_ptr(v_suf), _dev_ptr(out), _dev_ptr(lse),
                            _stream(stream)))


def c2kv_compose_attend(plan: Plan, pool: PoolDesc, q, k_suf, v_suf, out, lse=None,
                        stream=None):
    _check(_lib.c2kv_compose_attend(plan.handle, ctypes.byref(pool), _dev_ptr(q),
                                    _dev_ptr(k_suf), _dev_ptr(v_suf), _dev_ptr(out),
                                    _dev_ptr(lse), _stream(stream)))


def c2kv_compose_attend_static(plan: Plan, pool: PoolDesc, q, k_suf, v_suf, out, lse=None,
                               stream=None):
    """c2kv_compose_attend with the tables and partials in the library's static
    device array (no workspace, no upload needed)."""
    _check(_lib.c2kv_compose_attend_static(plan.handle, ctypes.byref(pool), _dev_ptr(q),
                                           _dev_ptr(k_suf), _dev_ptr(v_suf), _dev_ptr(out),
                                           _dev_ptr(lse), _stream(stream)))


def c2kv_load(plan: Plan, src: PoolDesc, dst: PoolDesc, stream=None):
    _check(_lib.c2kv_load(plan.handle, ctypes.byref(src), ctypes.byref(dst), _stream(stream)))


class HostPool:
    """A pool in page-locked host memory from c2kv_host_alloc, filled from numpy
    storage arrays (bf16 as uint16 bit patterns).  `desc` points kernels at it
    for reads in place over the host link; it is also a c2kv_load source."""

    def __init__(self, pool_k: np.ndarray, pool_v: np.ndarray, dtype: str,
                 k_scale: Optional[np.ndarray] = None, v_scale: Optional[np.ndarray] = None):
        self._host = []
        code = {"f32": C2KV_F32, "bf16": C2KV_BF16, "i8": C2KV_I8}[dtype]
        if pool_k.shape != pool_v.shape:
            raise ValueError("pool K and V must have the same shape")
        self.nbytes = 0
        ptrs = [self._put(a) for a in (pool_k, pool_v, k_scale, v_scale)]
        self.desc = PoolDesc(code, ptrs[0], ptrs[1], ptrs[2], ptrs[3], int(pool_k.shape[0]))

    def _put(self, a: Optional[np.ndarray]):
        if a is None:
            return None
        a = np.ascontiguousarray(a)
        host, dev = ctypes.c_void_p(), ctypes.c_void_p()
        _check(_lib.c2kv_host_alloc(max(a.nbytes, 1), ctypes.byref(host), ctypes.byref(dev)))
        self._host.append(host)
        ctypes.memmove(host, a.ctypes.data, a.nbytes)
        self.nbytes += a.nbytes
        return dev.value

    def close(self):
        lib_ = _lib
        while self._host and lib_ is not None:
            lib_.c2kv_host_free(self._host.pop())

    def __del__(self):
        self.close()


def timing_enable(on: bool = True):
    _check(_lib.c2kv_timing_enable(1 if on else 0))


def timing_reset():
    _check(_lib.c2kv_timing_reset())


def timing_read(name: str):
    ms = ctypes.c_double()
    n = ctypes.c_int64()
    _check(_lib.c2kv_timing_read(name.encode(), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


# ---- tensor helpers (host <-> device marshalling) ------------------------------

def to_device(a: np.ndarray, dtype: str):
    """numpy storage array -> device tensor ('bf16' arrays are uint16 bit patterns)."""
    import torch
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    elif dtype == "f32":
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    elif dtype == "i8":
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.int8))
    else:
        raise ValueError(dtype)
    return t.to("cuda")


def to_numpy_f64(t) -> np.ndarray:
    import torch
    return t.detach().to(torch.float64).cpu().numpy()
