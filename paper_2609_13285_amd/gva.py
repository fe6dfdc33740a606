"""Thin ctypes binding of libgva.so (declared in include/gva.h).

Argument marshalling only: every function here checks the tensors it is
given (device, dtype, shape, contiguity), passes raw device pointers and the
current HIP stream, and raises :class:`GvaError` on a non-zero status.  All
arithmetic runs in the HIP kernels.  There is no fallback: if libgva.so is
missing, the first call raises.
"""

from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Tuple

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libgva.so")

GVA_OK, GVA_ERR_INVALID_ARG, GVA_ERR_UNSUPPORTED, GVA_ERR_HIP, GVA_ERR_SCRATCH = 0, -1, -2, -3, -4
GVA_STATIC_SCRATCH_BYTES = 16 << 20
GVA_DTYPE_F32, GVA_DTYPE_BF16 = 0, 1
GVA_MAX_SPLITS = 256
EXPORTS = ("gva_append_kv", "gva_absorb_query", "gva_decode_attention", "gva_combine",
           "gva_gqa_decode_attention", "gva_paged_append_kv", "gva_paged_decode_attention",
           "gva_rope_decode_attention", "gva_prefill_absorb", "gva_prefill_attention",
           "gva_gqa_prefill_attention", "gva_pick_splits", "gva_prefer_fused", "gva_status_string",
           "gva_version", "gva_decode_workspace_size", "gva_decode_step", "gva_decode_step_static")
GVA_MAX_PAGES = 4096
PROBE_EXPORTS = ("gva_probe_read",)      # include/gva_probe.h


class GvaError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed: {status_string(status)} ({status})")


class GvaDims(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_groups", ctypes.c_int32), ("d_v", ctypes.c_int32),
                ("d_c", ctypes.c_int32), ("d_r", ctypes.c_int32),
                ("t_max", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("rope_base", ctypes.c_double), ("scale", ctypes.c_double)]

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.bfloat16 if self.dtype == GVA_DTYPE_BF16 else torch.float32

    def __repr__(self):
        return ("GvaDims(" + ", ".join(f"{k}={getattr(self, k)}" for k, _ in self._fields_) + ")")


class GvaPaging(ctypes.Structure):
    _fields_ = [("page_rows", ctypes.c_int32), ("max_pages", ctypes.c_int32),
                ("n_pages", ctypes.c_int32)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libgva.so (once).  Raises GvaError-like RuntimeError if absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run `python -m paper_2609_13285_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, I32 = ctypes.c_void_p, ctypes.c_int32
        D = ctypes.POINTER(GvaDims)
        L.gva_append_kv.argtypes = [D, P, P, P, P, P, P, I32, P]
        L.gva_absorb_query.argtypes = [D, P, P, P, P, P, P]
        L.gva_decode_attention.argtypes = [D, P, P, P, P, P, P, P, P, P, I32, I32, P, P, P]
        L.gva_combine.argtypes = [D, P, P, I32, P, P, P]
        L.gva_gqa_decode_attention.argtypes = [D, P, I32, P, P, P, I32, I32, P, P, P]
        L.gva_rope_decode_attention.argtypes = [D, P, P, P, P, I32, I32, P, P, P]
        L.gva_prefill_absorb.argtypes = [D, I32, P, P, P, P, P, P]
        L.gva_prefill_attention.argtypes = [D, I32, P, P, P, P, P, P, P, P]
        L.gva_gqa_prefill_attention.argtypes = [D, I32, P, P, P, P, P, P, P]
        PG = ctypes.POINTER(GvaPaging)
        L.gva_paged_append_kv.argtypes = [D, PG, P, P, P, P, P, P, P, I32, P]
        L.gva_paged_decode_attention.argtypes = [D, PG, P, P, P, P, P, P, P, P, P, P, I32, I32, P, P, P]
        L.gva_pick_splits.argtypes = [D, I32, ctypes.c_int64, I32, ctypes.POINTER(I32)]
        L.gva_prefer_fused.argtypes = [D, I32, I32, I32]
        L.gva_decode_workspace_size.argtypes = [D, I32, I32, ctypes.POINTER(ctypes.c_size_t)]
        L.gva_decode_step.argtypes = [D, P, P, P, P, P, P, P, I32, I32, P, ctypes.c_size_t, P, P, P]
        L.gva_decode_step_static.argtypes = [D, P, P, P, P, P, P, P, I32, I32, P, P, P]
        L.gva_status_string.argtypes = [ctypes.c_int]
        L.gva_status_string.restype = ctypes.c_char_p
        L.gva_version.argtypes = []
        L.gva_probe_read.argtypes = [P, ctypes.c_int64, I32, P, P]
        for name in ("gva_append_kv", "gva_absorb_query", "gva_decode_attention", "gva_combine",
                     "gva_gqa_decode_attention", "gva_paged_append_kv", "gva_paged_decode_attention",
                     "gva_rope_decode_attention", "gva_prefill_absorb", "gva_prefill_attention",
                     "gva_gqa_prefill_attention", "gva_pick_splits", "gva_version", "gva_probe_read",
                     "gva_decode_workspace_size", "gva_decode_step", "gva_decode_step_static"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


class _Recorder:
    """Stands in for the loaded library while prepare() runs a binding call:
    records each C call with its marshalled arguments instead of making it."""

    def __init__(self, real):
        self._real = real
        self.calls = []

    def __getattr__(self, name):
        fn = getattr(self._real, name)

        def record(*args):
            self.calls.append((name, fn, args))
            return GVA_OK
        return record


def prepare(call, *args, **kwargs):
    """Check and marshal one binding call now (``call`` is one of this
    module's gva_* functions, with its usual arguments) and return a
    zero-argument function that makes the same C calls again -- the same
    device pointers, sizes and stream -- without the per-call Python checks.
    For loops whose tensors stay where they are (timing, serving); the
    caller keeps the tensors alive.  Each re-issue still checks the status
    the library returns."""
    global _lib
    real = lib()
    rec = _Recorder(real)
    _lib = rec
    try:
        call(*args, **kwargs)
    finally:
        _lib = real
    calls = tuple(rec.calls)

    def run():
        for name, fn, a in calls:
            st = fn(*a)
            if st != GVA_OK:
                raise GvaError(name, st)
    run.calls = calls
    return run


def status_string(status: int) -> str:
    return lib().gva_status_string(int(status)).decode()


def make_dims(batch: int, n_heads: int, n_groups: int, d_v: int, d_c: int, d_r: int,
              t_max: int, dtype, rope_base: float = 10000.0, scale: float = 0.0) -> GvaDims:
    if isinstance(dtype, torch.dtype):
        code = {torch.bfloat16: GVA_DTYPE_BF16, torch.float32: GVA_DTYPE_F32}[dtype]
    elif isinstance(dtype, str):
        code = {"bf16": GVA_DTYPE_BF16, "f32": GVA_DTYPE_F32}[dtype]
    else:
        code = int(dtype)
    return GvaDims(batch, n_heads, n_groups, d_v, d_c, d_r, t_max, code, float(rope_base), float(scale))


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _in_use_on(stream, *tensors):
    """Tell torch's caching allocator that ``tensors``, allocated on the
    current stream, are also read by kernels enqueued on ``stream``, so their
    memory is not handed out again before that work is done."""
    if stream is None:
        return
    s = stream if isinstance(stream, torch.cuda.Stream) else torch.cuda.ExternalStream(int(stream))
    if s.cuda_stream == torch.cuda.current_stream().cuda_stream:
        return
    for t in tensors:
        if t is not None:
            t.record_stream(s)


def _ptr(t: Optional[torch.Tensor], name: str, dtype=None, shape=None):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return ctypes.c_void_p(t.data_ptr())


def _check(fn: str, status: int):
    if status != GVA_OK:
        raise GvaError(fn, status)


def gva_append_kv(dims: GvaDims, v_cache, kr_cache, v_new, kr_new, seq, pos, stream=None):
    d = dims
    dt = d.torch_dtype
    n = seq.numel()
    st = lib().gva_append_kv(
        ctypes.byref(d),
        _ptr(v_cache, "v_cache", dt, (d.batch, d.n_groups, d.t_max, d.d_v)),
        _ptr(kr_cache, "kr_cache", dt, (d.batch, d.t_max, d.d_r)),
        _ptr(v_new, "v_new", dt, (n, d.n_groups, d.d_v)),
        _ptr(kr_new, "kr_new", dt, (n, d.d_r)),
        _ptr(seq, "seq", torch.int32, (n,)), _ptr(pos, "pos", torch.int32, (n,)),
        n, _stream(stream))
    _check("gva_append_kv", st)


def gva_absorb_query(dims: GvaDims, q, m, lens, q_abs, q_rot, stream=None):
    d = dims
    dt = d.torch_dtype
    st = lib().gva_absorb_query(
        ctypes.byref(d),
        _ptr(q, "q", dt, (d.batch, d.n_heads, d.d_c + d.d_r)),
        _ptr(m, "m", dt, (d.n_heads, d.d_v, d.d_c)),
        _ptr(lens, "lens", torch.int32, (d.batch,)),
        _ptr(q_abs, "q_abs", torch.float32, (d.batch, d.n_heads, d.d_v)),
        _ptr(q_rot, "q_rot", torch.float32, (d.batch, d.n_heads, d.d_r)),
        _stream(stream))
    _check("gva_absorb_query", st)


def gva_decode_attention(dims: GvaDims, v_cache, kr_cache, lens, num_splits: int, o_part, lse_part,
                         q=None, m=None, q_abs=None, q_rot=None, v_new=None, kr_new=None,
                         split_rows: int = 0, stream=None):
    d = dims
    dt = d.torch_dtype
    S = int(num_splits)
    st = lib().gva_decode_attention(
        ctypes.byref(d),
        _ptr(q, "q", dt, (d.batch, d.n_heads, d.d_c + d.d_r)),
        _ptr(m, "m", dt, (d.n_heads, d.d_v, d.d_c)),
        _ptr(q_abs, "q_abs", torch.float32, (d.batch, d.n_heads, d.d_v)),
        _ptr(q_rot, "q_rot", torch.float32, (d.batch, d.n_heads, d.d_r)),
        _ptr(v_cache, "v_cache", dt, (d.batch, d.n_groups, d.t_max, d.d_v)),
        _ptr(kr_cache, "kr_cache", dt, (d.batch, d.t_max, d.d_r)),
        _ptr(lens, "lens", torch.int32, (d.batch,)),
        _ptr(v_new, "v_new", dt, (d.batch, d.n_groups, d.d_v)),
        _ptr(kr_new, "kr_new", dt, (d.batch, d.d_r)),
        S,
        int(split_rows),
        _ptr(o_part, "o_part", torch.float32, (d.batch, d.n_heads, S, d.d_v)),
        _ptr(lse_part, "lse_part", torch.float32, (d.batch, d.n_heads, S)),
        _stream(stream))
    _check("gva_decode_attention", st)


def gva_combine(dims: GvaDims, o_part, lse_part, num_splits: int, o, lse=None, stream=None):
    d = dims
    S = int(num_splits)
    st = lib().gva_combine(
        ctypes.byref(d),
        _ptr(o_part, "o_part", torch.float32, (d.batch, d.n_heads, S, d.d_v)),
        _ptr(lse_part, "lse_part", torch.float32, (d.batch, d.n_heads, S)),
        S,
        _ptr(o, "o", torch.float32, (d.batch, d.n_heads, d.d_v)),
        _ptr(lse, "lse", torch.float32, (d.batch, d.n_heads)),
        _stream(stream))
    _check("gva_combine", st)


def gva_decode_workspace_size(dims: GvaDims, num_splits: int, split_rows: int = 0) -> int:
    """Workspace bytes gva_decode_step needs for this plan on the current device."""
    n = ctypes.c_size_t(0)
    _check("gva_decode_workspace_size",
           lib().gva_decode_workspace_size(ctypes.byref(dims), int(num_splits), int(split_rows), ctypes.byref(n)))
    return int(n.value)


def workspace_for(dims: GvaDims, num_splits: int, split_rows: int = 0, device="cuda") -> Optional[torch.Tensor]:
    """A device buffer for gva_decode_step (None when the plan needs none);
    torch's allocator aligns it to 256 bytes or more."""
    n = gva_decode_workspace_size(dims, num_splits, split_rows)
    return torch.empty(n, dtype=torch.uint8, device=device) if n else None


def gva_decode_step(dims: GvaDims, q, m, v_cache, kr_cache, lens, num_splits: int, o, lse, workspace=None,
                    v_new=None, kr_new=None, split_rows: int = 0, stream=None):
    """One whole decode step (absorb + attention + combine) into o / lse."""
    d = dims
    dt = d.torch_dtype
    S = int(num_splits)
    if workspace is not None and (workspace.dtype != torch.uint8 or workspace.dim() != 1):
        raise ValueError("workspace must be a 1-D uint8 tensor")
    st = lib().gva_decode_step(
        ctypes.byref(d),
        _ptr(q, "q", dt, (d.batch, d.n_heads, d.d_c + d.d_r)),
        _ptr(m, "m", dt, (d.n_heads, d.d_v, d.d_c)),
        _ptr(v_cache, "v_cache", dt, (d.batch, d.n_groups, d.t_max, d.d_v)),
        _ptr(kr_cache, "kr_cache", dt, (d.batch, d.t_max, d.d_r)),
        _ptr(lens, "lens", torch.int32, (d.batch,)),
        _ptr(v_new, "v_new", dt, (d.batch, d.n_groups, d.d_v)),
        _ptr(kr_new, "kr_new", dt, (d.batch, d.d_r)),
        S, int(split_rows),
        _ptr(workspace, "workspace"),
        0 if workspace is None else workspace.numel(),
        _ptr(o, "o", torch.float32, (d.batch, d.n_heads, d.d_v)),
        _ptr(lse, "lse", torch.float32, (d.batch, d.n_heads)),
        _stream(stream))
    _check("gva_decode_step", st)


def gva_decode_step_static(dims: GvaDims, q, m, v_cache, kr_cache, lens, num_splits: int, o, lse,
                           v_new=None, kr_new=None, split_rows: int = 0, stream=None):
    """gva_decode_step with its workspace in the library's static per-device
    scratch buffer: for callers that cannot allocate."""
    d = dims
    dt = d.torch_dtype
    st = lib().gva_decode_step_static(
        ctypes.byref(d),
        _ptr(q, "q", dt, (d.batch, d.n_heads, d.d_c + d.d_r)),
        _ptr(m, "m", dt, (d.n_heads, d.d_v, d.d_c)),
        _ptr(v_cache, "v_cache", dt, (d.batch, d.n_groups, d.t_max, d.d_v)),
        _ptr(kr_cache, "kr_cache", dt, (d.batch, d.t_max, d.d_r)),
        _ptr(lens, "lens", torch.int32, (d.batch,)),
        _ptr(v_new, "v_new", dt, (d.batch, d.n_groups, d.d_v)),
        _ptr(kr_new, "kr_new", dt, (d.batch, d.d_r)),
        int(num_splits), int(split_rows),
        _ptr(o, "o", torch.float32, (d.batch, d.n_heads, d.d_v)),
        _ptr(lse, "lse", torch.float32, (d.batch, d.n_heads)),
        _stream(stream))
    _check("gva_decode_step_static", st)


def gva_gqa_decode_attention(dims: GvaDims, q, k_cache, v_cache, lens, num_splits: int, o_part,
                             lse_part, split_rows: int = 0, stream=None):
    """The matched-GQA baseline; ``q`` is [B, H, q_stride] with the query's
    first d_v entries used."""
    d = dims
    dt = d.torch_dtype
    S = int(num_splits)
    if not isinstance(q, torch.Tensor) or q.dim() != 3:
        raise ValueError("q must be a [B, H, q_stride] tensor")
    st = lib().gva_gqa_decode_attention(
        ctypes.byref(d),
        _ptr(q, "q", dt, (d.batch, d.n_heads, q.shape[-1])),
        int(q.shape[-1]),
        _ptr(k_cache, "k_cache", dt, (d.batch, d.n_groups, d.t_max, d.d_v)),
        _ptr(v_cache, "v_cache", dt, (d.batch, d.n_groups, d.t_max, d.d_v)),
        _ptr(lens, "lens", torch.int32, (d.batch,)),
        S,
        int(split_rows),
        _ptr(o_part, "o_part", torch.float32, (d.batch, d.n_heads, S, d.d_v)),
        _ptr(lse_part, "lse_part", torch.float32, (d.batch, d.n_heads, S)),
        _stream(stream))
    _check("gva_gqa_decode_attention", st)


def gva_rope_decode_attention(dims: GvaDims, q, m, v_cache, lens, num_splits: int, o_part, lse_part,
                              split_rows: int = 0, stream=None):
    """GVA with ordinary RoPE (keys reconstructed and rotated per position):
    ``q`` [B, H, d_c], ``m`` [H, d_v, d_c], dims.d_r == 0."""
    d = dims
    dt = d.torch_dtype
    S = int(num_splits)
    st = lib().gva_rope_decode_attention(
        ctypes.byref(d),
        _ptr(q, "q", dt, (d.batch, d.n_heads, d.d_c)),
        _ptr(m, "m", dt, (d.n_heads, d.d_v, d.d_c)),
        _ptr(v_cache, "v_cache", dt, (d.batch, d.n_groups, d.t_max, d.d_v)),
        _ptr(lens, "lens", torch.int32, (d.batch,)),
        S,
        int(split_rows),
        _ptr(o_part, "o_part", torch.float32, (d.batch, d.n_heads, S, d.d_v)),
        _ptr(lse_part, "lse_part", torch.float32, (d.batch, d.n_heads, S)),
        _stream(stream))
    _check("gva_rope_decode_attention", st)


def gva_prefill_absorb(dims: GvaDims, n_new: int, q, m, lens, q_abs, q_rot, stream=None):
    """Absorb and rotate a prompt's queries: q [B, n_new, H, d_c+d_r]."""
    d = dims
    N = int(n_new)
    st = lib().gva_prefill_absorb(
        ctypes.byref(d), N,
        _ptr(q, "q", d.torch_dtype, (d.batch, N, d.n_heads, d.d_c + d.d_r)),
        _ptr(m, "m", d.torch_dtype, (d.n_heads, d.d_v, d.d_c)),
        _ptr(lens, "lens", torch.int32, (d.batch,)),
        _ptr(q_abs, "q_abs", torch.float32, (d.batch, N, d.n_heads, d.d_v)),
        _ptr(q_rot, "q_rot", torch.float32, (d.batch, N, d.n_heads, d.d_r)) if d.d_r > 0 else None,
        _stream(stream))
    _check("gva_prefill_absorb", st)


def gva_prefill_attention(dims: GvaDims, n_new: int, q_abs, q_rot, v_cache, kr_cache, lens, o, lse,
                          stream=None):
    """Causal attention for each sequence's last n_new cached rows."""
    d = dims
    N = int(n_new)
    dt = d.torch_dtype
    st = lib().gva_prefill_attention(
        ctypes.byref(d), N,
        _ptr(q_abs, "q_abs", torch.float32, (d.batch, N, d.n_heads, d.d_v)),
        _ptr(q_rot, "q_rot", torch.float32, (d.batch, N, d.n_heads, d.d_r)) if d.d_r > 0 else None,
        _ptr(v_cache, "v_cache", dt, (d.batch, d.n_groups, d.t_max, d.d_v)),
        _ptr(kr_cache, "kr_cache", dt, (d.batch, d.t_max, d.d_r)) if d.d_r > 0 else None,
        _ptr(lens, "lens", torch.int32, (d.batch,)),
        _ptr(o, "o", torch.float32, (d.batch, N, d.n_heads, d.d_v)),
        _ptr(lse, "lse", torch.float32, (d.batch, N, d.n_heads)),
        _stream(stream))
    _check("gva_prefill_attention", st)


def gva_gqa_prefill_attention(dims: GvaDims, n_new: int, q, k_cache, v_cache, lens, o, lse, stream=None):
    """The matched-GQA causal prefill: q [B, n_new, H, d_v] fp32."""
    d = dims
    N = int(n_new)
    dt = d.torch_dtype
    st = lib().gva_gqa_prefill_attention(
        ctypes.byref(d), N,
        _ptr(q, "q", torch.float32, (d.batch, N, d.n_heads, d.d_v)),
        _ptr(k_cache, "k_cache", dt, (d.batch, d.n_groups, d.t_max, d.d_v)),
        _ptr(v_cache, "v_cache", dt, (d.batch, d.n_groups, d.t_max, d.d_v)),
        _ptr(lens, "lens", torch.int32, (d.batch,)),
        _ptr(o, "o", torch.float32, (d.batch, N, d.n_heads, d.d_v)),
        _ptr(lse, "lse", torch.float32, (d.batch, N, d.n_heads)),
        _stream(stream))
    _check("gva_gqa_prefill_attention", st)


def gva_paged_append_kv(dims: GvaDims, paging: GvaPaging, v_pool, kr_pool, block_table, v_new, kr_new,
                        seq, pos, stream=None):
    d, pg = dims, paging
    dt = d.torch_dtype
    n = int(seq.numel())
    st = lib().gva_paged_append_kv(
        ctypes.byref(d), ctypes.byref(pg),
        _ptr(v_pool, "v_pool", dt, (pg.n_pages, d.n_groups, pg.page_rows, d.d_v)),
        _ptr(kr_pool, "kr_pool", dt, (pg.n_pages, pg.page_rows, d.d_r)),
        _ptr(block_table, "block_table", torch.int32, (d.batch, pg.max_pages)),
        _ptr(v_new, "v_new", dt, (n, d.n_groups, d.d_v)),
        _ptr(kr_new, "kr_new", dt, (n, d.d_r)),
        _ptr(seq, "seq", torch.int32, (n,)),
        _ptr(pos, "pos", torch.int32, (n,)),
        n, _stream(stream))
    _check("gva_paged_append_kv", st)


def gva_paged_decode_attention(dims: GvaDims, paging: GvaPaging, v_pool, kr_pool, block_table, lens,
                               num_splits: int, o_part, lse_part, q=None, m=None, q_abs=None, q_rot=None,
                               v_new=None, kr_new=None, split_rows: int = 0, stream=None):
    d, pg = dims, paging
    dt = d.torch_dtype
    S = int(num_splits)
    st = lib().gva_paged_decode_attention(
        ctypes.byref(d), ctypes.byref(pg),
        _ptr(q, "q", dt, (d.batch, d.n_heads, d.d_c + d.d_r)),
        _ptr(m, "m", dt, (d.n_heads, d.d_v, d.d_c)),
        _ptr(q_abs, "q_abs", torch.float32, (d.batch, d.n_heads, d.d_v)),
        _ptr(q_rot, "q_rot", torch.float32, (d.batch, d.n_heads, d.d_r)),
        _ptr(v_pool, "v_pool", dt, (pg.n_pages, d.n_groups, pg.page_rows, d.d_v)),
        _ptr(kr_pool, "kr_pool", dt, (pg.n_pages, pg.page_rows, d.d_r)),
        _ptr(block_table, "block_table", torch.int32, (d.batch, pg.max_pages)),
        _ptr(lens, "lens", torch.int32, (d.batch,)),
        _ptr(v_new, "v_new", dt, (d.batch, d.n_groups, d.d_v)),
        _ptr(kr_new, "kr_new", dt, (d.batch, d.d_r)),
        S, int(split_rows),
        _ptr(o_part, "o_part", torch.float32, (d.batch, d.n_heads, S, d.d_v)),
        _ptr(lse_part, "lse_part", torch.float32, (d.batch, d.n_heads, S)),
        _stream(stream))
    _check("gva_paged_decode_attention", st)


def make_paging(dims: GvaDims, page_rows: int, n_pages: int) -> GvaPaging:
    if dims.t_max % page_rows:
        raise ValueError("t_max must be a whole number of pages")
    return GvaPaging(int(page_rows), dims.t_max // int(page_rows), int(n_pages))


def to_pages(v_tiled: torch.Tensor, kr_tiled: torch.Tensor, block_table: torch.Tensor, paging: GvaPaging,
             fill=0.0):
    """Page pools holding tiled contiguous caches [B,G,T,d_v] / [B,T,d_r]
    (library layout) at the pages the block table names: page block (p, g)
    of the pool is the page_rows-row slice of stream (b, g) that
    block_table[b][t / page_rows] = p maps there.  Pages no entry names
    hold ``fill``.  Storage plumbing: a page boundary is a layout-tile
    boundary, so the slices move as they are."""
    B, G, T, dv = v_tiled.shape
    PR, MP = paging.page_rows, paging.max_pages
    v_pool = torch.full((paging.n_pages, G, PR, dv), fill, dtype=v_tiled.dtype, device=v_tiled.device)
    kr_pool = torch.full((paging.n_pages, PR, kr_tiled.shape[-1]), fill, dtype=kr_tiled.dtype,
                         device=kr_tiled.device)
    bt = block_table.to(torch.long).to(v_tiled.device)
    vb = v_tiled.reshape(B, G, MP, PR, dv).permute(0, 2, 1, 3, 4)      # [B, MP, G, PR, dv]
    kb = kr_tiled.reshape(B, MP, PR, kr_tiled.shape[-1])
    valid = (bt >= 0) & (bt < paging.n_pages)
    v_pool[bt[valid]] = vb[valid]
    kr_pool[bt[valid]] = kb[valid]
    return v_pool, kr_pool


def from_pages(v_pool: torch.Tensor, kr_pool: torch.Tensor, block_table: torch.Tensor, paging: GvaPaging):
    """Inverse of :func:`to_pages` for every block-table entry: the tiled
    contiguous caches [B,G,T,d_v] / [B,T,d_r] the pools hold."""
    n_pages, G, PR, dv = v_pool.shape
    B, MP = block_table.shape
    bt = block_table.to(torch.long).to(v_pool.device).clamp(0, n_pages - 1)
    v = v_pool[bt].permute(0, 2, 1, 3, 4).reshape(B, G, MP * PR, dv)
    kr = kr_pool[bt].reshape(B, MP * PR, kr_pool.shape[-1])
    return v.contiguous(), kr.contiguous()


def gva_pick_splits(dims: GvaDims, max_len: int = 0, total_len: int = 0, n_cu: int = 0,
                    chunked: bool = True) -> Tuple[int, int]:
    """(num_splits, split_rows); ``chunked=False`` asks for even splits only."""
    rows = ctypes.c_int32(-1)
    S = lib().gva_pick_splits(ctypes.byref(dims), int(max_len), int(total_len), int(n_cu),
                              ctypes.byref(rows) if chunked else None)
    return int(S), (int(rows.value) if chunked else 0)


def plan_for(dims: GvaDims, lens: torch.Tensor, n_cu: int = 0, chunked: bool = True) -> Tuple[int, int]:
    """gva_pick_splits for the lengths in ``lens`` (host copy)."""
    L = lens.detach().to("cpu", torch.int64).clamp(0, dims.t_max)
    return gva_pick_splits(dims, int(L.max()) if L.numel() else 0, int(L.sum()), n_cu, chunked)


def splits_for(dims: GvaDims, lens: torch.Tensor, n_cu: int = 0) -> int:
    """The even-split count gva_pick_splits picks for ``lens``."""
    return plan_for(dims, lens, n_cu, chunked=False)[0]


def device_cu_count(device=None) -> int:
    """Compute units of the current (or given) GPU."""
    return int(torch.cuda.get_device_properties(device if device is not None else
                                                torch.cuda.current_device()).multi_processor_count)


def gva_prefer_fused(dims: GvaDims, num_splits: int, split_rows: int = 0, n_cu: int = 0) -> bool:
    """The library's choice between the fused absorption and one
    gva_absorb_query launch for a decode launch of this plan."""
    return bool(lib().gva_prefer_fused(ctypes.byref(dims), int(num_splits), int(split_rows), int(n_cu)))


def prefer_fused(dims: GvaDims, num_splits: int, n_cu: int = 0, split_rows: int = 0) -> bool:
    """gva_prefer_fused (kept under its former name for callers)."""
    return gva_prefer_fused(dims, num_splits, split_rows, n_cu)


def gva_version() -> int:
    return int(lib().gva_version())


def tiled(x: torch.Tensor) -> torch.Tensor:
    """A row-major cache [..., T, D] rearranged into the library's tiled
    layout (same shape and dtype): tiles of 16 rows, inside a tile the
    16-byte row pieces ordered piece-major (include/gva.h).  Storage
    plumbing for callers that fill a cache themselves instead of through
    gva_append_kv."""
    *lead, T, D = x.shape
    P = 16 // x.element_size()
    if T % 16 or D % P:
        raise ValueError(f"tiled layout needs T % 16 == 0 and D % {P} == 0")
    y = x.reshape(*lead, T // 16, 16, D // P, P).transpose(-3, -2).contiguous()
    return y.reshape(*lead, T, D)


def untiled(y: torch.Tensor) -> torch.Tensor:
    """Inverse of :func:`tiled`: the row-major view of a tiled cache."""
    *lead, T, D = y.shape
    P = 16 // y.element_size()
    x = y.reshape(*lead, T // 16, D // P, 16, P).transpose(-3, -2).contiguous()
    return x.reshape(*lead, T, D)


class DecodeBuffers:
    """Device buffers for one decode step's split partials and outputs."""

    def __init__(self, dims: GvaDims, num_splits: int, device="cuda"):
        d = dims
        self.num_splits = int(num_splits)
        self.o_part = torch.empty(d.batch, d.n_heads, self.num_splits, d.d_v, dtype=torch.float32, device=device)
        self.lse_part = torch.empty(d.batch, d.n_heads, self.num_splits, dtype=torch.float32, device=device)
        self.o = torch.empty(d.batch, d.n_heads, d.d_v, dtype=torch.float32, device=device)
        self.lse = torch.empty(d.batch, d.n_heads, dtype=torch.float32, device=device)


def decode(dims: GvaDims, q, m, v_cache, kr_cache, lens, num_splits: int,
           bufs: Optional[DecodeBuffers] = None, fused: Optional[bool] = None,
           v_new=None, kr_new=None, split_rows: int = 0,
           stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Absorb + attention + combine for one step; returns (o, lse) fp32.

    ``fused`` runs the absorption inside the attention kernel; otherwise
    gva_absorb_query runs first and the attention kernel reads its output.
    ``v_new``/``kr_new`` are the current token's rows: the attention call
    stores them at cache row len-1 (as gva_append_kv would) and attends over
    them in the same launch.
    """
    S = int(num_splits)
    if fused is None:
        fused = gva_prefer_fused(dims, S, split_rows)
    if bufs is None or bufs.num_splits != S:
        bufs = DecodeBuffers(dims, S, device=v_cache.device)
        _in_use_on(stream, bufs.o_part, bufs.lse_part, bufs.o, bufs.lse)
    pend = dict(v_new=v_new, kr_new=kr_new if dims.d_r > 0 else None, split_rows=split_rows)
    if fused:
        gva_decode_attention(dims, v_cache, kr_cache, lens, S, bufs.o_part, bufs.lse_part,
                             q=q, m=m, stream=stream, **pend)
    else:
        q_abs = torch.empty(dims.batch, dims.n_heads, dims.d_v, dtype=torch.float32, device=v_cache.device)
        q_rot = torch.empty(dims.batch, dims.n_heads, dims.d_r, dtype=torch.float32, device=v_cache.device)
        _in_use_on(stream, q_abs, q_rot)
        gva_absorb_query(dims, q, m, lens, q_abs, q_rot, stream=stream)
        gva_decode_attention(dims, v_cache, kr_cache, lens, S, bufs.o_part, bufs.lse_part,
                             q_abs=q_abs, q_rot=q_rot if dims.d_r > 0 else None, stream=stream, **pend)
    if S == 1:   # a single split's partial is already the final result
        return bufs.o_part.view(dims.batch, dims.n_heads, dims.d_v), bufs.lse_part.view(dims.batch, dims.n_heads)
    gva_combine(dims, bufs.o_part, bufs.lse_part, S, bufs.o, bufs.lse, stream=stream)
    return bufs.o, bufs.lse


def gqa_decode(dims: GvaDims, q, k_cache, v_cache, lens, num_splits: int,
               bufs: Optional[DecodeBuffers] = None, split_rows: int = 0,
               stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Matched-GQA attention + combine for one step; returns (o, lse) fp32."""
    S = int(num_splits)
    if bufs is None or bufs.num_splits != S:
        bufs = DecodeBuffers(dims, S, device=v_cache.device)
        _in_use_on(stream, bufs.o_part, bufs.lse_part, bufs.o, bufs.lse)
    gva_gqa_decode_attention(dims, q, k_cache, v_cache, lens, S, bufs.o_part, bufs.lse_part,
                             split_rows=split_rows, stream=stream)
    if S == 1:
        return bufs.o_part.view(dims.batch, dims.n_heads, dims.d_v), bufs.lse_part.view(dims.batch, dims.n_heads)
    gva_combine(dims, bufs.o_part, bufs.lse_part, S, bufs.o, bufs.lse, stream=stream)
    return bufs.o, bufs.lse


def rope_decode(dims: GvaDims, q, m, v_cache, lens, num_splits: int,
                bufs: Optional[DecodeBuffers] = None, split_rows: int = 0,
                stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Ordinary-RoPE GVA attention + combine for one step; returns (o, lse) fp32."""
    S = int(num_splits)
    if bufs is None or bufs.num_splits != S:
        bufs = DecodeBuffers(dims, S, device=v_cache.device)
        _in_use_on(stream, bufs.o_part, bufs.lse_part, bufs.o, bufs.lse)
    gva_rope_decode_attention(dims, q, m, v_cache, lens, S, bufs.o_part, bufs.lse_part,
                              split_rows=split_rows, stream=stream)
    if S == 1:
        return bufs.o_part.view(dims.batch, dims.n_heads, dims.d_v), bufs.lse_part.view(dims.batch, dims.n_heads)
    gva_combine(dims, bufs.o_part, bufs.lse_part, S, bufs.o, bufs.lse, stream=stream)
    return bufs.o, bufs.lse


def prefill(dims: GvaDims, q, m, v_cache, kr_cache, lens, stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Absorb + causal attention for a prompt whose rows are the last
    q.shape[1] cached rows of each sequence; returns (o, lse) fp32."""
    d = dims
    B, N = q.shape[0], q.shape[1]
    dev = v_cache.device
    q_abs = torch.empty(B, N, d.n_heads, d.d_v, dtype=torch.float32, device=dev)
    q_rot = torch.empty(B, N, d.n_heads, d.d_r, dtype=torch.float32, device=dev)
    o = torch.empty(B, N, d.n_heads, d.d_v, dtype=torch.float32, device=dev)
    lse = torch.empty(B, N, d.n_heads, dtype=torch.float32, device=dev)
    _in_use_on(stream, q_abs, q_rot, o, lse)
    gva_prefill_absorb(d, N, q, m, lens, q_abs, q_rot, stream=stream)
    gva_prefill_attention(d, N, q_abs, q_rot, v_cache, kr_cache, lens, o, lse, stream=stream)
    return o, lse


def probe_read_bandwidth(nbytes: int = 2 << 30, reps: int = 10, stream=None) -> Tuple[float, int]:
    """Achievable HBM streaming-read GB/s (gva_probe_read): the best of a few
    workgroup counts over a ``nbytes`` buffer (larger than the 256 MB
    last-level cache).  Returns (GB/s, workgroups of the best run)."""
    buf = torch.empty(nbytes // 4, dtype=torch.int32, device="cuda").fill_(1)
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    st = _stream(stream)
    n_cu = torch.cuda.get_device_properties(buf.device).multi_processor_count
    best = (0.0, 0)
    for per_cu in (2, 4, 8, 16):
        wg = per_cu * n_cu
        _check("gva_probe_read", lib().gva_probe_read(ctypes.c_void_p(buf.data_ptr()), nbytes, wg,
                                                      ctypes.c_void_p(sink.data_ptr()), st))
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            lib().gva_probe_read(ctypes.c_void_p(buf.data_ptr()), nbytes, wg,
                                 ctypes.c_void_p(sink.data_ptr()), st)
        b.record()
        torch.cuda.synchronize()
        gbs = nbytes * reps / (a.elapsed_time(b) * 1e-3) / 1e9
        if gbs > best[0]:
            best = (gbs, wg)
    del buf
    return best


def probe_read_time(nbytes: int, copies: int = 2, reps: int = 50, stream=None) -> Tuple[float, int]:
    """Mean duration (ms) of one gva_probe_read launch over ``nbytes``, each
    launch reading the next of ``copies`` buffers (whose total can then
    exceed the 256 MB last-level cache), ``reps`` launches back to back
    between two events; the best of a few workgroup counts.  Returns
    (ms, workgroups)."""
    nbytes = (int(nbytes) + 15) // 16 * 16
    bufs = [torch.ones(nbytes // 4, dtype=torch.int32, device="cuda") for _ in range(max(1, int(copies)))]
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    st = _stream(stream)
    ev_stream = stream if isinstance(stream, torch.cuda.Stream) else torch.cuda.current_stream()
    n_cu = torch.cuda.get_device_properties(bufs[0].device).multi_processor_count
    best = (math.inf, 0)
    for per_cu in (1, 2, 4):
        wg = per_cu * n_cu
        launch = lambda i: _check("gva_probe_read", lib().gva_probe_read(
            ctypes.c_void_p(bufs[i % len(bufs)].data_ptr()), nbytes, wg, ctypes.c_void_p(sink.data_ptr()), st))
        for i in range(5):
            launch(i)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(ev_stream)
        for i in range(reps):
            launch(i)
        b.record(ev_stream)
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / reps
        if ms < best[0]:
            best = (ms, wg)
    del bufs
    return best


def paged_decode(dims: GvaDims, paging: GvaPaging, q, m, v_pool, kr_pool, block_table, lens, num_splits: int,
                 bufs: Optional[DecodeBuffers] = None, fused: Optional[bool] = None, v_new=None, kr_new=None,
                 split_rows: int = 0, stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """decode() on paged caches."""
    S = int(num_splits)
    if fused is None:
        fused = gva_prefer_fused(dims, S, split_rows)
    if bufs is None or bufs.num_splits != S:
        bufs = DecodeBuffers(dims, S, device=v_pool.device)
        _in_use_on(stream, bufs.o_part, bufs.lse_part, bufs.o, bufs.lse)
    pend = dict(v_new=v_new, kr_new=kr_new if dims.d_r > 0 else None, split_rows=split_rows)
    if fused:
        gva_paged_decode_attention(dims, paging, v_pool, kr_pool, block_table, lens, S, bufs.o_part,
                                   bufs.lse_part, q=q, m=m, stream=stream, **pend)
    else:
        q_abs = torch.empty(dims.batch, dims.n_heads, dims.d_v, dtype=torch.float32, device=v_pool.device)
        q_rot = torch.empty(dims.batch, dims.n_heads, dims.d_r, dtype=torch.float32, device=v_pool.device)
        _in_use_on(stream, q_abs, q_rot)
        gva_absorb_query(dims, q, m, lens, q_abs, q_rot, stream=stream)
        gva_paged_decode_attention(dims, paging, v_pool, kr_pool, block_table, lens, S, bufs.o_part,
                                   bufs.lse_part, q_abs=q_abs, q_rot=q_rot if dims.d_r > 0 else None,
                                   stream=stream, **pend)
    if S == 1:
        return bufs.o_part.view(dims.batch, dims.n_heads, dims.d_v), bufs.lse_part.view(dims.batch, dims.n_heads)
    gva_combine(dims, bufs.o_part, bufs.lse_part, S, bufs.o, bufs.lse, stream=stream)
    return bufs.o, bufs.lse
