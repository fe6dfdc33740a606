"""fp64 CPU oracle for the GVA decode step (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It wraps ``gva_oracle.c`` (plain C,
built with gcc) through ctypes and never touches the HIP library.

Every function takes CPU torch tensors in their storage dtype (float64,
float32 or bfloat16); the C code upcasts each element exactly to fp64.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Tuple

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gva_oracle.c")
# GVA_ORACLE_LIB names another build of gva_oracle.c to load (the
# sanitizer test runs the pins against an address/UB-sanitized build)
LIB_PATH = os.environ.get("GVA_ORACLE_LIB") or os.path.join(_HERE, "libgva_oracle.so")

_F64, _F32, _BF16 = 0, 1, 2
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (IEEE semantics, no fast-math)."""
    if force or not os.path.exists(LIB_PATH):
        tmp = LIB_PATH + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
               "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build(force=True)
        lib = ctypes.CDLL(LIB_PATH)
        P, I, D = ctypes.c_void_p, ctypes.c_int, ctypes.c_double
        lib.gva_oracle_round_bf16.argtypes = [D]
        lib.gva_oracle_round_bf16.restype = ctypes.c_uint16
        lib.gva_oracle_rope.argtypes = [P, I, ctypes.c_int64, D, P]
        lib.gva_oracle_rope.restype = None
        lib.gva_oracle_append.argtypes = [I, I, I, I, I, P, P, I, P, P, I, P, P, I, D]
        lib.gva_oracle_append.restype = I
        lib.gva_oracle_absorb.argtypes = [I, I, I, I, I, P, I, P, I, P, D, P, P]
        lib.gva_oracle_absorb.restype = None
        lib.gva_oracle_decode.argtypes = [I, I, I, I, I, I, I, P, I, P, I, P, P, I,
                                          P, P, P, D, D, I, P, P, P, P]
        lib.gva_oracle_decode.restype = None
        lib.gva_oracle_combine.argtypes = [I, I, I, P, P, P, P]
        lib.gva_oracle_combine.restype = None
        lib.gva_oracle_gqa_decode.argtypes = [I, I, I, I, I, I, I, P, I, P, P, I, P, D, I, P, P]
        lib.gva_oracle_gqa_decode.restype = None
        lib.gva_oracle_rope_decode.argtypes = [I, I, I, I, I, I, P, I, P, I, P, I, P, D, D,
                                               ctypes.c_int64, I, P, P]
        lib.gva_oracle_rope_decode.restype = None
        lib.gva_oracle_prefill.argtypes = [I, I, I, I, I, I, I, I, P, I, P, I, P, P, I, P, D, D, I, P, P]
        lib.gva_oracle_prefill.restype = None
        lib.gva_oracle_max_threads.argtypes = []
        lib.gva_oracle_max_threads.restype = I
        _lib = lib
    return _lib


def _code(t: torch.Tensor) -> int:
    return {torch.float64: _F64, torch.float32: _F32, torch.bfloat16: _BF16}[t.dtype]


def _cpu(t: torch.Tensor) -> torch.Tensor:
    if t.device.type != "cpu":
        raise ValueError("oracle inputs must be CPU tensors")
    return t.contiguous()


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def max_threads() -> int:
    return _load().gva_oracle_max_threads()


def round_bf16_bits(x: float) -> int:
    """Nearest bfloat16 to the double ``x`` (ties to even), as 16 raw bits."""
    return int(_load().gva_oracle_round_bf16(float(x)))


def rope(x: torch.Tensor, pos: int, base: float = 10000.0) -> torch.Tensor:
    """RoPE of one row (x R_pos^T), fp64."""
    xd = _cpu(x.to(torch.float64).reshape(-1))
    y = torch.empty_like(xd)
    _load().gva_oracle_rope(_ptr(xd), xd.numel(), int(pos), float(base), _ptr(y))
    return y


def append(v_cache: torch.Tensor, kr_cache: torch.Tensor, v_new: torch.Tensor,
           kr_new: torch.Tensor, seq: torch.Tensor, pos: torch.Tensor,
           rope_base: float = 10000.0) -> int:
    """Write new rows into the caches in place; returns the number skipped."""
    B, G, T, dv = v_cache.shape
    dr = kr_cache.shape[-1]
    for t in (v_cache, kr_cache):
        if not t.is_contiguous() or t.device.type != "cpu":
            raise ValueError("caches must be contiguous CPU tensors")
    if v_new.dtype != kr_new.dtype:
        raise ValueError("v_new and kr_new must share a dtype")
    vn, kn = _cpu(v_new), _cpu(kr_new)
    s32, p32 = _cpu(seq.to(torch.int32)), _cpu(pos.to(torch.int32))
    n = s32.numel()
    return _load().gva_oracle_append(B, G, T, dv, dr, _ptr(v_cache), _ptr(kr_cache),
                                     _code(v_cache), _ptr(vn), _ptr(kn), _code(vn),
                                     _ptr(s32), _ptr(p32), n, float(rope_base))


def absorb(q: torch.Tensor, m: torch.Tensor, lens: torch.Tensor, d_r: int,
           rope_base: float = 10000.0) -> Tuple[torch.Tensor, torch.Tensor]:
    """Absorbed query q~ [B,H,d_v] and rotated positional query [B,H,d_r], fp64."""
    B, H, w = q.shape
    Hm, dv, dc = m.shape
    assert Hm == H and w == dc + d_r
    qc, mc, lc = _cpu(q), _cpu(m), _cpu(lens.to(torch.int32))
    qa = torch.empty(B, H, dv, dtype=torch.float64)
    qr = torch.empty(B, H, max(d_r, 0), dtype=torch.float64)
    _load().gva_oracle_absorb(B, H, dv, dc, d_r, _ptr(qc), _code(qc), _ptr(mc), _code(mc),
                              _ptr(lc), float(rope_base), _ptr(qa), _ptr(qr))
    return qa, qr


def decode(q: torch.Tensor, m: torch.Tensor, v: torch.Tensor, kr: torch.Tensor,
           lens: torch.Tensor, scale: float = 0.0, rope_base: float = 10000.0,
           t_begin: Optional[torch.Tensor] = None, t_end: Optional[torch.Tensor] = None,
           n_threads: int = 0, want_query: bool = False):
    """One GVA decode step in fp64: returns (o [B,H,d_v], lse [B,H]).

    With ``want_query`` also returns the absorbed and rotated queries.
    ``t_begin``/``t_end`` restrict every sequence to a row range (a split).
    """
    B, G, T, dv = v.shape
    H = q.shape[1]
    dr = kr.shape[-1]
    dc = m.shape[2]
    if q.shape != (B, H, dc + dr) or m.shape != (H, dv, dc) or kr.shape[:2] != (B, T):
        raise ValueError("inconsistent shapes")
    if H % G:
        raise ValueError("H must be a multiple of G")
    if v.dtype != kr.dtype:
        raise ValueError("v and kr must share a dtype")
    qc, mc, vc, kc = _cpu(q), _cpu(m), _cpu(v), _cpu(kr)
    lc = _cpu(lens.to(torch.int32))
    tb = None if t_begin is None else _cpu(t_begin.to(torch.int32))
    te = None if t_end is None else _cpu(t_end.to(torch.int32))
    o = torch.empty(B, H, dv, dtype=torch.float64)
    lse = torch.empty(B, H, dtype=torch.float64)
    qa = torch.empty(B, H, dv, dtype=torch.float64) if want_query else None
    qr = torch.empty(B, H, max(dr, 1), dtype=torch.float64) if want_query else None
    _load().gva_oracle_decode(B, H, G, T, dv, dc, dr, _ptr(qc), _code(qc), _ptr(mc), _code(mc),
                              _ptr(vc), _ptr(kc), _code(vc), _ptr(lc), _ptr(tb), _ptr(te),
                              float(scale), float(rope_base), int(n_threads),
                              _ptr(o), _ptr(lse), _ptr(qa), _ptr(qr))
    if want_query:
        return o, lse, qa, qr[..., :dr]
    return o, lse


def combine(o_part: torch.Tensor, lse_part: torch.Tensor) -> Tuple[torch.Tensor, torch.Tensor]:
    """Log-sum-exp merge of split partials: o_part [..., S, d_v], lse_part [..., S]."""
    lead = lse_part.shape[:-1]
    S = lse_part.shape[-1]
    dv = o_part.shape[-1]
    op = _cpu(o_part.to(torch.float64)).reshape(-1, S, dv)
    lp = _cpu(lse_part.to(torch.float64)).reshape(-1, S)
    rows = lp.shape[0]
    o = torch.empty(rows, dv, dtype=torch.float64)
    lse = torch.empty(rows, dtype=torch.float64)
    _load().gva_oracle_combine(rows, S, dv, _ptr(op), _ptr(lp), _ptr(o), _ptr(lse))
    return o.reshape(*lead, dv), lse.reshape(lead)


def gqa_decode(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, lens: torch.Tensor,
               d_k: Optional[int] = None, scale: float = 0.0, n_threads: int = 0):
    """Matched GQA decode in fp64 with an explicit key cache k [B,G,T,d_k]."""
    B, G, T, dv = v.shape
    H = q.shape[1]
    dk = k.shape[-1] if d_k is None else d_k
    qc, kc, vc = _cpu(q), _cpu(k), _cpu(v)
    if kc.dtype != vc.dtype:
        raise ValueError("k and v must share a dtype")
    lc = _cpu(lens.to(torch.int32))
    o = torch.empty(B, H, dv, dtype=torch.float64)
    lse = torch.empty(B, H, dtype=torch.float64)
    _load().gva_oracle_gqa_decode(B, H, G, T, dv, dk, qc.shape[-1], _ptr(qc), _code(qc),
                                  _ptr(kc), _ptr(vc), _code(vc), _ptr(lc), float(scale),
                                  int(n_threads), _ptr(o), _ptr(lse))
    return o, lse


def rope_decode(q: torch.Tensor, m: torch.Tensor, v: torch.Tensor, lens: torch.Tensor,
                rope_base: float = 10000.0, scale: float = 0.0, shift: int = 0, n_threads: int = 0):
    """GVA without decoupled RoPE in fp64: keys reconstructed (v M_h) and
    rotated over their full width d_c, query rotated at L-1.  q [B,H,d_c]."""
    B, G, T, dv = v.shape
    H, dc = q.shape[1], q.shape[2]
    qc, mc, vc = _cpu(q), _cpu(m), _cpu(v)
    lc = _cpu(lens.to(torch.int32))
    o = torch.empty(B, H, dv, dtype=torch.float64)
    lse = torch.empty(B, H, dtype=torch.float64)
    _load().gva_oracle_rope_decode(B, H, G, T, dv, dc, _ptr(qc), _code(qc), _ptr(mc), _code(mc),
                                   _ptr(vc), _code(vc), _ptr(lc), float(scale), float(rope_base),
                                   int(shift), int(n_threads), _ptr(o), _ptr(lse))
    return o, lse


def prefill(q: torch.Tensor, m: torch.Tensor, v: torch.Tensor, kr: torch.Tensor, lens: torch.Tensor,
            scale: float = 0.0, rope_base: float = 10000.0, n_threads: int = 0):
    """Causal prefill in fp64: q [B, N, H, d_c+d_r] holds the queries of each
    sequence's last N cached rows (query i at position lens-N+i).
    Returns o [B, N, H, d_v], lse [B, N, H]."""
    B, N, H, W = q.shape
    _, G, T, dv = v.shape
    dr = kr.shape[-1]
    dc = W - dr
    if m.shape != (H, dv, dc) or kr.shape[:2] != (B, T) or H % G:
        raise ValueError("inconsistent shapes")
    qc, mc, vc, kc = _cpu(q), _cpu(m), _cpu(v), _cpu(kr)
    if kc.dtype != vc.dtype:
        raise ValueError("v and kr caches must share a dtype")
    lc = _cpu(lens.to(torch.int32))
    o = torch.empty(B, N, H, dv, dtype=torch.float64)
    lse = torch.empty(B, N, H, dtype=torch.float64)
    _load().gva_oracle_prefill(B, N, H, G, T, dv, dc, dr, _ptr(qc), _code(qc), _ptr(mc), _code(mc),
                               _ptr(vc), _ptr(kc), _code(vc), _ptr(lc), float(scale), float(rope_base),
                               int(n_threads), _ptr(o), _ptr(lse))
    return o, lse
