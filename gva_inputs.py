"""Seeded synthetic inputs for the GVA decode step.

This module only draws random numbers and casts them to the storage dtype.
It holds none of the attention arithmetic, so both the fp64 oracle and the
HIP path can consume its tensors without sharing any method code.

Shapes follow the paper's decode state (Algorithm 1; Section 3.3 and 3.4):

* ``q``      [B, H, d_c + d_r]  per-head query, content slice first, then the
                                 positional slice (unrotated)
* ``v``      [B, G, T_max, d_v] grouped value cache
* ``kr``     [B, T_max, d_r]     shared positional key cache, already rotated
                                 (rotation keeps N(0, I) invariant, so a
                                 standard-normal draw is a valid stored cache)
* ``m``      [H, d_v, d_c]       per-head key-reconstruction maps M_h,
                                 N(0, 1/d_v) as in the scale-matched init
                                 (Appendix A, eq. scale-init with unit sigmas)
* ``lens``   [B] int32           cached length per sequence (query at len-1)
* ``v_new``  [B, G, d_v]         the decode step's new value rows
* ``kr_new`` [B, d_r]            the decode step's new positional key rows,
                                 unrotated (x W_r in eq. krope)
* ``k_gqa``  [B, G, T_max, d_v]  explicit key cache for the matched-GQA
                                 comparison (ragged workload only)

Draw order from one ``torch.Generator`` seeded with ``seed``: q, v, kr, m,
lens, k_gqa (if any), v_new, kr_new.  bf16 workloads cast each fp32 draw
once with round-to-nearest-even.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional

import torch

__all__ = ["Workload", "WORKLOADS", "make_inputs", "prefill_queries", "workload"]


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    t_max: int
    n_heads: int
    n_groups: int
    d_v: int
    d_c: int
    d_r: int
    dtype: str = "bf16"          # storage dtype: "f32" or "bf16"
    lengths: str = "full"        # "full" | "uniform_half" | "log_uniform"
    len_min: int = 0             # lower end for "log_uniform"
    rope_base: float = 10000.0
    gqa: bool = False            # also draw an explicit GQA key cache

    @property
    def heads_per_group(self) -> int:
        return self.n_heads // self.n_groups

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS: Dict[str, Workload] = {
    # Tiny fp32 decode step: B1, T256, H8, G2, d 64/64/16.
    "tiny_f32": Workload("tiny_f32", 1, 256, 8, 2, 64, 64, 16, dtype="f32"),
    # 350M-model head shapes: B8, T2048, H16, G4, d 64/64/16, bf16.
    "gva350m_b8_t2k": Workload("gva350m_b8_t2k", 8, 2048, 16, 4, 64, 64, 16),
    # Bandwidth headline: B32, T8192, H32, G8, d 128/128/16, bf16.
    "b32_t8k": Workload("b32_t8k", 32, 8192, 32, 8, 128, 128, 16),
    # The paper's wider positional slice (d_r = 24) at the bandwidth-headline
    # shape: B32, T8192, H32, G8, d 128/128/24, bf16.
    "b32_t8k_dr24": Workload("b32_t8k_dr24", 32, 8192, 32, 8, 128, 128, 24),
    # Long context: B4, T<=131072 (lengths U[T/2, T]), H32, G8, d 128/128/32.
    "long_b4_t128k": Workload("long_b4_t128k", 4, 131072, 32, 8, 128, 128, 32,
                              lengths="uniform_half"),
    # Ragged mixed batch: B64, lengths log-uniform in [128, 32768], H16, G2.
    "ragged_b64": Workload("ragged_b64", 64, 32768, 16, 2, 128, 128, 16,
                           lengths="log_uniform", len_min=128, gqa=True),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def _torch_dtype(name: str) -> torch.dtype:
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def _draw_lengths(w: Workload, g: torch.Generator) -> torch.Tensor:
    if w.lengths == "full":
        return torch.full((w.batch,), w.t_max, dtype=torch.int32)
    if w.lengths == "uniform_half":
        # integers uniform on [T/2, T], both ends included
        return torch.randint(w.t_max // 2, w.t_max + 1, (w.batch,), generator=g,
                             dtype=torch.int64).to(torch.int32)
    if w.lengths == "log_uniform":
        lo, hi = math.log(w.len_min), math.log(w.t_max)
        u = torch.rand((w.batch,), generator=g, dtype=torch.float64)
        n = torch.exp(lo + u * (hi - lo)).round()
        return n.clamp(w.len_min, w.t_max).to(torch.int32)
    raise ValueError(f"unknown length recipe {w.lengths!r}")


def make_inputs(w: Workload, seed: int, lens: Optional[torch.Tensor] = None) -> Dict[str, torch.Tensor]:
    """Draw every tensor of one decode step on the CPU.

    ``lens`` overrides the drawn lengths (the draw still happens, so the
    streams of later tensors do not move).
    """
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    B, T, H, G = w.batch, w.t_max, w.n_heads, w.n_groups
    dv, dc, dr = w.d_v, w.d_c, w.d_r
    dt = _torch_dtype(w.dtype)

    def normal(*shape, std=1.0):
        x = torch.randn(shape, generator=g, dtype=torch.float32)
        if std != 1.0:
            x.mul_(std)
        return x.to(dt)

    out: Dict[str, torch.Tensor] = {}
    out["q"] = normal(B, H, dc + dr)
    out["v"] = normal(B, G, T, dv)
    out["kr"] = normal(B, T, dr)
    out["m"] = normal(H, dv, dc, std=1.0 / math.sqrt(dv))
    drawn = _draw_lengths(w, g)
    out["lens"] = drawn if lens is None else lens.to(torch.int32).clone()
    if w.gqa:
        out["k_gqa"] = normal(B, G, T, dv)
    out["v_new"] = normal(B, G, dv)
    out["kr_new"] = normal(B, dr)
    return out


def gqa_keys(w: Workload, seed: int) -> torch.Tensor:
    """The matched-GQA baseline's explicit key cache, [B, G, T, d_v] in the
    storage dtype, N(0, 1) like the value cache, from its own generator
    seeded with ``seed``: for workloads whose draw (make_inputs) has none."""
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed) + 104729)
    x = torch.randn((w.batch, w.n_groups, w.t_max, w.d_v), generator=g, dtype=torch.float32)
    return x.to(_torch_dtype(w.dtype))


def prefill_queries(w: Workload, seed: int, n_new: int, gqa: bool = False) -> torch.Tensor:
    """A prompt's queries, [B, n_new, H, d_c + d_r] in the storage dtype
    (or, with ``gqa``, the matched-GQA queries [B, n_new, H, d_v] in fp32),
    N(0, 1) from their own generator seeded with ``seed``."""
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed) + 7919)
    width = w.d_v if gqa else w.d_c + w.d_r
    x = torch.randn((w.batch, int(n_new), w.n_heads, width), generator=g, dtype=torch.float32)
    return x if gqa else x.to(_torch_dtype(w.dtype))
