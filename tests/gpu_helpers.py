"""Shared plumbing for the GPU parity tests: upload seeded inputs, run the
HIP path through the C ABI, run the oracle on the same CPU tensors."""

from __future__ import annotations

import sys
from typing import Dict, Optional

import torch

import gva_inputs
from paper_2609_13285_amd import gva

# max-abs error gates for the attention output
TOL = {"f32": 2e-3, "bf16": 1.5e-2}


def note(msg: str):
    """Name the case before a GPU step, so a crash still says what ran."""
    sys.stdout.write(f"[gpu] {msg}\n")
    sys.stdout.flush()


def dims_of(w: gva_inputs.Workload) -> gva.GvaDims:
    return gva.make_dims(w.batch, w.n_heads, w.n_groups, w.d_v, w.d_c, w.d_r, w.t_max,
                         w.dtype, w.rope_base)


def upload(inp: Dict[str, torch.Tensor]) -> Dict[str, torch.Tensor]:
    """Copy the inputs to the GPU; the caches go in the library's tiled layout."""
    out = {}
    for k, v in inp.items():
        out[k] = gva.tiled(v).cuda() if k in ("v", "kr", "k_gqa") else v.cuda()
    return out


def run_decode(w, dev: Dict[str, torch.Tensor], S: int, fused: bool = True, lens=None,
               split_rows: int = 0):
    """Absorb + attention + combine on the GPU; returns CPU tensors
    (o, lse, o_part, lse_part)."""
    d = dims_of(w)
    L = dev["lens"] if lens is None else lens
    bufs = gva.DecodeBuffers(d, S)
    o, lse = gva.decode(d, dev["q"], dev["m"], dev["v"], dev["kr"], L, S, bufs=bufs, fused=fused,
                        split_rows=split_rows)
    torch.cuda.synchronize()
    return o.cpu(), lse.cpu(), bufs.o_part.cpu(), bufs.lse_part.cpu()


def max_abs(a: torch.Tensor, b: torch.Tensor) -> float:
    return float((a.double() - b.double()).abs().max()) if a.numel() else 0.0


def lse_err(a: torch.Tensor, b: torch.Tensor) -> float:
    """max |a - b| over entries where the reference is finite; -inf must match."""
    a, b = a.double(), b.double()
    fin = torch.isfinite(b)
    assert torch.equal(torch.isneginf(a), torch.isneginf(b)), "empty rows disagree"
    return float((a[fin] - b[fin]).abs().max()) if fin.any() else 0.0


def sub_batch(inp: Dict[str, torch.Tensor], idx) -> Dict[str, torch.Tensor]:
    """The per-sequence tensors restricted to the sequences in idx (CPU)."""
    idx = torch.as_tensor(idx, dtype=torch.long)
    out = dict(inp)
    for k in ("q", "v", "kr", "lens", "v_new", "kr_new", "k_gqa"):
        if k in inp:
            out[k] = inp[k].index_select(0, idx).contiguous()
    return out
