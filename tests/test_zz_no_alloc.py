"""gva_decode_step_static: the decode step for callers that cannot allocate
device memory, its workspace in the library's static per-device scratch
buffer.  Two calls in a row through the C ABI, the second with a smaller
input, each checked bit for bit against gva_decode_step with a caller
workspace (the same launches) and against the fp64 oracle within the gates;
then the first shape again, so a smaller call's leftovers in the shared
buffer are shown not to matter."""

import pytest
import torch

import gva_inputs
import oracle
from gpu_helpers import TOL, dims_of, lse_err, max_abs, note, upload
from paper_2609_13285_amd import gva

pytestmark = pytest.mark.gpu

CASES = [
    # ragged lengths, bounded chunks over a grid past two workgroups per CU:
    # the absorbed queries and the split partials both live in the scratch
    (gva_inputs.Workload("static_ragged", 40, 2048, 16, 2, 128, 128, 16), 8, 256, 31),
    # smaller: three even splits, the absorption fused (partials only)
    (gva_inputs.Workload("static_small", 6, 512, 8, 2, 64, 64, 16), 3, 0, 37),
]


def _one(w, S, rows, seed):
    g = torch.Generator().manual_seed(seed)
    lens = torch.randint(1, w.t_max + 1, (w.batch,), generator=g, dtype=torch.int32)
    lens[0] = 0
    lens[-1] = w.t_max
    inp = gva_inputs.make_inputs(w, seed, lens=lens)
    d = dims_of(w)
    dev = upload(inp)
    v2, kr2 = dev["v"].clone(), dev["kr"].clone()
    need = gva.gva_decode_workspace_size(d, S, rows)
    assert 0 < need <= gva.GVA_STATIC_SCRATCH_BYTES
    o = torch.full((w.batch, w.n_heads, w.d_v), float("nan"), device="cuda")
    lse = torch.full((w.batch, w.n_heads), float("nan"), device="cuda")
    note(f"static-scratch step {w.name} S={S} rows={rows} (workspace {need} B)")
    gva.gva_decode_step_static(d, dev["q"], dev["m"], dev["v"], dev["kr"], dev["lens"], S, o, lse,
                               v_new=dev["v_new"], kr_new=dev["kr_new"], split_rows=rows)
    ws = gva.workspace_for(d, S, rows)
    o2 = torch.empty_like(o)
    lse2 = torch.empty_like(lse)
    gva.gva_decode_step(d, dev["q"], dev["m"], v2, kr2, dev["lens"], S, o2, lse2, workspace=ws,
                        v_new=dev["v_new"], kr_new=dev["kr_new"], split_rows=rows)
    torch.cuda.synchronize()
    assert torch.equal(o, o2) and torch.equal(lse, lse2), w.name
    assert torch.equal(dev["v"], v2) and torch.equal(dev["kr"], kr2), w.name
    v_ref, k_ref = inp["v"].clone(), inp["kr"].clone()
    live = lens > 0
    oracle.append(v_ref, k_ref, inp["v_new"][live], inp["kr_new"][live],
                  torch.arange(w.batch, dtype=torch.int32)[live], (lens - 1)[live].to(torch.int32), w.rope_base)
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], v_ref, k_ref, lens, rope_base=w.rope_base)
    err, lerr = max_abs(o.cpu(), o_ref), lse_err(lse.cpu(), lse_ref)
    note(f"static-scratch step {w.name}: max|o-o_ref| = {err:.3e}  max|lse-lse_ref| = {lerr:.3e}")
    assert err <= TOL[w.dtype] and err <= 1e-4 and lerr <= 1e-3, (w.name, err, lerr)


def test_static_scratch_step_two_calls_then_the_first_again():
    for w, S, rows, seed in CASES + CASES[:1]:
        _one(w, S, rows, seed)
