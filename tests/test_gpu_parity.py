"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on
the same seeded inputs, element by element.

Gates (max-abs on the attention output): 2e-3 for fp32 storage, 1.5e-2 for
bf16 storage.  The kernels keep the absorbed query and the softmax weights
as bf16 high+low pairs with fp32 accumulation, so the observed error is far
below the gate; ``QUALITY`` pins that margin so an accuracy regression
fails loudly even while it is still inside the gate.
"""

import math

import pytest
import torch

import gva_inputs
import oracle
from splits import split_bounds
from gpu_helpers import TOL, dims_of, lse_err, max_abs, note, run_decode, sub_batch, upload
from paper_2609_13285_amd import gva

pytestmark = pytest.mark.gpu

# expected accuracy of this implementation (well inside the gates)
QUALITY = {"f32": 2e-5, "bf16": 1e-4}


def _check(w, o, lse, o_ref, lse_ref, label):
    err = max_abs(o, o_ref)
    lerr = lse_err(lse, lse_ref)
    note(f"{label}: max|o-o_ref| = {err:.3e}  max|lse-lse_ref| = {lerr:.3e}")
    assert err <= TOL[w.dtype], (label, err)
    assert err <= QUALITY[w.dtype], (label, err)
    assert lerr <= 1e-3, (label, lerr)


# ------------------------------------------------------------ small workloads
@pytest.mark.parametrize("name", ["tiny_f32", "gva350m_b8_t2k"])
@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("fused", [True, False])
def test_decode_matches_oracle(name, seed, fused):
    w = gva_inputs.workload(name)
    inp = gva_inputs.make_inputs(w, seed)
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], inp["v"], inp["kr"], inp["lens"],
                                   rope_base=w.rope_base)
    dev = upload(inp)
    S = gva.splits_for(dims_of(w), inp["lens"])
    for splits in sorted({1, 3, S}):
        note(f"{name} seed={seed} fused={fused} S={splits}")
        o, lse, _, _ = run_decode(w, dev, splits, fused=fused)
        _check(w, o, lse, o_ref, lse_ref, f"{name}/s{seed}/S{splits}/fused={fused}")


@pytest.mark.parametrize("name", ["tiny_f32", "gva350m_b8_t2k"])
def test_split_partials_match_oracle(name):
    w = gva_inputs.workload(name)
    inp = gva_inputs.make_inputs(w, 5, lens=torch.tensor([w.t_max - 7] + [w.t_max // 3] * (w.batch - 1)))
    dev = upload(inp)
    for S, rows in ((2, 0), (7, 0), (5, 64), (3, 96)):
        note(f"{name} partials S={S} split_rows={rows}")
        _, _, o_part, lse_part = run_decode(w, dev, S, split_rows=rows)
        begins, ends = split_bounds(inp["lens"], S, tile=32, split_rows=rows)
        for s in range(S):
            o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], inp["v"], inp["kr"], inp["lens"],
                                           t_begin=begins[s], t_end=ends[s])
            # an empty split past the first writes only its lse
            live = (ends[s] > begins[s]) | (s == 0)
            err = max_abs(o_part[live][:, :, s], o_ref[live])
            assert err <= QUALITY[w.dtype], (S, rows, s, err)
            assert lse_err(lse_part[:, :, s], lse_ref) <= 1e-3


def test_random_shapes_sweep():
    # 40 seeded random cases over the supported shape space: H/G, G, d_v,
    # d_c (incl. widths that are not powers of two), d_r (incl. 0), batch,
    # capacity, lengths (0, 1, capacity and random), even and bounded-chunk
    # splits, fused and separate absorption, bf16 and fp32 storage
    rng = torch.Generator().manual_seed(2609)
    pick = lambda xs: xs[int(torch.randint(len(xs), (1,), generator=rng))]
    for case in range(40):
        dtype = "f32" if case % 8 == 7 else "bf16"
        hpg, G = pick([1, 2, 4, 8]), pick([1, 2, 3])
        dv, dc = pick([64, 128]), pick([32, 64, 96, 128, 160, 224, 256])
        dr = pick([0, 8, 16, 24, 32, 40, 48, 64])
        B, T = pick([1, 2, 3, 5]), 16 * pick([2, 3, 7, 16, 25])
        w = gva_inputs.Workload("sweep", B, T, hpg * G, G, dv, dc, dr, dtype=dtype)
        lens = torch.randint(0, T + 1, (B,), generator=rng, dtype=torch.int32)
        lens[0] = pick([0, 1, T, int(lens[0])])
        S = pick([1, 2, 3, 5])
        rows = pick([0, 0, 32, 64, 96])
        fused = bool(pick([True, False]))
        inp = gva_inputs.make_inputs(w, 100 + case, lens=lens)
        o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], inp["v"], inp["kr"], inp["lens"],
                                       rope_base=w.rope_base)
        label = (f"sweep {case}: {dtype} H{hpg * G} G{G} dv{dv} dc{dc} dr{dr} B{B} T{T} "
                 f"lens={lens.tolist()} S{S} rows{rows} fused={fused}")
        note(label)
        o, lse, _, _ = run_decode(w, upload(inp), S, fused=fused, split_rows=rows)
        _check(w, o, lse, o_ref, lse_ref, label)


@pytest.mark.parametrize("fused", [True, False])
def test_f32_query_rows_not_16_byte_aligned(fused):
    # fp32 storage takes any d_c: with d_c + d_r odd the query rows are not
    # 16-byte aligned and the absorption reads them element by element
    for dc, dr in ((37, 8), (64, 4), (5, 0)):
        w = gva_inputs.Workload("f32_odd", 3, 96, 8, 2, 64, dc, dr, dtype="f32")
        lens = torch.tensor([96, 41, 1], dtype=torch.int32)
        inp = gva_inputs.make_inputs(w, 61, lens=lens)
        o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], inp["v"], inp["kr"], inp["lens"],
                                       rope_base=w.rope_base)
        for S in (1, 2):
            label = f"f32 dc{dc} dr{dr} fused={fused} S{S}"
            note(label)
            o, lse, _, _ = run_decode(w, upload(inp), S, fused=fused)
            _check(w, o, lse, o_ref, lse_ref, label)


# ------------------------------------------------------------------ shapes
SHAPES = [
    # (H, G, d_v, d_c, d_r)
    (8, 8, 64, 64, 16),     # H/G = 1 (MHA-shaped)
    (8, 4, 128, 64, 8),     # H/G = 2, d_c != d_v
    (16, 4, 64, 96, 24),    # H/G = 4, d_r = 24 (the paper's wider variant)
    (16, 2, 128, 128, 32),  # H/G = 8
    (8, 1, 128, 32, 64),    # MQA-shaped, two positional K-chunks
    (16, 4, 128, 160, 0),   # value-only GVA (no positional slice)
    (8, 2, 64, 128, 40),
]


@pytest.mark.parametrize("H,G,dv,dc,dr", SHAPES)
def test_shape_sweep_bf16(H, G, dv, dc, dr):
    w = gva_inputs.Workload("sweep", 3, 304, H, G, dv, dc, dr)
    lens = torch.tensor([300, 1, 97], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 11, lens=lens)
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], inp["v"], inp["kr"], inp["lens"])
    dev = upload(inp)
    for S in (1, 4):
        for fused in (True, False):
            note(f"sweep H={H} G={G} dv={dv} dc={dc} dr={dr} S={S} fused={fused}")
            o, lse, _, _ = run_decode(w, dev, S, fused=fused)
            _check(w, o, lse, o_ref, lse_ref, f"sweep/{H}/{G}/{dv}/{dc}/{dr}/S{S}")


@pytest.mark.parametrize("H,G,dv,dc,dr", [(8, 2, 64, 64, 16), (6, 3, 40, 24, 8), (8, 1, 256, 48, 64)])
def test_shape_sweep_f32(H, G, dv, dc, dr):
    w = gva_inputs.Workload("sweep32", 2, 208, H, G, dv, dc, dr, dtype="f32")
    lens = torch.tensor([200, 65], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 13, lens=lens)
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], inp["v"], inp["kr"], inp["lens"])
    dev = upload(inp)
    for S in (1, 3):
        note(f"f32 sweep H={H} G={G} dv={dv} dc={dc} dr={dr} S={S}")
        o, lse, _, _ = run_decode(w, dev, S, fused=True)
        _check(w, o, lse, o_ref, lse_ref, f"f32/{H}/{G}/{dv}/{dc}/{dr}/S{S}")


# -------------------------------------------------------------- edge cases
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_ragged_and_degenerate_lengths(dtype):
    T = 144
    w = gva_inputs.Workload("edge", 10, T, 8, 2, 64, 64, 16, dtype=dtype)
    # empty, single row, tile boundaries, full, beyond capacity (clamped), negative
    lens = torch.tensor([0, 1, 31, 32, 33, 64, 65, T, T + 50, -3], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 17, lens=lens)
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], inp["v"], inp["kr"], inp["lens"])
    dev = upload(inp)
    for S in (1, 2, 5, 64):
        note(f"edge lengths {dtype} S={S}")
        o, lse, _, _ = run_decode(w, dev, S)
        _check(w, o, lse, o_ref, lse_ref, f"edge/{dtype}/S{S}")
        for b in (0, 9):        # empty sequences: o = 0, lse = -inf
            assert torch.all(o[b] == 0) and torch.all(torch.isneginf(lse[b]))


def test_uninitialised_rows_past_length_are_never_used():
    # rows beyond each length hold NaN; they must not leak into the result
    w = gva_inputs.Workload("nan_tail", 2, 96, 8, 2, 128, 128, 16)
    lens = torch.tensor([45, 77], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 19, lens=lens)
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], inp["v"], inp["kr"], inp["lens"])
    for b, L in enumerate(lens.tolist()):
        inp["v"][b, :, L:] = float("nan")
        inp["kr"][b, L:] = float("nan")
    dev = upload(inp)
    for S in (1, 3):
        note(f"nan tail S={S}")
        o, lse, _, _ = run_decode(w, dev, S)
        assert torch.isfinite(o).all()
        _check(w, o, lse, o_ref, lse_ref, f"nan_tail/S{S}")


def test_split_count_invariance_and_determinism():
    w = gva_inputs.workload("gva350m_b8_t2k")
    inp = gva_inputs.make_inputs(w, 23)
    dev = upload(inp)
    note("split invariance")
    # up to GVA_MAX_SPLITS: 256 even splits of 2048 rows are 64 of 32 rows
    # and 192 empty ones
    outs = {S: run_decode(w, dev, S)[0] for S in (1, 2, 7, 64, gva.GVA_MAX_SPLITS)}
    outs["chunks"] = run_decode(w, dev, 64, split_rows=32)[0]     # 64 bounded chunks of 32 rows
    for S, o in outs.items():
        assert max_abs(o, outs[1]) <= 2 * QUALITY["bf16"], S
    again = run_decode(w, dev, 7)[0]
    assert torch.equal(again, outs[7])          # bitwise deterministic
    again = run_decode(w, dev, 64, split_rows=32)[0]
    assert torch.equal(again, outs["chunks"])


# ------------------------------------------------- absorb, append, combine
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_absorb_query_matches_oracle(dtype):
    w = gva_inputs.Workload("absorb", 4, 4096, 16, 4, 128, 96, 32, dtype=dtype)
    lens = torch.tensor([1, 17, 4096, 2500], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 29, lens=lens)
    qa_ref, qr_ref = oracle.absorb(inp["q"], inp["m"], inp["lens"], d_r=w.d_r)
    dev = upload(inp)
    qa = torch.empty(4, 16, 128, dtype=torch.float32, device="cuda")
    qr = torch.empty(4, 16, 32, dtype=torch.float32, device="cuda")
    note(f"absorb {dtype}")
    gva.gva_absorb_query(dims_of(w), dev["q"], dev["m"], dev["lens"], qa, qr)
    torch.cuda.synchronize()
    scale = float(qa_ref.abs().max())
    assert max_abs(qa.cpu(), qa_ref) <= 1e-5 * scale
    assert max_abs(qr.cpu(), qr_ref) <= 1e-6 * float(qr_ref.abs().max())


def test_absorb_query_wide_positional_slice_many_rows():
    # d_r = 64 over 40 rows: a 16-row block of the bf16 absorption has 512
    # positional pairs, two per thread (regression: only the first 256 were
    # rotated)
    w = gva_inputs.Workload("absorb", 40, 512, 4, 2, 64, 64, 64, dtype="bf16")
    inp = gva_inputs.make_inputs(w, 31)
    qa_ref, qr_ref = oracle.absorb(inp["q"], inp["m"], inp["lens"], d_r=w.d_r)
    dev = upload(inp)
    qa = torch.empty(40, 4, 64, dtype=torch.float32, device="cuda")
    qr = torch.full((40, 4, 64), float("nan"), dtype=torch.float32, device="cuda")
    note("absorb bf16 d_r=64 B=40")
    gva.gva_absorb_query(dims_of(w), dev["q"], dev["m"], dev["lens"], qa, qr)
    torch.cuda.synchronize()
    assert max_abs(qa.cpu(), qa_ref) <= 1e-5 * float(qa_ref.abs().max())
    assert max_abs(qr.cpu(), qr_ref) <= 1e-6 * float(qr_ref.abs().max())


def test_absorb_query_multi_pass_shapes():
    # d_v = 256 and d_c = 320: M_h goes through LDS in two 128-row passes of
    # three column segments (128, 128, 64), 33 rows in three row blocks
    w = gva_inputs.Workload("absorb", 33, 512, 4, 2, 256, 320, 16, dtype="bf16")
    inp = gva_inputs.make_inputs(w, 37)
    qa_ref, qr_ref = oracle.absorb(inp["q"], inp["m"], inp["lens"], d_r=w.d_r)
    dev = upload(inp)
    qa = torch.full((33, 4, 256), float("nan"), dtype=torch.float32, device="cuda")
    qr = torch.empty(33, 4, 16, dtype=torch.float32, device="cuda")
    note("absorb bf16 d_v=256 d_c=320 B=33")
    gva.gva_absorb_query(dims_of(w), dev["q"], dev["m"], dev["lens"], qa, qr)
    torch.cuda.synchronize()
    assert max_abs(qa.cpu(), qa_ref) <= 1e-5 * float(qa_ref.abs().max())
    assert max_abs(qr.cpu(), qr_ref) <= 1e-6 * float(qr_ref.abs().max())


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_append_matches_oracle_bitwise(dtype):
    B, G, T, dv, dr = 3, 4, 131072, 64, 32
    w = gva_inputs.Workload("append", B, T, 8, G, dv, 64, dr, dtype=dtype)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    g = torch.Generator().manual_seed(31)
    v0 = torch.randn(B, G, T, dv, generator=g).to(tdt)
    k0 = torch.randn(B, T, dr, generator=g).to(tdt)
    n = 64
    v_new = torch.randn(n, G, dv, generator=g).to(tdt)
    k_new = torch.randn(n, dr, generator=g).to(tdt)
    seq = torch.randint(0, B, (n,), generator=g, dtype=torch.int32)
    pos = torch.randint(0, T, (n,), generator=g, dtype=torch.int32)
    pos[:4] = torch.tensor([0, 1, T - 1, 131071 - 3], dtype=torch.int32)
    # unique (seq, pos) so that no two rows race; two rows are out of range
    key = seq.long() * T + pos.long()
    keep = torch.ones(n, dtype=torch.bool)
    seen = set()
    for r in range(n):
        if int(key[r]) in seen:
            keep[r] = False
        seen.add(int(key[r]))
    v_new, k_new, seq, pos = v_new[keep], k_new[keep], seq[keep], pos[keep]
    seq[-1] = B            # skipped
    pos[-2] = -1           # skipped
    v_ref, k_ref = v0.clone(), k0.clone()
    assert oracle.append(v_ref, k_ref, v_new, k_new, seq, pos, w.rope_base) == 2
    vd, kd = gva.tiled(v0).cuda(), gva.tiled(k0).cuda()
    note(f"append {dtype}")
    gva.gva_append_kv(dims_of(w), vd, kd, v_new.cuda(), k_new.cuda(), seq.cuda(), pos.cuda())
    torch.cuda.synchronize()
    itype = torch.int16 if dtype == "bf16" else torch.int32
    assert torch.equal(gva.untiled(vd.cpu()).view(itype), v_ref.view(itype))
    assert torch.equal(gva.untiled(kd.cpu()).view(itype), k_ref.view(itype))


def test_combine_matches_oracle():
    B, H, S, dv = 3, 4, 9, 128
    g = torch.Generator().manual_seed(37)
    o_part = torch.randn(B, H, S, dv, generator=g)
    lse_part = torch.randn(B, H, S, generator=g) * 5
    lse_part[0, 0, :4] = -math.inf
    lse_part[1, 2, :] = -math.inf          # every split empty
    o_ref, lse_ref = oracle.combine(o_part, lse_part)
    w = gva_inputs.Workload("combine", B, 64, H, 1, dv, 64, 0)
    o = torch.empty(B, H, dv, device="cuda")
    lse = torch.empty(B, H, device="cuda")
    note("combine")
    gva.gva_combine(dims_of(w), o_part.cuda(), lse_part.cuda(), S, o, lse)
    torch.cuda.synchronize()
    assert max_abs(o.cpu(), o_ref) <= 1e-5
    assert lse_err(lse.cpu(), lse_ref) <= 1e-5
    assert torch.all(o.cpu()[1, 2] == 0)


def test_full_step_append_then_decode():
    # Algorithm 1 end to end: write the step's new rows at position len-1,
    # then attend over [0, len).
    w = gva_inputs.workload("gva350m_b8_t2k")
    inp = gva_inputs.make_inputs(w, 41, lens=torch.tensor([2048, 1500, 7, 1, 2048, 33, 900, 64]))
    B = w.batch
    seq = torch.arange(B, dtype=torch.int32)
    pos = (inp["lens"] - 1).to(torch.int32)
    v_ref, k_ref = inp["v"].clone(), inp["kr"].clone()
    oracle.append(v_ref, k_ref, inp["v_new"], inp["kr_new"], seq, pos, w.rope_base)
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], v_ref, k_ref, inp["lens"])
    dev = upload(inp)
    d = dims_of(w)
    note("full step")
    gva.gva_append_kv(d, dev["v"], dev["kr"], dev["v_new"], dev["kr_new"], seq.cuda(), pos.cuda())
    o, lse, _, _ = run_decode(w, dev, 4)
    _check(w, o, lse, o_ref, lse_ref, "full_step")


def test_decode_on_a_side_stream():
    # the binding's temporaries (absorbed queries, partials) are allocated on
    # the current stream and read on the caller's: the caching allocator is
    # told so, and the result equals the same step on the current stream
    w = gva_inputs.workload("gva350m_b8_t2k")
    inp = gva_inputs.make_inputs(w, 5)
    dev = upload({k: inp[k] for k in ("q", "m", "v", "kr", "lens")})
    d = dims_of(w)
    note("decode on a side stream")
    o_ref, lse_ref = gva.decode(d, dev["q"], dev["m"], dev["v"], dev["kr"], dev["lens"], 3, fused=False)
    o_ref, lse_ref = o_ref.clone(), lse_ref.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    o, lse = gva.decode(d, dev["q"], dev["m"], dev["v"], dev["kr"], dev["lens"], 3, fused=False, stream=side)
    junk = [torch.full((1 << 20,), float("nan"), device="cuda") for _ in range(8)]   # reuse bait
    torch.cuda.synchronize()
    del junk
    assert torch.equal(o, o_ref) and torch.equal(lse, lse_ref)


STEP_CASES = [
    # (workload, lengths, num_splits, split_rows): one split fused; several
    # splits fused; bounded chunks over a grid past two workgroups per CU, so
    # the absorption runs as its own launch into the workspace; fp32
    (gva_inputs.workload("gva350m_b8_t2k"), None, 1, 0),
    (gva_inputs.workload("gva350m_b8_t2k"), None, 3, 0),
    (gva_inputs.Workload("step_ragged", 40, 2048, 16, 2, 128, 128, 16), "ragged", 8, 256),
    (gva_inputs.workload("tiny_f32"), None, 2, 0),
]


@pytest.mark.parametrize("case", STEP_CASES, ids=lambda c: f"{c[0].name}-S{c[2]}-r{c[3]}")
@pytest.mark.parametrize("append", [False, True])
def test_decode_step_matches_the_separate_calls(case, append):
    w, lens_kind, S, rows = case
    lens = None
    if lens_kind == "ragged":
        g = torch.Generator().manual_seed(17)
        lens = torch.randint(1, w.t_max + 1, (w.batch,), generator=g, dtype=torch.int32)
        lens[:3] = torch.tensor([0, 1, w.t_max], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 13, lens=lens)
    d = dims_of(w)
    dev = upload(inp)
    v2, kr2 = dev["v"].clone(), dev["kr"].clone()
    pend = dict(v_new=dev["v_new"], kr_new=dev["kr_new"]) if append else {}
    fused = gva.gva_prefer_fused(d, S, rows)
    note(f"decode step {w.name} S={S} rows={rows} append={append} fused={fused}")
    ws = gva.workspace_for(d, S, rows)
    assert (ws is None) == (S == 1 and fused)
    o = torch.full((w.batch, w.n_heads, w.d_v), float("nan"), device="cuda")
    lse = torch.full((w.batch, w.n_heads), float("nan"), device="cuda")
    gva.gva_decode_step(d, dev["q"], dev["m"], dev["v"], dev["kr"], dev["lens"], S, o, lse, workspace=ws,
                        split_rows=rows, **pend)
    pend2 = dict(v_new=dev["v_new"], kr_new=dev["kr_new"]) if append else {}
    o2, lse2 = gva.decode(d, dev["q"], dev["m"], v2, kr2, dev["lens"], S, fused=fused, split_rows=rows, **pend2)
    torch.cuda.synchronize()
    assert torch.equal(o, o2) and torch.equal(lse, lse2)
    assert torch.equal(dev["v"], v2) and torch.equal(dev["kr"], kr2)
    v_ref, k_ref = inp["v"], inp["kr"]
    if append:
        v_ref, k_ref = v_ref.clone(), k_ref.clone()
        seq = torch.arange(w.batch, dtype=torch.int32)
        L = inp["lens"].clamp(0, w.t_max)
        live = L > 0
        oracle.append(v_ref, k_ref, inp["v_new"][live], inp["kr_new"][live], seq[live], (L - 1)[live].to(torch.int32),
                      w.rope_base)
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], v_ref, k_ref, inp["lens"], rope_base=w.rope_base)
    _check(w, o.cpu(), lse.cpu(), o_ref, lse_ref, f"step {w.name} S{S}")


# Shapes on both sides of the split planner's thresholds for uniform
# lengths: (B, H, G, d_v = d_c, T) and the plan it must pick there.
PLANNER_CASES = [
    ((8, 16, 4, 64, 1024), 1),       # 128 KiB of value rows per stream: no split
    ((8, 16, 4, 64, 1536), 6),       # 192 KiB: six splits of 32 KiB
    ((1, 32, 8, 128, 8192), 16),     # eight streams: 32 would fill the CUs, capped at 16
    ((16, 32, 8, 128, 4096), 2),     # 128 streams: two splits each
]


@pytest.mark.parametrize("shape,S_expected", PLANNER_CASES)
def test_planner_choice_step_matches_oracle(shape, S_expected):
    # the plan gva_pick_splits makes for the shape, run as one
    # gva_decode_step with the current token's rows, against the oracle's
    # append + decode of every sequence
    B, H, G, D, T = shape
    w = gva_inputs.Workload("planner", B, T, H, G, D, D, 16, dtype="bf16")
    inp = gva_inputs.make_inputs(w, 61)
    d = dims_of(w)
    S, rows = gva.plan_for(d, inp["lens"], n_cu=256)
    assert (S, rows) == (S_expected, 0)
    dev = upload(inp)
    ws = gva.workspace_for(d, S, rows)
    o = torch.full((B, H, D), float("nan"), device="cuda")
    lse = torch.full((B, H), float("nan"), device="cuda")
    note(f"planner {shape}: step S={S}")
    gva.gva_decode_step(d, dev["q"], dev["m"], dev["v"], dev["kr"], dev["lens"], S, o, lse, workspace=ws,
                        split_rows=rows, v_new=dev["v_new"], kr_new=dev["kr_new"])
    torch.cuda.synchronize()
    v_ref, k_ref = inp["v"].clone(), inp["kr"].clone()
    L = inp["lens"].clamp(0, T)
    oracle.append(v_ref, k_ref, inp["v_new"], inp["kr_new"], torch.arange(B, dtype=torch.int32),
                  (L - 1).to(torch.int32), w.rope_base)
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], v_ref, k_ref, inp["lens"], rope_base=w.rope_base)
    _check(w, o.cpu(), lse.cpu(), o_ref, lse_ref, f"planner {shape} S{S}")


# ----------------------------------------------- full-size workloads
def full_size_picks(lens: torch.Tensor, n_spread: int = 12):
    """The sequences a full-size test checks against the oracle: every one of
    a batch of up to 32; otherwise the first, the last and n_spread spread
    evenly over the length ranks (the shortest and the longest included)."""
    B = lens.numel()
    if B <= 32:
        return list(range(B))
    order = torch.argsort(lens, stable=True).tolist()
    ranks = {round(k * (B - 1) / (n_spread - 1)) for k in range(n_spread)}
    return sorted({0, B - 1} | {order[r] for r in ranks})


@pytest.mark.slow
@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("name", ["b32_t8k", "b32_t8k_dr24", "long_b4_t128k", "ragged_b64"])
def test_full_size_sampled(name, seed):
    w = gva_inputs.workload(name)
    note(f"{name} seed {seed}: drawing inputs")
    inp = gva_inputs.make_inputs(w, seed)
    d = dims_of(w)
    S, rows = gva.plan_for(d, inp["lens"])     # the launch configuration bench.py times
    dev = upload({k: inp[k] for k in ("q", "m", "v", "kr", "lens")})
    note(f"{name} seed {seed}: decode S={S} split_rows={rows}")
    o, lse, _, _ = run_decode(w, dev, S, fused=gva.prefer_fused(d, S, split_rows=rows), split_rows=rows)
    del dev
    torch.cuda.empty_cache()
    picks = full_size_picks(inp["lens"])
    assert len(picks) >= min(8, w.batch)
    sub = sub_batch(inp, picks)
    note(f"{name} seed {seed}: oracle on {len(picks)} sequences")
    o_ref, lse_ref = oracle.decode(sub["q"], sub["m"], sub["v"], sub["kr"], sub["lens"])
    idx = torch.tensor(picks)
    _check(w, o[idx], lse[idx], o_ref, lse_ref, f"{name}/seed{seed}/{len(picks)} sequences")
    assert torch.isfinite(o).all()


# ---------------------------------------------- current token from the step
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_current_token_row_matches_append_then_decode(dtype):
    # The attention call appends row len-1 from v_new/kr_new and attends over
    # it without reading it back: the cache's copy of that row is NaN here,
    # so reading it would poison the output.  After the call the caches hold
    # exactly what gva_append_kv stores.
    T = 160
    w = gva_inputs.Workload("pending", 6, T, 16, 4, 64, 64, 16, dtype=dtype)
    lens = torch.tensor([T, 1, 33, 64, 97, 2], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 43, lens=lens)
    B = w.batch
    seq = torch.arange(B, dtype=torch.int32)
    pos = (inp["lens"] - 1).to(torch.int32)
    v_ref, k_ref = inp["v"].clone(), inp["kr"].clone()
    oracle.append(v_ref, k_ref, inp["v_new"], inp["kr_new"], seq, pos, w.rope_base)
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], v_ref, k_ref, inp["lens"])
    itype = torch.int16 if dtype == "bf16" else torch.int32
    d = dims_of(w)
    for b in range(B):
        inp["v"][b, :, int(pos[b])] = float("nan")
        inp["kr"][b, int(pos[b])] = float("nan")
    for S in (1, 3):
        for fused in (True, False):
            note(f"pending row {dtype} S={S} fused={fused}")
            dev = upload(inp)
            o, lse = gva.decode(d, dev["q"], dev["m"], dev["v"], dev["kr"], dev["lens"], S,
                                fused=fused, v_new=dev["v_new"], kr_new=dev["kr_new"])
            torch.cuda.synchronize()
            _check(w, o.cpu(), lse.cpu(), o_ref, lse_ref, f"pending/{dtype}/S{S}/fused={fused}")
            assert torch.equal(gva.untiled(dev["v"].cpu()).view(itype), v_ref.view(itype))
            assert torch.equal(gva.untiled(dev["kr"].cpu()).view(itype), k_ref.view(itype))


def test_append_and_attend_in_one_launch_full_step():
    # Algorithm 1 as the bench runs it on the 350M-model shape: the attention
    # call appends the step's rows and attends over them; a repeated step at
    # the same position leaves the caches unchanged (the append is idempotent).
    w = gva_inputs.workload("gva350m_b8_t2k")
    inp = gva_inputs.make_inputs(w, 47, lens=torch.tensor([2048, 1500, 7, 1, 2048, 33, 900, 64]))
    B = w.batch
    seq = torch.arange(B, dtype=torch.int32)
    pos = (inp["lens"] - 1).to(torch.int32)
    v_ref, k_ref = inp["v"].clone(), inp["kr"].clone()
    oracle.append(v_ref, k_ref, inp["v_new"], inp["kr_new"], seq, pos, w.rope_base)
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], v_ref, k_ref, inp["lens"])
    dev = upload(inp)
    d = dims_of(w)
    S = gva.splits_for(d, inp["lens"])
    itype = torch.int16
    for rep in range(2):
        note(f"append+attend in one launch, S={S}, rep {rep}")
        o, lse = gva.decode(d, dev["q"], dev["m"], dev["v"], dev["kr"], dev["lens"], S,
                            v_new=dev["v_new"], kr_new=dev["kr_new"])
        torch.cuda.synchronize()
        _check(w, o.cpu(), lse.cpu(), o_ref, lse_ref, f"append+attend/rep{rep}")
        assert torch.equal(gva.untiled(dev["v"].cpu()).view(itype), v_ref.view(itype))
        assert torch.equal(gva.untiled(dev["kr"].cpu()).view(itype), k_ref.view(itype))


# ------------------------------------------------ matched-GQA baseline kernel
@pytest.mark.parametrize("hpg,dv", [(1, 64), (2, 128), (4, 64), (4, 128), (8, 128)])
def test_gqa_baseline_matches_oracle(hpg, dv):
    G = 2
    w = gva_inputs.Workload("gqa", 5, 304, G * hpg, G, dv, dv, 16, dtype="bf16", gqa=True)
    lens = torch.tensor([304, 0, 1, 33, 207], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 11, lens=lens)
    o_ref, lse_ref = oracle.gqa_decode(inp["q"], inp["k_gqa"], inp["v"], inp["lens"], d_k=dv)
    dev = upload(inp)
    d = dims_of(w)
    for S, rows in ((1, 0), (3, 0), (8, 0), (10, 32), (3, 64)):
        note(f"gqa hpg={hpg} dv={dv} S={S} split_rows={rows}")
        o, lse = gva.gqa_decode(d, dev["q"], dev["k_gqa"], dev["v"], dev["lens"], S, split_rows=rows)
        torch.cuda.synchronize()
        _check(w, o.cpu(), lse.cpu(), o_ref, lse_ref, f"gqa/hpg{hpg}/dv{dv}/S{S}/rows{rows}")


def test_gqa_baseline_partials_and_untouched_caches():
    # every split partial against the oracle on that split's rows; the
    # caches are read only
    w = gva_inputs.Workload("gqa", 3, 208, 16, 2, 128, 128, 16, dtype="bf16", gqa=True)
    lens = torch.tensor([208, 95, 17], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 5, lens=lens)
    dev = upload(inp)
    k0, v0 = dev["k_gqa"].clone(), dev["v"].clone()
    d = dims_of(w)
    S = 4
    bufs = gva.DecodeBuffers(d, S)
    gva.gva_gqa_decode_attention(d, dev["q"], dev["k_gqa"], dev["v"], dev["lens"], S,
                                 bufs.o_part, bufs.lse_part)
    torch.cuda.synchronize()
    op, lp = bufs.o_part.cpu(), bufs.lse_part.cpu()
    for s, (lo, hi) in enumerate(zip(*split_bounds(inp["lens"], S))):
        for b in range(w.batch):
            a, e = int(lo[b]), int(hi[b])
            if a >= e:
                assert torch.all(lp[b, :, s] == float("-inf"))
                if s == 0:
                    assert torch.all(op[b, :, s] == 0)
                continue
            sl = slice(b, b + 1)
            o_ref, lse_ref = oracle.gqa_decode(inp["q"][sl], inp["k_gqa"][sl, :, a:e].contiguous(),
                                               inp["v"][sl, :, a:e].contiguous(),
                                               torch.tensor([e - a], dtype=torch.int32), d_k=w.d_v)
            _check(w, op[sl, :, s], lp[sl, :, s], o_ref, lse_ref, f"gqa partial b{b} s{s}")
    assert torch.equal(dev["k_gqa"], k0) and torch.equal(dev["v"], v0)


@pytest.mark.slow
@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("name", ["ragged_b64", "b32_t8k"])
def test_gqa_baseline_full_size_sampled(name, seed):
    # the matched-GQA kernel at the sizes bench.py compares it at (b32_t8k
    # carries no GQA key cache in its recipe: the comparison draws one)
    w = gva_inputs.workload(name)
    note(f"{name} gqa seed {seed}: drawing inputs")
    inp = gva_inputs.make_inputs(w, seed)
    if "k_gqa" not in inp:
        inp["k_gqa"] = gva_inputs.gqa_keys(w, seed)
    d = dims_of(w)
    S, rows = gva.plan_for(d, inp["lens"])
    dev = upload({k: inp[k] for k in ("q", "v", "k_gqa", "lens")})
    note(f"{name} gqa seed {seed}: decode S={S} split_rows={rows}")
    o, lse = gva.gqa_decode(d, dev["q"], dev["k_gqa"], dev["v"], dev["lens"], S, split_rows=rows)
    o, lse = o.cpu(), lse.cpu()
    del dev
    torch.cuda.empty_cache()
    picks = full_size_picks(inp["lens"])
    sub = sub_batch(inp, picks)
    note(f"{name} gqa seed {seed}: oracle on {len(picks)} sequences")
    o_ref, lse_ref = oracle.gqa_decode(sub["q"], sub["k_gqa"], sub["v"], sub["lens"], d_k=w.d_v)
    idx = torch.tensor(picks)
    _check(w, o[idx], lse[idx], o_ref, lse_ref, f"{name} gqa/seed{seed}/{len(picks)} sequences")
    assert torch.isfinite(o).all()


@pytest.mark.slow
def test_one_gib_value_stream():
    # a single value stream of 2^22 rows x 128 bf16 = 1 GiB (the layout
    # allows up to 2 GiB - 16 MiB per stream): the 32-bit buffer offsets
    # near the top of the stream, one workgroup streaming all of it, even
    # splits and bounded chunks, a length just short of capacity, and the
    # current row appended at row 2^22 - 6
    T = 1 << 22
    w = gva_inputs.Workload("one_gib", 1, T, 2, 1, 128, 64, 16)
    lens = torch.tensor([T - 5], dtype=torch.int32)
    note("one GiB stream: drawing inputs")
    inp = gva_inputs.make_inputs(w, 81, lens=lens)
    seq = torch.zeros(1, dtype=torch.int32)
    pos = (lens - 1).to(torch.int32)
    v_ref, k_ref = inp["v"].clone(), inp["kr"].clone()
    oracle.append(v_ref, k_ref, inp["v_new"], inp["kr_new"], seq, pos, w.rope_base)
    note("one GiB stream: oracle")
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], v_ref, k_ref, lens)
    del v_ref, k_ref
    d = dims_of(w)
    for S, rows in ((1, 0), (64, 0), (64, 65536)):
        note(f"one GiB stream: S={S} split_rows={rows}")
        dev = upload(inp)
        o, lse = gva.decode(d, dev["q"], dev["m"], dev["v"], dev["kr"], dev["lens"], S,
                            v_new=dev["v_new"], kr_new=dev["kr_new"], split_rows=rows)
        torch.cuda.synchronize()
        _check(w, o.cpu(), lse.cpu(), o_ref, lse_ref, f"one GiB/S{S}/rows{rows}")
        del dev
        torch.cuda.empty_cache()


# ------------------------------------------- bounded-chunk splits (ragged batches)
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("fused", [True, False])
def test_bounded_chunk_splits_match_oracle(dtype, fused):
    # no split of more than split_rows rows, a sequence's splits even; too
    # few splits share the rows evenly; empty splits write only their lse
    w = gva_inputs.Workload("chunks", 6, 1024, 16, 2, 128 if dtype == "bf16" else 64, 64, 16,
                            dtype=dtype)
    lens = torch.tensor([1024, 1, 0, 333, 64, 700], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 21, lens=lens)
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], inp["v"], inp["kr"], inp["lens"])
    dev = upload(inp)
    plan = gva.plan_for(dims_of(w), inp["lens"])
    for S, rows in sorted({(32, 32), (8, 128), (2, 128), (1, 64), plan}):
        note(f"chunks {dtype} fused={fused} S={S} split_rows={rows}")
        o, lse, _, _ = run_decode(w, dev, S, fused=fused, split_rows=rows)
        _check(w, o, lse, o_ref, lse_ref, f"chunks/{dtype}/fused={fused}/S{S}/rows{rows}")


def test_bounded_chunks_with_current_row():
    # the append folded into the attention launch, with bounded chunks: the
    # chunk holding row len-1 appends it
    w = gva_inputs.Workload("chunks_pending", 4, 512, 8, 2, 128, 128, 16)
    lens = torch.tensor([512, 97, 1, 256], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 23, lens=lens)
    seq = torch.arange(w.batch, dtype=torch.int32)
    pos = (lens - 1).to(torch.int32)
    v_ref, k_ref = inp["v"].clone(), inp["kr"].clone()
    oracle.append(v_ref, k_ref, inp["v_new"], inp["kr_new"], seq, pos, w.rope_base)
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], v_ref, k_ref, inp["lens"])
    d = dims_of(w)
    for S, rows in ((16, 32), (3, 96)):
        note(f"chunks + current row S={S} split_rows={rows}")
        dev = upload(inp)
        o, lse = gva.decode(d, dev["q"], dev["m"], dev["v"], dev["kr"], dev["lens"], S,
                            v_new=dev["v_new"], kr_new=dev["kr_new"], split_rows=rows)
        torch.cuda.synchronize()
        _check(w, o.cpu(), lse.cpu(), o_ref, lse_ref, f"chunks+current/S{S}/rows{rows}")
        assert torch.equal(gva.untiled(dev["v"].cpu()).view(torch.int16), v_ref.view(torch.int16))
        assert torch.equal(gva.untiled(dev["kr"].cpu()).view(torch.int16), k_ref.view(torch.int16))


# (batch, capacity, heads, groups, d_v, d_c, d_r, [(splits, split_rows)]): the
# slot map reads the lengths in blocks of ceil(B / 64) per lane, then (B > 64)
# scans the block holding the slot 64 sequences at a time; B = 4100 needs two
# such passes
LARGE_BATCH_CHUNKS = [
    (150, 512, 8, 2, 128, 64, 16, [(9, 64), (3, 128), (5, 32)]),
    (4100, 64, 2, 1, 64, 32, 8, [(3, 32), (1, 32)]),
]


@pytest.mark.parametrize("fused", [True, False])
@pytest.mark.parametrize("cfg", LARGE_BATCH_CHUNKS, ids=lambda c: f"B{c[0]}")
def test_bounded_chunk_slots_large_batch(cfg, fused):
    # bounded chunks over more than 64 sequences and B * S not a multiple of 8
    # (padding workgroups): every (b, h, s) partial is written exactly as the
    # oracle's split says, the buffers having been filled with NaN first
    B, T, H, G, dv, dc, dr, plans = cfg
    w = gva_inputs.Workload(f"chunks_b{B}", B, T, H, G, dv, dc, dr)
    g = torch.Generator().manual_seed(31)
    lens = torch.randint(0, w.t_max + 1, (w.batch,), generator=g, dtype=torch.int32)
    lens[::7] = 0
    lens[1::11] = w.t_max
    lens[2::13] = 1
    lens[3::17] = 64
    inp = gva_inputs.make_inputs(w, 33, lens=lens)
    d = dims_of(w)
    dev = upload(inp)
    q_abs = q_rot = None
    if not fused:
        q_abs = torch.empty(w.batch, w.n_heads, w.d_v, dtype=torch.float32, device="cuda")
        q_rot = torch.empty(w.batch, w.n_heads, w.d_r, dtype=torch.float32, device="cuda")
        gva.gva_absorb_query(d, dev["q"], dev["m"], dev["lens"], q_abs, q_rot)
    for S, rows in plans:
        assert (w.batch * S) % 8 != 0
        note(f"chunks B{B} fused={fused} S={S} split_rows={rows}")
        o_part = torch.full((w.batch, w.n_heads, S, w.d_v), math.nan, device="cuda")
        lse_part = torch.full((w.batch, w.n_heads, S), math.nan, device="cuda")
        gva.gva_decode_attention(d, dev["v"], dev["kr"], dev["lens"], S, o_part, lse_part,
                                 q=dev["q"] if fused else None, m=dev["m"] if fused else None,
                                 q_abs=q_abs, q_rot=q_rot, split_rows=rows)
        torch.cuda.synchronize()
        o_part, lse_part = o_part.cpu(), lse_part.cpu()
        begins, ends = split_bounds(inp["lens"], S, split_rows=rows)
        for s in range(S):
            o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], inp["v"], inp["kr"], inp["lens"],
                                           t_begin=begins[s], t_end=ends[s])
            assert not torch.isnan(lse_part[:, :, s]).any(), (S, rows, s, "lse not written")
            assert lse_err(lse_part[:, :, s], lse_ref) <= 1e-3, (S, rows, s)
            live = (ends[s] > begins[s]) | (s == 0)
            err = max_abs(o_part[live][:, :, s], o_ref[live])
            assert err <= QUALITY["bf16"], (S, rows, s, err)


# Even splits with B * S not a multiple of 8: the split-major slots in
# contiguous XCD ranges, some slot's groups on two XCDs.  (B, H, G, S):
# 21 x 8 streams (>= half the CUs: four waves per workgroup), and 5 x 8 x 3
# (few workgroups: eight waves each).
EVEN_PADDED = [(21, 32, 8, 1), (21, 32, 8, 3), (5, 32, 8, 3), (7, 16, 4, 2)]


@pytest.mark.parametrize("fused", [True, False])
@pytest.mark.parametrize("cfg", EVEN_PADDED, ids=lambda c: f"B{c[0]}H{c[1]}G{c[2]}S{c[3]}")
def test_even_split_slots_padded_grid(cfg, fused):
    # every (b, h, s) partial written exactly as the oracle's split says, the
    # buffers filled with NaN first
    B, H, G, S = cfg
    w = gva_inputs.Workload(f"even_b{B}", B, 640, H, G, 128, 128, 16)
    g = torch.Generator().manual_seed(41)
    lens = torch.randint(0, w.t_max + 1, (w.batch,), generator=g, dtype=torch.int32)
    lens[0], lens[-1] = w.t_max, 0
    inp = gva_inputs.make_inputs(w, 43, lens=lens)
    d = dims_of(w)
    dev = upload(inp)
    assert (w.batch * S) % 8 != 0
    note(f"even slots B{B} H{H} G{G} S={S} fused={fused}")
    q_abs = q_rot = None
    if not fused:
        q_abs = torch.empty(w.batch, w.n_heads, w.d_v, dtype=torch.float32, device="cuda")
        q_rot = torch.empty(w.batch, w.n_heads, w.d_r, dtype=torch.float32, device="cuda")
        gva.gva_absorb_query(d, dev["q"], dev["m"], dev["lens"], q_abs, q_rot)
    o_part = torch.full((w.batch, w.n_heads, S, w.d_v), math.nan, device="cuda")
    lse_part = torch.full((w.batch, w.n_heads, S), math.nan, device="cuda")
    gva.gva_decode_attention(d, dev["v"], dev["kr"], dev["lens"], S, o_part, lse_part,
                             q=dev["q"] if fused else None, m=dev["m"] if fused else None,
                             q_abs=q_abs, q_rot=q_rot)
    torch.cuda.synchronize()
    o_part, lse_part = o_part.cpu(), lse_part.cpu()
    begins, ends = split_bounds(inp["lens"], S)
    for s in range(S):
        o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], inp["v"], inp["kr"], inp["lens"],
                                       t_begin=begins[s], t_end=ends[s])
        assert not torch.isnan(lse_part[:, :, s]).any(), (cfg, s, "lse not written")
        assert lse_err(lse_part[:, :, s], lse_ref) <= 1e-3, (cfg, s)
        live = (ends[s] > begins[s]) | (s == 0)
        err = max_abs(o_part[live][:, :, s], o_ref[live])
        assert err <= QUALITY["bf16"], (cfg, s, err)


# ------------------------------------------------- writes stay in bounds
_GUARD = 4096          # sentinel elements on each side of an output (16 KB of fp32)
_SENTINEL = 0x7FC0DEAD  # a NaN bit pattern no kernel writes


def _guarded(shape):
    """A contiguous fp32 output with sentinel words before and after it."""
    n = math.prod(shape)
    big = torch.empty(n + 2 * _GUARD, dtype=torch.int32, device="cuda").fill_(_SENTINEL)
    return big, big[_GUARD:_GUARD + n].view(torch.float32).view(shape)


def _guards_intact(big):
    head, tail = big[:_GUARD], big[-_GUARD:]
    return bool((head == _SENTINEL).all()) and bool((tail == _SENTINEL).all())


def test_outputs_written_only_in_bounds():
    # every output buffer sits between two 16 KB runs of a sentinel; after
    # absorption, attention (fused and separate, even and bounded-chunk
    # splits, bf16 and fp32), combine, the GQA baseline, the ordinary-RoPE
    # contrast and the prefill, the sentinels must be untouched
    for dtype in ("bf16", "f32"):
        w = gva_inputs.Workload("guards", 3, 304, 8, 2, 128 if dtype == "bf16" else 64, 64, 16,
                                dtype=dtype)
        lens = torch.tensor([300, 1, 97], dtype=torch.int32)
        inp = gva_inputs.make_inputs(w, 71, lens=lens)
        d = dims_of(w)
        dev = upload(inp)
        B, H, dv, dr = w.batch, w.n_heads, w.d_v, w.d_r
        bigs = []
        qa_big, q_abs = _guarded((B, H, dv))
        qr_big, q_rot = _guarded((B, H, dr))
        bigs += [qa_big, qr_big]
        note(f"guards {dtype}: absorb")
        gva.gva_absorb_query(d, dev["q"], dev["m"], dev["lens"], q_abs, q_rot)
        for S, rows, fused in ((1, 0, True), (3, 0, False), (10, 32, True), (10, 32, False)):
            note(f"guards {dtype}: attention S={S} rows={rows} fused={fused}")
            op_big, o_part = _guarded((B, H, S, dv))
            lp_big, lse_part = _guarded((B, H, S))
            kw = dict(q=dev["q"], m=dev["m"]) if fused else dict(q_abs=q_abs, q_rot=q_rot)
            gva.gva_decode_attention(d, dev["v"], dev["kr"], dev["lens"], S, o_part, lse_part,
                                     split_rows=rows, **kw)
            o_big, o = _guarded((B, H, dv))
            l_big, lse = _guarded((B, H))
            gva.gva_combine(d, o_part, lse_part, S, o, lse)
            bigs += [op_big, lp_big, o_big, l_big]
        torch.cuda.synchronize()
        if dtype == "bf16":
            note("guards: GQA baseline and ordinary-RoPE contrast")
            k_gqa = gva.tiled(gva_inputs.gqa_keys(w, 71)).cuda()
            q_gqa = torch.randn(B, H, dv, generator=torch.Generator().manual_seed(72)).to(torch.bfloat16).cuda()
            for S, rows in ((2, 0), (10, 32)):
                op_big, o_part = _guarded((B, H, S, dv))
                lp_big, lse_part = _guarded((B, H, S))
                gva.gva_gqa_decode_attention(d, q_gqa, k_gqa, dev["v"], dev["lens"], S, o_part,
                                             lse_part, split_rows=rows)
                bigs += [op_big, lp_big]
            d0 = gva.make_dims(B, H, w.n_groups, dv, w.d_c, 0, w.t_max, w.dtype, w.rope_base)
            q0 = dev["q"][..., : w.d_c].contiguous()
            op_big, o_part = _guarded((B, H, 2, dv))
            lp_big, lse_part = _guarded((B, H, 2))
            gva.gva_rope_decode_attention(d0, q0, dev["m"], dev["v"], dev["lens"], 2, o_part, lse_part)
            bigs += [op_big, lp_big]
            note("guards: prefill")
            N = 90
            qp = gva_inputs.prefill_queries(w, 71, N).cuda()
            pa_big, pq_abs = _guarded((B, N, H, dv))
            pr_big, pq_rot = _guarded((B, N, H, dr))
            gva.gva_prefill_absorb(d, N, qp, dev["m"], dev["lens"], pq_abs, pq_rot)
            po_big, po = _guarded((B, N, H, dv))
            pl_big, plse = _guarded((B, N, H))
            gva.gva_prefill_attention(d, N, pq_abs, pq_rot, dev["v"], dev["kr"], dev["lens"], po, plse)
            bigs += [pa_big, pr_big, po_big, pl_big]
        torch.cuda.synchronize()
        bad = [i for i, big in enumerate(bigs) if not _guards_intact(big)]
        assert not bad, (dtype, bad)


def test_combine_never_reads_empty_partials():
    # partials of empty splits hold NaN: a combine that read them would
    # return NaN
    g = torch.Generator().manual_seed(9)
    B, H, S, dv = 3, 4, 70, 128
    o_part = torch.randn(B, H, S, dv, generator=g)
    lse_part = torch.randn(B, H, S, generator=g) * 3
    lse_part[0, :, 5:] = -math.inf
    lse_part[1, :, ::3] = -math.inf
    lse_part[2, 1, :] = -math.inf
    o_ref, lse_ref = oracle.combine(o_part, lse_part)
    o_part[torch.isneginf(lse_part)] = float("nan")
    w = gva_inputs.Workload("combine", B, 64, H, 1, dv, 64, 0)
    o = torch.empty(B, H, dv, device="cuda")
    lse = torch.empty(B, H, device="cuda")
    note("combine, NaN in empty partials")
    gva.gva_combine(dims_of(w), o_part.cuda(), lse_part.cuda(), S, o, lse)
    torch.cuda.synchronize()
    assert torch.isfinite(o.cpu()).all()
    assert max_abs(o.cpu(), o_ref) <= 1e-5
    assert lse_err(lse.cpu(), lse_ref) <= 1e-5


# ------------------------------------------------- HIP graph capture of steps
@pytest.mark.parametrize("S,fused", [(1, True), (3, False)])
def test_graph_capture_of_layer_steps(S, fused):
    # Several layers' decode steps (absorb, attention with the current row
    # appended in the same launch, combine) captured in one HIP graph.  The
    # library allocates, synchronises and clears nothing, so its launches
    # are capturable as they are.  Each replay, with eager work and
    # synchronisation between replays, must equal the eager result bit for
    # bit and match the oracle.
    w = gva_inputs.workload("gva350m_b8_t2k")
    d = dims_of(w)
    n_layers = 3
    layers = []
    for layer in range(n_layers):
        inp = gva_inputs.make_inputs(w, 100 + layer)
        seq = torch.arange(w.batch, dtype=torch.int32)
        pos = (inp["lens"] - 1).to(torch.int32)
        v_ref, k_ref = inp["v"].clone(), inp["kr"].clone()
        oracle.append(v_ref, k_ref, inp["v_new"], inp["kr_new"], seq, pos, w.rope_base)
        o_ref, _ = oracle.decode(inp["q"], inp["m"], v_ref, k_ref, inp["lens"])
        layers.append((upload(inp), gva.DecodeBuffers(d, S), o_ref))

    def run_layers():
        outs = []
        for dev, bufs, _ in layers:
            o, _ = gva.decode(d, dev["q"], dev["m"], dev["v"], dev["kr"], dev["lens"], S, bufs=bufs,
                              fused=fused, v_new=dev["v_new"], kr_new=dev["kr_new"])
            outs.append(o)
        return outs

    note(f"graph capture S={S} fused={fused}: eager")
    eager = [o.clone() for o in run_layers()]
    torch.cuda.synchronize()
    for o, (_, _, o_ref) in zip(eager, layers):
        assert max_abs(o.cpu(), o_ref) <= 1e-4
    run_layers()                                  # warm the capture stream's allocator state
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        graphed = run_layers()
    for rep in range(3):
        for o in graphed:
            o.zero_()
        scratch = torch.randn(1 << 16, device="cuda").sum()     # eager work between replays
        torch.cuda.synchronize()
        note(f"graph replay {rep}")
        g.replay()
        torch.cuda.synchronize()
        assert float(scratch) == float(scratch)
        for o, e in zip(graphed, eager):
            assert torch.equal(o, e), f"replay {rep} differs from eager"



# ------------------------------------------------------------ paged caches
def _paged_setup(w, seed, lens, page_rows, extra_pages=5):
    inp = gva_inputs.make_inputs(w, seed, lens=lens)
    d = dims_of(w)
    max_pages = w.t_max // page_rows
    n_pages = w.batch * max_pages + extra_pages
    g = torch.Generator().manual_seed(seed + 1)
    bt = torch.randperm(n_pages, generator=g)[: w.batch * max_pages].reshape(w.batch, max_pages).to(torch.int32)
    pg = gva.make_paging(d, page_rows, n_pages)
    return inp, d, pg, bt


@pytest.mark.parametrize("page_rows", [32, 64, 256])
def test_paged_decode_matches_oracle(page_rows):
    # the caches scattered over a pool in random page order; unused pages
    # hold NaN, so reading a wrong page poisons the output
    w = gva_inputs.Workload("paged", 6, 512, 16, 4, 128, 128, 16)
    lens = torch.tensor([512, 0, 1, page_rows - 1, page_rows + 1, 300], dtype=torch.int32)
    inp, d, pg, bt = _paged_setup(w, 31, lens, page_rows)
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], inp["v"], inp["kr"], inp["lens"])
    vp, kp = gva.to_pages(gva.tiled(inp["v"]), gva.tiled(inp["kr"]), bt, pg, fill=float("nan"))
    dev = upload({k: inp[k] for k in ("q", "m", "lens")})
    vp, kp, btd = vp.cuda(), kp.cuda(), bt.cuda()
    for S, rows, fused in ((1, 0, True), (3, 0, False), (12, 64, False), (2, 0, True)):
        note(f"paged page_rows={page_rows} S={S} split_rows={rows} fused={fused}")
        o, lse = gva.paged_decode(d, pg, dev["q"], dev["m"], vp, kp, btd, dev["lens"], S, fused=fused,
                                  split_rows=rows)
        torch.cuda.synchronize()
        _check(w, o.cpu(), lse.cpu(), o_ref, lse_ref, f"paged/{page_rows}/S{S}/rows{rows}/fused={fused}")


def test_paged_at_max_pages():
    # a sequence of GVA_MAX_PAGES = 4096 pages of 32 rows (131,072 rows), in
    # random pool order with NaN in the unused pages: one split holds all
    # 4096 page ids in LDS; also 7 even splits and bounded chunks of 4096 rows
    page_rows = 32
    w = gva_inputs.Workload("paged_max", 2, gva.GVA_MAX_PAGES * page_rows, 4, 1, 128, 64, 16)
    lens = torch.tensor([w.t_max - 3, 40000], dtype=torch.int32)
    inp, d, pg, bt = _paged_setup(w, 43, lens, page_rows)
    assert pg.max_pages == gva.GVA_MAX_PAGES
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], inp["v"], inp["kr"], inp["lens"])
    vp, kp = gva.to_pages(gva.tiled(inp["v"]), gva.tiled(inp["kr"]), bt, pg, fill=float("nan"))
    dev = upload({k: inp[k] for k in ("q", "m", "lens")})
    vp, kp, btd = vp.cuda(), kp.cuda(), bt.cuda()
    for S, rows, fused in ((1, 0, True), (7, 0, False), (32, 4096, True)):
        note(f"paged max pages S={S} split_rows={rows} fused={fused}")
        o, lse = gva.paged_decode(d, pg, dev["q"], dev["m"], vp, kp, btd, dev["lens"], S, fused=fused,
                                  split_rows=rows)
        torch.cuda.synchronize()
        _check(w, o.cpu(), lse.cpu(), o_ref, lse_ref, f"paged max/S{S}/rows{rows}/fused={fused}")


def test_paged_append_and_current_row():
    # the paged append and the current row appended in the attention launch
    # write exactly what the contiguous append writes, at the right pages
    page_rows = 64
    w = gva_inputs.Workload("paged", 4, 256, 8, 2, 128, 128, 16)
    lens = torch.tensor([256, 65, 1, 128], dtype=torch.int32)
    inp, d, pg, bt = _paged_setup(w, 37, lens, page_rows)
    seq = torch.arange(w.batch, dtype=torch.int32)
    pos = (lens - 1).to(torch.int32)
    v_ref, k_ref = inp["v"].clone(), inp["kr"].clone()
    oracle.append(v_ref, k_ref, inp["v_new"], inp["kr_new"], seq, pos, w.rope_base)
    o_ref, lse_ref = oracle.decode(inp["q"], inp["m"], v_ref, k_ref, inp["lens"])
    vp0, kp0 = gva.to_pages(gva.tiled(inp["v"]), gva.tiled(inp["kr"]), bt, pg)
    dev = upload({k: inp[k] for k in ("q", "m", "lens", "v_new", "kr_new")})
    btd = bt.cuda()
    itype = torch.int16
    # 1) the paged append call
    vp, kp = vp0.clone().cuda(), kp0.clone().cuda()
    note("paged append")
    gva.gva_paged_append_kv(d, pg, vp, kp, btd, dev["v_new"], dev["kr_new"], seq.cuda(), pos.cuda())
    torch.cuda.synchronize()
    v2, k2 = gva.from_pages(vp.cpu(), kp.cpu(), bt, pg)
    assert torch.equal(gva.untiled(v2).view(itype), v_ref.view(itype))
    assert torch.equal(gva.untiled(k2).view(itype), k_ref.view(itype))
    # 2) appended and attended in one launch
    for S, fused in ((1, True), (3, False)):
        vp, kp = vp0.clone().cuda(), kp0.clone().cuda()
        note(f"paged current row S={S} fused={fused}")
        o, lse = gva.paged_decode(d, pg, dev["q"], dev["m"], vp, kp, btd, dev["lens"], S, fused=fused,
                                  v_new=dev["v_new"], kr_new=dev["kr_new"])
        torch.cuda.synchronize()
        _check(w, o.cpu(), lse.cpu(), o_ref, lse_ref, f"paged current row S{S}")
        v2, k2 = gva.from_pages(vp.cpu(), kp.cpu(), bt, pg)
        assert torch.equal(gva.untiled(v2).view(itype), v_ref.view(itype))
        assert torch.equal(gva.untiled(k2).view(itype), k_ref.view(itype))


# ------------------------------------- GVA with ordinary RoPE (contrast path)
# W_h = rotation-paired q M_h is rounded to bf16 and the cos/sin weights are
# fp32, so this path is less exact than the absorbed one (which keeps the
# query as a bf16 high+low pair); its expected accuracy is pinned separately.
# A relative rounding of up to 2^-9 on each W entry moves a base-2 logit of
# rms ~1.4 by ~1.6e-3 rms; with one row dominating a short sequence and
# |v| up to ~4 that is a few 1e-3 on o (observed: <= 1.9e-3).
ROPE_QUALITY = 5e-3


def _rope_check(o, lse, o_ref, lse_ref, label):
    err = max_abs(o, o_ref)
    lerr = lse_err(lse, lse_ref)
    note(f"{label}: max|o-o_ref| = {err:.3e}  max|lse-lse_ref| = {lerr:.3e}")
    assert err <= TOL["bf16"], (label, err)
    assert err <= ROPE_QUALITY, (label, err)
    assert lerr <= 1e-2, (label, lerr)


def _rope_workload(hpg, dv, dc, T, B, G=2):
    return gva_inputs.Workload("rope", B, T, G * hpg, G, dv, dc, 0, dtype="bf16")


@pytest.mark.parametrize("hpg,dv,dc", [(1, 64, 64), (1, 128, 128), (2, 128, 64), (4, 64, 128),
                                       (4, 128, 128), (8, 64, 64), (8, 64, 128), (8, 128, 64)])
def test_rope_decode_matches_oracle(hpg, dv, dc):
    w = _rope_workload(hpg, dv, dc, 304, 5)
    lens = torch.tensor([304, 0, 1, 45, 263], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 13, lens=lens)
    for b, L in enumerate(lens.tolist()):       # rows past a length are never read
        inp["v"][b, :, L:] = float("nan")
    o_ref, lse_ref = oracle.rope_decode(inp["q"], inp["m"], inp["v"], inp["lens"], rope_base=w.rope_base)
    dev = upload({k: inp[k] for k in ("q", "m", "v", "lens")})
    d = dims_of(w)
    for S, rows in ((1, 0), (3, 0), (8, 0), (10, 32), (3, 64)):
        note(f"rope hpg={hpg} dv={dv} dc={dc} S={S} split_rows={rows}")
        o, lse = gva.rope_decode(d, dev["q"], dev["m"], dev["v"], dev["lens"], S, split_rows=rows)
        torch.cuda.synchronize()
        _rope_check(o.cpu(), lse.cpu(), o_ref, lse_ref, f"rope/hpg{hpg}/dv{dv}/dc{dc}/S{S}/rows{rows}")


def test_rope_decode_long_positions_and_read_only_cache():
    # positions up to 16K: the angle reduction has to hold far from zero
    w = _rope_workload(4, 128, 128, 16384, 2, G=1)
    lens = torch.tensor([16384, 9001], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 17, lens=lens)
    note("rope long positions: oracle")
    o_ref, lse_ref = oracle.rope_decode(inp["q"], inp["m"], inp["v"], inp["lens"], rope_base=w.rope_base)
    dev = upload({k: inp[k] for k in ("q", "m", "v", "lens")})
    v0 = dev["v"].clone()
    d = dims_of(w)
    for S in (1, 16):
        note(f"rope long positions S={S}")
        o, lse = gva.rope_decode(d, dev["q"], dev["m"], dev["v"], dev["lens"], S)
        torch.cuda.synchronize()
        _rope_check(o.cpu(), lse.cpu(), o_ref, lse_ref, f"rope long/S{S}")
    assert torch.equal(dev["v"], v0)


def test_rope_decode_differs_from_absorbed_gva():
    # the same q, M and values through the absorbed (no rotation, d_r = 0)
    # kernel give a different result: the contrast path is not the GVA path
    w = _rope_workload(4, 64, 64, 128, 2)
    inp = gva_inputs.make_inputs(w, 19, lens=torch.tensor([128, 77], dtype=torch.int32))
    dev = upload({k: inp[k] for k in ("q", "m", "v", "kr", "lens")})
    d = dims_of(w)
    note("rope vs absorbed")
    o_r, _ = gva.rope_decode(d, dev["q"], dev["m"], dev["v"], dev["lens"], 1)
    o_a, _, _, _ = run_decode(w, dev, 1)
    torch.cuda.synchronize()
    assert max_abs(o_r.cpu(), o_a) > 1e-2


@pytest.mark.slow
def test_rope_decode_full_size_sampled():
    # the bandwidth-headline shape (B32, T8192, H32, G8, d 128/128) with
    # ordinary RoPE: every output checked for finiteness, two sequences
    # against the oracle
    w = gva_inputs.workload("b32_t8k").replace(name="rope_b32_t8k", d_r=0)
    note("rope b32_t8k: drawing inputs")
    inp = gva_inputs.make_inputs(w, 0)
    d = dims_of(w)
    dev = upload({k: inp[k] for k in ("q", "m", "v", "lens")})
    note("rope b32_t8k: decode S=1")
    o, lse = gva.rope_decode(d, dev["q"], dev["m"], dev["v"], dev["lens"], 1)
    o, lse = o.cpu(), lse.cpu()
    del dev
    torch.cuda.empty_cache()
    picks = [0, w.batch - 1]
    sub = sub_batch(inp, picks)
    note(f"rope b32_t8k: oracle on sequences {picks}")
    o_ref, lse_ref = oracle.rope_decode(sub["q"], sub["m"], sub["v"], sub["lens"], rope_base=w.rope_base)
    idx = torch.tensor(picks)
    _rope_check(o[idx], lse[idx], o_ref, lse_ref, "rope b32_t8k/sampled")
    assert torch.isfinite(o).all()


# ------------------------------------------------------- prefill (causal)
# The prefill kernel feeds the matrix cores the absorbed and rotated queries
# as bf16 high + low pairs (~2^-17 relative, as the decode kernel does) and
# the softmax weights in fp16: a weight's relative rounding of 2^-12 moves o
# by about that much times the spread of the values (N(0, 1), maximum ~4
# over these caches), ~1e-3 at most, whatever the sharpness of the scores.
PREFILL_QUALITY = 2e-3


def _prefill_check(o, lse, o_ref, lse_ref, label):
    err = max_abs(o, o_ref)
    lerr = lse_err(lse, lse_ref)
    note(f"{label}: max|o-o_ref| = {err:.3e}  max|lse-lse_ref| = {lerr:.3e}")
    assert err <= TOL["bf16"], (label, err)
    assert err <= PREFILL_QUALITY, (label, err)
    assert lerr <= 1e-2, (label, lerr)


@pytest.mark.parametrize("B,N,dr", [(3, 90, 16), (3, 400, 32), (3, 1500, 64)])
def test_prefill_absorb_matches_oracle(B, N, dr):
    # every prompt row absorbed and rotated at its own position L-N+i
    # (1200 rows: 32 rows per workgroup; 4500 rows: 64 per workgroup, each
    # with a ragged last block)
    w = gva_inputs.Workload("prefill", B, 2048, 8, 2, 128, 96, dr, dtype="bf16")
    lens = torch.tensor([2048, 1600, N], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 41, lens=lens)
    q = gva_inputs.prefill_queries(w, 41, N)
    pos1 = (lens.view(B, 1) - N + torch.arange(N, dtype=torch.int32).view(1, N) + 1).reshape(-1)
    qa_ref, qr_ref = oracle.absorb(q.reshape(B * N, w.n_heads, -1), inp["m"], pos1.to(torch.int32), d_r=dr)
    d = dims_of(w)
    qa = torch.empty(B, N, w.n_heads, w.d_v, dtype=torch.float32, device="cuda")
    qr = torch.full((B, N, w.n_heads, dr), float("nan"), dtype=torch.float32, device="cuda")
    note(f"prefill absorb B={B} N={N} dr={dr}")
    gva.gva_prefill_absorb(d, N, q.cuda(), inp["m"].cuda(), lens.cuda(), qa, qr)
    torch.cuda.synchronize()
    qa, qr = qa.cpu().reshape(B * N, w.n_heads, -1), qr.cpu().reshape(B * N, w.n_heads, -1)
    assert max_abs(qa, qa_ref) <= 1e-5 * float(qa_ref.abs().max())
    assert max_abs(qr, qr_ref) <= 1e-6 * float(qr_ref.abs().max())


@pytest.mark.parametrize("hpg,dv,dr", [(1, 64, 16), (2, 128, 16), (4, 64, 0), (4, 128, 16),
                                       (8, 64, 32), (8, 128, 64)])
def test_prefill_matches_oracle(hpg, dv, dr):
    G = 2
    w = gva_inputs.Workload("prefill", 3, 320, G * hpg, G, dv, dv, dr, dtype="bf16")
    N = 100
    lens = torch.tensor([320, 150, 60], dtype=torch.int32)   # 60 < N: 40 rows see nothing
    inp = gva_inputs.make_inputs(w, 23, lens=lens)
    for b, L in enumerate(lens.tolist()):                     # rows past a length are never read
        inp["v"][b, :, L:] = float("nan")
        inp["kr"][b, L:] = float("nan")
    q = gva_inputs.prefill_queries(w, 23, N)
    note(f"prefill hpg={hpg} dv={dv} dr={dr}: oracle")
    o_ref, lse_ref = oracle.prefill(q, inp["m"], inp["v"], inp["kr"], lens, rope_base=w.rope_base)
    dev = upload({k: inp[k] for k in ("m", "v", "kr", "lens")})
    d = dims_of(w)
    note(f"prefill hpg={hpg} dv={dv} dr={dr}: GPU")
    o, lse = gva.prefill(d, q.cuda(), dev["m"], dev["v"], dev["kr"], dev["lens"])
    torch.cuda.synchronize()
    _prefill_check(o.cpu(), lse.cpu(), o_ref, lse_ref, f"prefill/hpg{hpg}/dv{dv}/dr{dr}")


@pytest.mark.parametrize("qscale", [2.5, 6.0])
def test_prefill_sharp_scores(qscale):
    # queries scaled by 2.5 and 6: scores spread that much wider than the
    # workloads'.  The running maximum keeps growing by less than the
    # lazy-rescale threshold, so weights run above 1 between rescales.  A
    # query rounded once to bf16 moves each logit by a fixed fraction of its
    # size (4.1e-2 max error at a scale of 6); the high + low pairs hold the
    # same bounds as at scale 1.
    w = gva_inputs.Workload("prefill", 2, 640, 8, 2, 128, 128, 16, dtype="bf16")
    N = 200
    lens = torch.tensor([640, 333], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 43, lens=lens)
    q = (gva_inputs.prefill_queries(w, 43, N).float() * qscale).to(torch.bfloat16)
    o_ref, lse_ref = oracle.prefill(q, inp["m"], inp["v"], inp["kr"], lens, rope_base=w.rope_base)
    dev = upload({k: inp[k] for k in ("m", "v", "kr", "lens")})
    note(f"prefill sharp scores x{qscale}: GPU")
    o, lse = gva.prefill(dims_of(w), q.cuda(), dev["m"], dev["v"], dev["kr"], dev["lens"])
    torch.cuda.synchronize()
    _prefill_check(o.cpu(), lse.cpu(), o_ref, lse_ref, f"prefill sharp scores x{qscale}")


# Prompts large enough that the launch takes the columns-per-wave prefill
# kernel (d_v = 128, d_r <= 32, at least 2 workgroups per CU -- 4 at
# H/G = 8 -- of 4 x 32 columns): (B, H/G, G, d_r, N, prefix rows of the
# other sequences, query scale).
PREFILL_WAVE_CASES = [
    (4, 4, 4, 16, 1024, 300, 1.0),
    (4, 8, 2, 16, 2048, 0, 1.0),
    (4, 1, 8, 0, 2048, 77, 1.0),
    (4, 2, 4, 32, 2048, 500, 1.0),
    (4, 4, 4, 16, 1024, 0, 6.0),
]


@pytest.mark.slow
@pytest.mark.parametrize("B,hpg,G,dr,N,prefix,qscale", PREFILL_WAVE_CASES)
def test_prefill_columns_per_wave_matches_oracle(B, hpg, G, dr, N, prefix, qscale):
    # every row of every prompt against the oracle; the first sequence's
    # prompt fills its cache from row 0, the others follow a cached prefix,
    # and rows past every length hold NaN
    n_cu = gva.device_cu_count()
    items = B * G * -(-N // (128 // hpg))
    assert items >= (4 if hpg >= 8 else 2) * n_cu, "the shape must take the columns-per-wave kernel"
    T = -(-(N + prefix) // 32) * 32              # the tiled layout's capacity granularity
    w = gva_inputs.Workload("prefill_wave", B, T, hpg * G, G, 128, 128, dr, dtype="bf16")
    lens = torch.tensor([N] + [N + prefix] * (B - 1), dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 47, lens=lens)
    for b, L in enumerate(lens.tolist()):
        inp["v"][b, :, L:] = float("nan")
        inp["kr"][b, L:] = float("nan")
    q = (gva_inputs.prefill_queries(w, 47, N).float() * qscale).to(torch.bfloat16)
    note(f"prefill per wave B={B} hpg={hpg} G={G} dr={dr} N={N}: oracle")
    o_ref, lse_ref = oracle.prefill(q, inp["m"], inp["v"], inp["kr"], lens, rope_base=w.rope_base)
    dev = upload({k: inp[k] for k in ("m", "v", "kr", "lens")})
    note(f"prefill per wave B={B} hpg={hpg} G={G} dr={dr} N={N}: GPU")
    o, lse = gva.prefill(dims_of(w), q.cuda(), dev["m"], dev["v"], dev["kr"], dev["lens"])
    torch.cuda.synchronize()
    _prefill_check(o.cpu(), lse.cpu(), o_ref, lse_ref, f"prefill per wave hpg{hpg} G{G} dr{dr} N{N} x{qscale}")


# The matched-GQA prefill at sizes that take its columns-per-wave kernel
# (16 columns per wave): (B, H/G, G, N, prefix rows of the other sequences).
GQA_PREFILL_WAVE_CASES = [
    (4, 4, 4, 512, 100),
    (4, 8, 2, 1024, 0),
    (4, 1, 8, 1024, 50),
]


@pytest.mark.slow
@pytest.mark.parametrize("B,hpg,G,N,prefix", GQA_PREFILL_WAVE_CASES)
def test_gqa_prefill_columns_per_wave_matches_oracle(B, hpg, G, N, prefix):
    # sampled prompt rows (every seventh and the last) as GQA decode steps of
    # the oracle over the rows each sees
    n_cu = gva.device_cu_count()
    items = B * G * -(-N // (64 // hpg))
    assert items >= (4 if hpg >= 8 else 2) * n_cu, "the shape must take the columns-per-wave kernel"
    T = -(-(N + prefix) // 32) * 32
    w = gva_inputs.Workload("gqa_prefill_wave", B, T, G * hpg, G, 128, 128, 0, dtype="bf16", gqa=True)
    lens = torch.tensor([N] + [N + prefix] * (B - 1), dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 53, lens=lens)
    q = gva_inputs.prefill_queries(w, 53, N, gqa=True)
    dev = upload({k: inp[k] for k in ("v", "k_gqa", "lens")})
    d = dims_of(w)
    o = torch.empty(B, N, w.n_heads, 128, dtype=torch.float32, device="cuda")
    lse = torch.empty(B, N, w.n_heads, dtype=torch.float32, device="cuda")
    note(f"gqa prefill per wave B={B} hpg={hpg} G={G} N={N}")
    gva.gva_gqa_prefill_attention(d, N, q.cuda(), dev["k_gqa"], dev["v"], dev["lens"], o, lse)
    torch.cuda.synchronize()
    o, lse = o.cpu(), lse.cpu()
    rows = sorted(set(range(0, N, 7)) | {N - 1})
    o_ref = torch.zeros(B, len(rows), w.n_heads, 128, dtype=torch.float64)
    lse_ref = torch.full((B, len(rows), w.n_heads), float("-inf"), dtype=torch.float64)
    for r, i in enumerate(rows):
        p = lens - N + i
        oi, li = oracle.gqa_decode(q[:, i].contiguous(), inp["k_gqa"], inp["v"], (p + 1).clamp(min=0), d_k=128)
        o_ref[:, r] = oi
        lse_ref[:, r] = li
    idx = torch.tensor(rows)
    _prefill_check(o[:, idx], lse[:, idx], o_ref, lse_ref, f"gqa prefill per wave hpg{hpg} G{G} N{N}")


def test_prefill_after_append_of_the_prompt():
    # Algorithm 1's append for every prompt row (gva_append_kv), then the
    # prefill over the appended caches, against the oracle doing the same
    w = gva_inputs.Workload("prefill", 2, 256, 8, 2, 128, 128, 16, dtype="bf16")
    N = 70
    lens = torch.tensor([200, 70], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 29, lens=lens)
    g = torch.Generator().manual_seed(31)
    v_new = torch.randn(w.batch * N, w.n_groups, w.d_v, generator=g).to(torch.bfloat16)
    kr_new = torch.randn(w.batch * N, w.d_r, generator=g).to(torch.bfloat16)
    seq = torch.arange(w.batch, dtype=torch.int32).repeat_interleave(N)
    pos = (lens.repeat_interleave(N) - N + torch.arange(N, dtype=torch.int32).repeat(w.batch)).to(torch.int32)
    v_ref, k_ref = inp["v"].clone(), inp["kr"].clone()
    oracle.append(v_ref, k_ref, v_new, kr_new, seq, pos, rope_base=w.rope_base)
    q = gva_inputs.prefill_queries(w, 29, N)
    o_ref, lse_ref = oracle.prefill(q, inp["m"], v_ref, k_ref, lens, rope_base=w.rope_base)
    dev = upload({k: inp[k] for k in ("m", "v", "kr", "lens")})
    d = dims_of(w)
    note("prefill after append: GPU")
    gva.gva_append_kv(d, dev["v"], dev["kr"], v_new.cuda(), kr_new.cuda(), seq.cuda(), pos.cuda())
    o, lse = gva.prefill(d, q.cuda(), dev["m"], dev["v"], dev["kr"], dev["lens"])
    torch.cuda.synchronize()
    _prefill_check(o.cpu(), lse.cpu(), o_ref, lse_ref, "prefill after append")


@pytest.mark.parametrize("hpg,dv", [(1, 64), (4, 128), (8, 64)])
def test_gqa_prefill_matches_oracle(hpg, dv):
    # the matched-GQA prefill row by row: row i is a GQA decode step over
    # the first p+1 rows (the oracle's GQA definition)
    G = 2
    w = gva_inputs.Workload("gqa_prefill", 2, 192, G * hpg, G, dv, dv, 0, dtype="bf16", gqa=True)
    N = 50
    lens = torch.tensor([192, 30], dtype=torch.int32)
    inp = gva_inputs.make_inputs(w, 37, lens=lens)
    q = gva_inputs.prefill_queries(w, 37, N, gqa=True)
    dev = upload({k: inp[k] for k in ("v", "k_gqa", "lens")})
    d = dims_of(w)
    o = torch.empty(w.batch, N, w.n_heads, dv, dtype=torch.float32, device="cuda")
    lse = torch.empty(w.batch, N, w.n_heads, dtype=torch.float32, device="cuda")
    note(f"gqa prefill hpg={hpg} dv={dv}")
    gva.gva_gqa_prefill_attention(d, N, q.cuda(), dev["k_gqa"], dev["v"], dev["lens"], o, lse)
    torch.cuda.synchronize()
    o, lse = o.cpu(), lse.cpu()
    o_ref = torch.zeros(w.batch, N, w.n_heads, dv, dtype=torch.float64)
    lse_ref = torch.full((w.batch, N, w.n_heads), float("-inf"), dtype=torch.float64)
    for i in range(N):
        p = lens - N + i
        live = p >= 0
        if not live.any():
            continue
        oi, li = oracle.gqa_decode(q[:, i].contiguous(), inp["k_gqa"], inp["v"], (p + 1).clamp(min=0),
                                   d_k=dv)
        o_ref[live, i] = oi[live]
        lse_ref[live, i] = li[live]
    _prefill_check(o, lse, o_ref, lse_ref, f"gqa prefill/hpg{hpg}/dv{dv}")


@pytest.mark.slow
def test_prefill_full_size_sampled():
    # a 4096-token prompt at the bandwidth-headline head shapes (H32, G8,
    # d 128/128/16): every output finite, sampled rows against decode steps
    # of the oracle over the truncated cache
    w = gva_inputs.workload("b32_t8k").replace(name="prefill_b1_t4k", batch=1, t_max=4096)
    N = 4096
    inp = gva_inputs.make_inputs(w, 0, lens=torch.tensor([N], dtype=torch.int32))
    q = gva_inputs.prefill_queries(w, 0, N)
    dev = upload({k: inp[k] for k in ("m", "v", "kr", "lens")})
    d = dims_of(w)
    note("prefill b1 t4k: GPU")
    o, lse = gva.prefill(d, q.cuda(), dev["m"], dev["v"], dev["kr"], dev["lens"])
    o, lse = o.cpu(), lse.cpu()
    assert torch.isfinite(o).all() and torch.isfinite(lse).all()
    for i in (0, 1, 31, 32, 1000, 2047, 4095):
        note(f"prefill b1 t4k: oracle row {i}")
        o_ref, lse_ref = oracle.decode(q[:, i].contiguous(), inp["m"], inp["v"], inp["kr"],
                                       torch.tensor([i + 1], dtype=torch.int32))
        _prefill_check(o[:, i], lse[:, i], o_ref, lse_ref, f"prefill b1 t4k/row{i}")
