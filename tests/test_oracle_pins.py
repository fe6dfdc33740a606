"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself: each check goes through an
independent route (explicit key reconstruction K_h = V_g(h) M_h fed to
torch's textbook scaled-dot-product attention, the complex-exponential form
of RoPE, closed forms, exact rational rounding, figures the paper prints).
"""

import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from splits import split_bounds

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- references
def rope_complex(x, pos, base=10000.0):
    """RoFormer's complex form: pair (x_2i, x_2i+1) as x_2i + i x_2i+1 times
    exp(i * pos * base^(-2i/d))."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    if d == 0:
        return x.copy()
    theta = base ** (-np.arange(0, d, 2, dtype=np.float64) / d)
    z = (x[..., 0::2] + 1j * x[..., 1::2]) * np.exp(1j * pos * theta)
    out = np.empty_like(x)
    out[..., 0::2] = z.real
    out[..., 1::2] = z.imag
    return out


def explicit_decode(q, m, v, kr, lens, scale=None, base=10000.0):
    """Materialise K_h = V_g(h) M_h (eq. kvm / knope), concatenate the shared
    rotated key (eq. krope), and run textbook SDPA in float64."""
    q, m, v, kr = (t.to(torch.float64) for t in (q, m, v, kr))
    B, G, T, dv = v.shape
    H = q.shape[1]
    dc = m.shape[2]
    dr = kr.shape[-1]
    hpg = H // G
    scale = 1.0 / math.sqrt(dc + dr) if scale is None else scale
    o = torch.zeros(B, H, dv, dtype=torch.float64)
    lse = torch.full((B, H), -math.inf, dtype=torch.float64)
    for b in range(B):
        L = int(lens[b])
        if L == 0:
            continue
        for h in range(H):
            g = h // hpg
            K = v[b, g, :L] @ m[h]                               # [L, d_c]
            Kfull = torch.cat([K, kr[b, :L]], dim=1)             # [L, d_c+d_r]
            qr = torch.from_numpy(rope_complex(q[b, h, dc:].numpy(), L - 1, base))
            qfull = torch.cat([q[b, h, :dc], qr])
            o[b, h] = F.scaled_dot_product_attention(
                qfull.view(1, 1, 1, -1), Kfull.view(1, 1, L, -1),
                v[b, g, :L].reshape(1, 1, L, dv), scale=scale).view(dv)
            lse[b, h] = torch.logsumexp((Kfull @ qfull) * scale, dim=0)
    return o, lse


def tiny_inputs(seed, B=2, H=4, G=2, T=37, dv=16, dc=12, dr=8, lens=None,
                dtype=torch.float64):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn(B, H, dc + dr, generator=g, dtype=torch.float64)
    v = torch.randn(B, G, T, dv, generator=g, dtype=torch.float64)
    kr = torch.randn(B, T, dr, generator=g, dtype=torch.float64)
    m = torch.randn(H, dv, dc, generator=g, dtype=torch.float64) / math.sqrt(dv)
    if lens is None:
        lens = torch.randint(1, T + 1, (B,), generator=g, dtype=torch.int32)
    return [t.to(dtype) for t in (q, m, v, kr)] + [torch.as_tensor(lens, dtype=torch.int32)]


# ------------------------------------------------------ absorption + scores
@pytest.mark.parametrize("dr", [0, 4, 8])
@pytest.mark.parametrize("H,G", [(4, 2), (4, 1), (4, 4), (6, 3)])
def test_absorbed_matches_explicit_reconstruction(orc, dr, H, G):
    # non-square M (d_v=16, d_c=12) so a transposed map cannot pass
    q, m, v, kr, lens = tiny_inputs(7 + dr + 10 * H + G, H=H, G=G, dr=dr)
    o, lse = orc.decode(q, m, v, kr, lens)
    o_ref, lse_ref = explicit_decode(q, m, v, kr, lens)
    assert torch.allclose(o, o_ref, rtol=0, atol=1e-12)
    assert torch.allclose(lse, lse_ref, rtol=0, atol=1e-12)


def test_absorbed_query_is_q_times_m_transpose(orc):
    q, m, v, kr, lens = tiny_inputs(3)
    qa, qr = orc.absorb(q, m, lens, d_r=kr.shape[-1])
    dc = m.shape[2]
    for b in range(q.shape[0]):
        for h in range(q.shape[1]):
            # eq. absorb as a matrix-vector product in numpy
            want = q[b, h, :dc].numpy() @ m[h].numpy().T
            np.testing.assert_allclose(qa[b, h].numpy(), want, rtol=0, atol=1e-13)
            want_r = rope_complex(q[b, h, dc:].numpy(), int(lens[b]) - 1)
            np.testing.assert_allclose(qr[b, h].numpy(), want_r, rtol=0, atol=1e-13)


def test_bf16_storage_upcast_is_exact(orc):
    q, m, v, kr, lens = tiny_inputs(11, dtype=torch.bfloat16)
    o, lse = orc.decode(q, m, v, kr, lens)
    o_ref, lse_ref = explicit_decode(q, m, v, kr, lens)
    assert torch.allclose(o, o_ref, rtol=0, atol=1e-12)
    assert torch.allclose(lse, lse_ref, rtol=0, atol=1e-12)


# ------------------------------------------------------------------ softmax
def test_weights_sum_to_one_and_match_softmax(orc):
    # V = identity rows (d_v = T) makes o equal the attention weights.
    T, dc, dr = 9, 5, 4
    g = torch.Generator().manual_seed(5)
    q = torch.randn(1, 2, dc + dr, generator=g, dtype=torch.float64)
    m = torch.randn(2, T, dc, generator=g, dtype=torch.float64)
    kr = torch.randn(1, T, dr, generator=g, dtype=torch.float64)
    v = torch.eye(T, dtype=torch.float64).view(1, 1, T, T)
    lens = torch.tensor([T], dtype=torch.int32)
    o, lse = orc.decode(q, m, v, kr, lens)
    assert torch.allclose(o.sum(-1), torch.ones(1, 2, dtype=torch.float64), atol=1e-13)
    for h in range(2):
        K = torch.cat([m[h], kr[0]], dim=1)      # V = I, so K_h = M_h
        qf = torch.cat([q[0, h, :dc],
                        torch.from_numpy(rope_complex(q[0, h, dc:].numpy(), T - 1))])
        w = torch.softmax(K @ qf / math.sqrt(dc + dr), dim=0)
        assert torch.allclose(o[0, h], w, rtol=0, atol=1e-14)


def test_zero_query_gives_mean_value(orc):
    q, m, v, kr, lens = tiny_inputs(13)
    q.zero_()
    o, lse = orc.decode(q, m, v, kr, lens)
    for b in range(q.shape[0]):
        L = int(lens[b])
        for h in range(q.shape[1]):
            g = h // (q.shape[1] // v.shape[1])
            assert torch.allclose(o[b, h], v[b, g, :L].mean(0), rtol=0, atol=1e-14)
            assert abs(float(lse[b, h]) - math.log(L)) < 1e-14


def test_single_row_returns_that_value(orc):
    q, m, v, kr, _ = tiny_inputs(17)
    lens = torch.tensor([1, 1], dtype=torch.int32)
    o, _ = orc.decode(q, m, v, kr, lens)
    for b in range(2):
        for h in range(4):
            assert torch.equal(o[b, h], v[b, h // 2, 0])


def test_two_rows_closed_form(orc):
    q, m, v, kr, _ = tiny_inputs(19)
    lens = torch.tensor([2, 2], dtype=torch.int32)
    o, _ = orc.decode(q, m, v, kr, lens)
    dc, dr = m.shape[2], kr.shape[-1]
    c = 1 / math.sqrt(dc + dr)
    for b in range(2):
        for h in range(4):
            g = h // 2
            qr = rope_complex(q[b, h, dc:].numpy(), 1)
            s = [c * (float(q[b, h, :dc] @ (v[b, g, t] @ m[h])) + float(np.dot(qr, kr[b, t].numpy())))
                 for t in range(2)]
            sig = 1 / (1 + math.exp(s[1] - s[0]))
            want = sig * v[b, g, 0] + (1 - sig) * v[b, g, 1]
            assert torch.allclose(o[b, h], want, rtol=0, atol=1e-14)


def test_empty_sequence(orc):
    q, m, v, kr, _ = tiny_inputs(23)
    lens = torch.tensor([0, 5], dtype=torch.int32)
    o, lse = orc.decode(q, m, v, kr, lens)
    assert torch.all(o[0] == 0) and torch.all(torch.isinf(lse[0])) and torch.all(lse[0] < 0)
    assert torch.all(torch.isfinite(lse[1]))


# ---------------------------------------------------------- special cases
def test_no_positional_slice_is_content_attention(orc):
    # d_r = 0 (value-only GVA): softmax(q~ V^T / sqrt(d_c)) V
    q, m, v, kr, lens = tiny_inputs(29, dr=0)
    o, _ = orc.decode(q, m, v, kr, lens)
    for b in range(2):
        L = int(lens[b])
        for h in range(4):
            g = h // 2
            K = v[b, g, :L] @ m[h]
            ref = F.scaled_dot_product_attention(q[b, h].view(1, 1, 1, -1), K.view(1, 1, L, -1),
                                                 v[b, g, :L].reshape(1, 1, L, -1)).view(-1)
            assert torch.allclose(o[b, h], ref, rtol=0, atol=1e-13)


def test_identity_map_is_shared_kv_attention(orc):
    # M_h = I, d_r = 0, d_c = d_v: keys equal values (the shared-KV cut)
    dv = 12
    q, _, v, kr, lens = tiny_inputs(31, dv=dv, dc=dv, dr=0)
    m = torch.eye(dv, dtype=torch.float64).expand(4, dv, dv).contiguous()
    o, _ = orc.decode(q, m, v, kr, lens)
    for b in range(2):
        L = int(lens[b])
        for h in range(4):
            vv = v[b, h // 2, :L].reshape(1, 1, L, dv)
            ref = F.scaled_dot_product_attention(q[b, h].view(1, 1, 1, dv), vv, vv).view(dv)
            assert torch.allclose(o[b, h], ref, rtol=0, atol=1e-13)


# -------------------------------------------------------------------- RoPE
def test_rope_matches_complex_form_and_invariants(orc):
    g = torch.Generator().manual_seed(37)
    for dr in (2, 8, 16, 32):
        x = torch.randn(dr, generator=g, dtype=torch.float64)
        assert torch.equal(orc.rope(x, 0), x)                       # R_0 = I
        for pos in (1, 17, 1000, 131071):
            y = orc.rope(x, pos)
            # the angle pos*theta carries one fp64 ulp (~2e-16 * pos) in both forms
            tol = 1e-13 + 4e-16 * pos * float(x.abs().max())
            np.testing.assert_allclose(y.numpy(), rope_complex(x.numpy(), pos), rtol=0, atol=tol)
            assert abs(float(y.norm()) - float(x.norm())) < 1e-12   # rotation
    # 2-D closed form: theta_0 = 1, so (1, 0) at position p is (cos p, sin p)
    y = orc.rope(torch.tensor([1.0, 0.0], dtype=torch.float64), 3)
    assert abs(float(y[0]) - math.cos(3)) < 1e-15 and abs(float(y[1]) - math.sin(3)) < 1e-15


def test_rope_relative_position(orc):
    # <x R_p^T, y R_t^T> = x R_{t-p} y^T depends on t - p only
    g = torch.Generator().manual_seed(41)
    x = torch.randn(16, generator=g, dtype=torch.float64)
    y = torch.randn(16, generator=g, dtype=torch.float64)
    ref = float(orc.rope(x, 100) @ orc.rope(y, 93))
    for p in (7, 250, 4096, 90000):
        assert abs(float(orc.rope(x, p) @ orc.rope(y, p - 7)) - ref) < 1e-11


def test_position_shift_leaves_output_unchanged(orc):
    # Rotate the same raw keys at positions t and t + D (through the append
    # step) and place the query at L-1 and L-1+D: relative positions agree.
    B, G, H, T, dv, dc, dr, D = 1, 2, 4, 20, 8, 6, 8, 1234
    g = torch.Generator().manual_seed(43)
    q = torch.randn(B, H, dc + dr, generator=g, dtype=torch.float64)
    m = torch.randn(H, dv, dc, generator=g, dtype=torch.float64)
    vraw = torch.randn(T, G, dv, generator=g, dtype=torch.float64)
    kraw = torch.randn(T, dr, generator=g, dtype=torch.float64)

    def build(offset):
        Tm = T + offset
        v = torch.zeros(B, G, Tm, dv, dtype=torch.float64)
        kr = torch.zeros(B, Tm, dr, dtype=torch.float64)
        pos = torch.arange(T, dtype=torch.int32) + offset
        orc.append(v, kr, vraw, kraw, torch.zeros(T, dtype=torch.int32), pos)
        return v, kr, Tm

    v0, k0, _ = build(0)
    v1, k1, Tm = build(D)
    o0, l0 = orc.decode(q, m, v0, k0, torch.tensor([T], dtype=torch.int32))
    o1, l1 = orc.decode(q, m, v1, k1, torch.tensor([Tm], dtype=torch.int32),
                        t_begin=torch.tensor([D], dtype=torch.int32))
    assert torch.allclose(o0, o1, rtol=0, atol=1e-12)
    assert torch.allclose(l0, l1, rtol=0, atol=1e-11)


# ----------------------------------------------------------- split/combine
@pytest.mark.parametrize("S,rows", [(1, 0), (2, 0), (3, 0), (7, 0), (64, 0),
                                    (5, 32), (2, 32), (20, 8), (1, 64)])
def test_split_and_combine_equals_unsplit(orc, S, rows):
    # even splits, and bounded chunks (including too few splits, where the
    # S splits share the rows evenly and exceed the bound)
    q, m, v, kr, lens = tiny_inputs(47, T=150, lens=[150, 61])
    o, lse = orc.decode(q, m, v, kr, lens)
    begins, ends = split_bounds(lens, S, tile=8, split_rows=rows)
    parts = [orc.decode(q, m, v, kr, lens, t_begin=bg, t_end=en) for bg, en in zip(begins, ends)]
    o_part = torch.stack([p[0] for p in parts], dim=2)     # [B,H,S,dv]
    lse_part = torch.stack([p[1] for p in parts], dim=2)   # [B,H,S]
    oc, lc = orc.combine(o_part, lse_part)
    assert torch.allclose(oc, o, rtol=0, atol=1e-12)
    assert torch.allclose(lc, lse, rtol=0, atol=1e-12)


@pytest.mark.parametrize("rows", [0, 32, 256])
def test_split_bounds_cover_each_sequence(orc, rows):
    lens = torch.tensor([0, 1, 31, 32, 33, 1000, 8192], dtype=torch.int32)
    for S in (1, 2, 5, 16):
        begins, ends = split_bounds(lens, S, tile=32, split_rows=rows)
        for b in range(lens.numel()):
            covered, sizes = [], []
            L = int(lens[b])
            for s in range(S):
                bg, en = int(begins[s][b]), int(ends[s][b])
                assert bg % 32 == 0 or bg == L
                if rows and -(-L // rows) <= S:
                    assert en - bg <= rows          # bounded chunks
                covered.extend(range(bg, en))
                sizes.append(en - bg)
            assert covered == list(range(L))
            # the splits with rows come first, all of one size but the last
            nz = [z for z in sizes if z > 0]
            assert sizes[:len(nz)] == nz and len(set(nz[:-1])) <= 1 and (not nz or nz[-1] <= nz[0])
            if rows and L > 0:
                assert len(nz) == min(S, -(-L // rows))


# ------------------------------------------------------------------ append
def _nearest_bf16_bits(x: float) -> int:
    """Nearest bfloat16 to x by exact rational comparison of its neighbours."""
    f = np.float32(x)
    bits = int(np.array([f]).view(np.uint32)[0]) >> 16
    cands = {(bits + d) & 0xFFFF for d in (-1, 0, 1, 2)}
    fx = Fraction(x)
    best = None
    for c in sorted(cands):
        cv = float(np.array([c << 16], dtype=np.uint32).view(np.float32)[0])
        if not math.isfinite(cv):
            continue
        key = (abs(Fraction(cv) - fx), c & 1)   # nearest, then even mantissa
        if best is None or key < best[0]:
            best = (key, c)
    return best[1]


def test_round_bf16_single_rounding(orc):
    # ties go to even; a double just above a tie must round up even though
    # rounding first to float32 would land on the tie (double rounding)
    one = 0x3F80
    assert orc.round_bf16_bits(1.0 + 2.0 ** -8) == one
    assert orc.round_bf16_bits(1.0 + 3 * 2.0 ** -8) == one + 2
    assert orc.round_bf16_bits(1.0 + 2.0 ** -8 + 2.0 ** -40) == one + 1
    assert orc.round_bf16_bits(-(1.0 + 2.0 ** -8 + 2.0 ** -40)) == 0x8000 | (one + 1)
    assert orc.round_bf16_bits(0.0) == 0 and orc.round_bf16_bits(-0.0) == 0x8000
    # the largest finite bf16 is 2^128 - 2^120; halfway to 2^128 is 2^128 - 2^119
    assert orc.round_bf16_bits(2.0 ** 128 - 2.0 ** 119 - 2.0 ** 100) == 0x7F7F
    assert orc.round_bf16_bits(2.0 ** 128 - 2.0 ** 119 + 2.0 ** 100) == 0x7F80   # +inf
    g = torch.Generator().manual_seed(53)
    x32 = torch.randn(4000, generator=g) * torch.exp2(torch.randint(-20, 20, (4000,), generator=g).float())
    ref = x32.to(torch.bfloat16).view(torch.int16).to(torch.int32) & 0xFFFF
    got = torch.tensor([orc.round_bf16_bits(float(x)) for x in x32], dtype=torch.int32)
    assert torch.equal(got, ref)
    x64 = torch.randn(500, generator=g, dtype=torch.float64)
    for x in x64.tolist():
        assert orc.round_bf16_bits(x) == _nearest_bf16_bits(x)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_append_writes_rows_and_rotated_key(orc, dtype):
    B, G, T, dv, dr = 3, 2, 40, 8, 16
    g = torch.Generator().manual_seed(59)
    v = torch.zeros(B, G, T, dv, dtype=dtype)
    kr = torch.zeros(B, T, dr, dtype=dtype)
    n = 6
    v_new = torch.randn(n, G, dv, generator=g).to(dtype)
    k_new = torch.randn(n, dr, generator=g).to(dtype)
    seq = torch.tensor([0, 2, 1, 0, 5, 2], dtype=torch.int32)     # row 4: bad seq
    pos = torch.tensor([0, 39, 17, 3, 1, 40], dtype=torch.int32)  # row 5: bad pos
    skipped = orc.append(v, kr, v_new, k_new, seq, pos)
    assert skipped == 2
    for r in range(4):
        b, p = int(seq[r]), int(pos[r])
        assert torch.equal(v[b, :, p], v_new[r])
        rot = rope_complex(k_new[r].double().numpy(), p)
        if dtype == torch.float32:
            want = torch.from_numpy(rot.astype(np.float32))
            assert torch.equal(kr[b, p], want)
        else:
            want = torch.tensor([_nearest_bf16_bits(float(x)) for x in rot], dtype=torch.int32)
            got = kr[b, p].view(torch.int16).to(torch.int32) & 0xFFFF
            assert torch.equal(got, want)
    written = {(int(seq[r]), int(pos[r])) for r in range(4)}
    for b in range(B):
        for p in range(T):
            if (b, p) not in written:
                assert torch.all(v[b, :, p] == 0) and torch.all(kr[b, p] == 0)


# -------------------------------------------------------------- GQA oracle
def test_gqa_oracle_is_textbook_sdpa(orc):
    g = torch.Generator().manual_seed(61)
    B, H, G, T, d = 2, 4, 2, 30, 16
    q = torch.randn(B, H, d + 4, generator=g, dtype=torch.float64)
    k = torch.randn(B, G, T, d, generator=g, dtype=torch.float64)
    v = torch.randn(B, G, T, d, generator=g, dtype=torch.float64)
    lens = torch.tensor([30, 11], dtype=torch.int32)
    o, lse = orc.gqa_decode(q, k, v, lens, d_k=d)
    for b in range(B):
        L = int(lens[b])
        for h in range(H):
            kk = k[b, h // 2, :L].reshape(1, 1, L, d)
            vv = v[b, h // 2, :L].reshape(1, 1, L, d)
            ref = F.scaled_dot_product_attention(q[b, h, :d].view(1, 1, 1, d), kk, vv).view(d)
            assert torch.allclose(o[b, h], ref, rtol=0, atol=1e-13)


# ------------------------------------- GVA without decoupled RoPE (Sec. 3.2)
def explicit_rope_decode(q, m, v, lens, scale=None, base=10000.0, shift=0):
    """Keys materialised as k_t = v_t M_h and rotated at t + shift over their
    whole width, the query rotated at L-1+shift, textbook SDPA in float64."""
    q, m, v = (t.to(torch.float64) for t in (q, m, v))
    B, G, T, dv = v.shape
    H, dc = q.shape[1], q.shape[2]
    hpg = H // G
    scale = 1.0 / math.sqrt(dc) if scale is None else scale
    o = torch.zeros(B, H, dv, dtype=torch.float64)
    lse = torch.full((B, H), -math.inf, dtype=torch.float64)
    for b in range(B):
        L = int(lens[b])
        if L == 0:
            continue
        for h in range(H):
            g = h // hpg
            K = (v[b, g, :L] @ m[h]).numpy()
            Kr = np.stack([rope_complex(K[t], t + shift, base) for t in range(L)])
            qr = rope_complex(q[b, h].numpy(), L - 1 + shift, base)
            Kt = torch.from_numpy(Kr)
            qt = torch.from_numpy(qr)
            o[b, h] = F.scaled_dot_product_attention(
                qt.view(1, 1, 1, dc), Kt.view(1, 1, L, dc),
                v[b, g, :L].reshape(1, 1, L, dv), scale=scale).view(dv)
            lse[b, h] = torch.logsumexp((Kt @ qt) * scale, dim=0)
    return o, lse


def rope_tiny_inputs(seed, B=2, H=4, G=2, T=29, dv=16, dc=12, lens=None):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn(B, H, dc, generator=g, dtype=torch.float64)
    v = torch.randn(B, G, T, dv, generator=g, dtype=torch.float64)
    m = torch.randn(H, dv, dc, generator=g, dtype=torch.float64) / math.sqrt(dv)
    if lens is None:
        lens = torch.randint(1, T + 1, (B,), generator=g, dtype=torch.int32)
    return q, m, v, torch.as_tensor(lens, dtype=torch.int32)


@pytest.mark.parametrize("H,G", [(4, 2), (4, 1), (6, 3)])
def test_rope_decode_matches_explicit_construction(orc, H, G):
    # non-square M (d_v=16, d_c=12): a transposed map cannot pass
    q, m, v, lens = rope_tiny_inputs(71 + H + G, H=H, G=G, lens=[29, 9])
    o, lse = orc.rope_decode(q, m, v, lens)
    o_ref, lse_ref = explicit_rope_decode(q, m, v, lens)
    assert torch.allclose(o, o_ref, rtol=0, atol=1e-12)
    assert torch.allclose(lse, lse_ref, rtol=0, atol=1e-12)


def test_rope_decode_scores_are_a_relative_rotation(orc):
    # With pairs as complex numbers, RoPE(x, P) . RoPE(y, t) = Re(x conj(y)
    # e^{-i theta d}), d = t - P; per pair that is a cos(theta d) + b sin(theta d)
    # with a = x_2i y_2i + x_2i+1 y_2i+1 and b = x_2i+1 y_2i - x_2i y_2i+1.
    # A two-row cache with one zero row makes the weights that closed form.
    dc, dv, L = 8, 8, 2
    g = torch.Generator().manual_seed(73)
    q = torch.randn(1, 1, dc, generator=g, dtype=torch.float64)
    m = torch.eye(dv, dtype=torch.float64).view(1, dv, dc)
    v = torch.zeros(1, 1, L, dv, dtype=torch.float64)
    v[0, 0, 1] = torch.randn(dv, generator=g, dtype=torch.float64)
    o, lse = orc.rope_decode(q, m, v, torch.tensor([L], dtype=torch.int32))
    # row 1 is the query's own position: d = 0, the score is plain q . v_1
    s1 = float(q[0, 0] @ v[0, 0, 1]) / math.sqrt(dc)
    w1 = 1.0 / (1.0 + math.exp(-s1))              # row 0 scores 0
    assert torch.allclose(o[0, 0], w1 * v[0, 0, 1], rtol=0, atol=1e-14)
    assert abs(float(lse[0, 0]) - math.log(1.0 + math.exp(s1))) < 1e-14
    # move the nonzero row to position 0: d = -1 rotates each pair by -theta_i
    v2 = v.flip(2).contiguous()
    o2, _ = orc.rope_decode(q, m, v2, torch.tensor([L], dtype=torch.int32))
    x, y = q[0, 0].numpy(), v2[0, 0, 0].numpy()
    theta = 10000.0 ** (-np.arange(0, dc, 2, dtype=np.float64) / dc)
    dot = x[0::2] * y[0::2] + x[1::2] * y[1::2]
    cross = x[1::2] * y[0::2] - x[0::2] * y[1::2]
    s0 = float(np.sum(dot * np.cos(-theta) + cross * np.sin(-theta))) / math.sqrt(dc)
    w0 = 1.0 / (1.0 + math.exp(-s0))
    assert torch.allclose(o2[0, 0], w0 * v2[0, 0, 0], rtol=0, atol=1e-14)


def test_rope_decode_shift_and_edge_cases(orc):
    q, m, v, lens = rope_tiny_inputs(79, lens=[29, 1])
    o, lse = orc.rope_decode(q, m, v, lens)
    o2, lse2 = orc.rope_decode(q, m, v, lens, shift=4321)
    assert torch.allclose(o, o2, rtol=0, atol=1e-10)
    assert torch.allclose(lse, lse2, rtol=0, atol=1e-10)
    for h in range(4):                            # one row: its value, any query
        assert torch.allclose(o[1, h], v[1, h // 2, 0], rtol=0, atol=1e-15)
    o0, lse0 = orc.rope_decode(q, m, v, torch.tensor([0, 3], dtype=torch.int32))
    assert torch.all(o0[0] == 0) and torch.all(torch.isneginf(lse0[0]))
    # the rotation is not absorbable: the decoupled-RoPE decode with d_r = 0
    # (no rotation anywhere) gives a different result on the same inputs
    oa, _ = orc.decode(q, m, v, torch.zeros(2, v.shape[2], 0, dtype=torch.float64), lens)
    assert (oa[0] - o[0]).abs().max() > 1e-3


# ------------------------------------------------ prefill (causal, Sec. 3.3)
def _prefill_inputs(seed, B=2, N=5, H=4, G=2, T=37, dv=16, dc=12, dr=8, lens=(37, 3)):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn(B, N, H, dc + dr, generator=g, dtype=torch.float64)
    v = torch.randn(B, G, T, dv, generator=g, dtype=torch.float64)
    kr = torch.randn(B, T, dr, generator=g, dtype=torch.float64)
    m = torch.randn(H, dv, dc, generator=g, dtype=torch.float64) / math.sqrt(dv)
    return q, m, v, kr, torch.tensor(lens, dtype=torch.int32)


@pytest.mark.parametrize("H,G,dr", [(4, 2, 8), (4, 1, 0), (6, 3, 4)])
def test_prefill_matches_masked_explicit_attention(orc, H, G, dr):
    # explicit keys [V M_h, kr] over every cached row, a boolean causal mask
    # (t <= p) and textbook SDPA; rows whose position is negative are empty
    q, m, v, kr, lens = _prefill_inputs(83 + H + dr, H=H, G=G, dr=dr)
    B, N, _, W = q.shape
    dc, hpg = W - dr, H // G
    o, lse = orc.prefill(q, m, v, kr, lens)
    for b in range(B):
        L = int(lens[b])
        for i in range(N):
            p = L - N + i
            for h in range(H):
                if p < 0:
                    assert torch.all(o[b, i, h] == 0) and math.isinf(float(lse[b, i, h]))
                    continue
                g = h // hpg
                K = torch.cat([v[b, g, :L] @ m[h], kr[b, :L]], dim=1)
                qr = torch.from_numpy(rope_complex(q[b, i, h, dc:].numpy(), p))
                qf = torch.cat([q[b, i, h, :dc], qr])
                mask = (torch.arange(L) <= p).view(1, 1, 1, L)
                scale = 1.0 / math.sqrt(W)
                ref = F.scaled_dot_product_attention(qf.view(1, 1, 1, -1), K.view(1, 1, L, -1),
                                                     v[b, g, :L].reshape(1, 1, L, -1), attn_mask=mask,
                                                     scale=scale).view(-1)
                assert torch.allclose(o[b, i, h], ref, rtol=0, atol=1e-12)
                lref = torch.logsumexp((K[: p + 1] @ qf) * scale, dim=0)
                assert abs(float(lse[b, i, h]) - float(lref)) < 1e-12


def test_prefill_rows_are_decode_steps(orc):
    # Algorithm 1 run token by token: query i of the prompt is one decode step
    # over the first p+1 rows
    q, m, v, kr, lens = _prefill_inputs(89, lens=(37, 20))
    o, lse = orc.prefill(q, m, v, kr, lens)
    N = q.shape[1]
    for i in range(N):
        p = lens - N + i
        od, ld = orc.decode(q[:, i].contiguous(), m, v, kr, p + 1)
        assert torch.allclose(o[:, i], od, rtol=0, atol=1e-13)
        assert torch.allclose(lse[:, i], ld, rtol=0, atol=1e-13)


def test_prefill_first_prompt_row_is_its_value(orc):
    # a prompt that fills the cache from row 0: its first query sees one row
    q, m, v, kr, lens = _prefill_inputs(97, N=6, lens=(6, 6))
    o, _ = orc.prefill(q, m, v, kr, lens)
    for h in range(4):
        assert torch.equal(o[:, 0, h], v[:, h // 2, 0])


# ------------------------------------------------- figures the paper prints
def _golden_rows(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([float(x) for x in line.split()])
    return rows


def test_cache_savings_match_paper():
    from paper_2609_13285_amd import traffic
    for G, dh, dr, printed, tol in _golden_rows("paper_cache_savings.txt"):
        G, dh, dr = int(G), int(dh), int(dr)
        saved = 100.0 * (1.0 - traffic.cache_ratio(G, dh, dr))
        assert abs(saved - printed) <= tol, (G, dh, dr, saved, printed)
        T = 1000
        ratio = traffic.cache_scalars_gva(T, G, dh, dr) / traffic.cache_scalars_gqa(T, G, dh)
        assert abs(ratio - traffic.cache_ratio(G, dh, dr)) < 1e-15


def test_flat_attention_at_tiny_scale_matches_paper(orc):
    (n, sigma, printed, tol), = _golden_rows("flat_attention_10pos.txt")
    n = int(n)
    g = torch.Generator().manual_seed(67)
    # V = I makes the output the weight vector; with V = I the content keys
    # are the rows of M_h, drawn at scale sigma like the query.
    q = torch.randn(1, 1, n, generator=g, dtype=torch.float64) * sigma
    m = torch.randn(1, n, n, generator=g, dtype=torch.float64) * sigma
    v = torch.eye(n, dtype=torch.float64).view(1, 1, n, n)
    kr = torch.zeros(1, n, 0, dtype=torch.float64)
    o, _ = orc.decode(q, m, v, kr, torch.tensor([n], dtype=torch.int32))
    assert torch.all((o - printed).abs() <= tol)
