"""The C ABI without a GPU: libgva.so loads, exports every entry point that
include/gva.h declares, and host-side validation rejects bad arguments
before anything is enqueued (no compute call runs here)."""

import ctypes
import os
import re

import pytest

from paper_2609_13285_amd import gva

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gva.h")

# fake device pointers: aligned, never dereferenced because validation fails first
A = 0x10000


def declared_functions(header=HEADER):
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(gva_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_four_calls():
    names = declared_functions()
    for n in ("gva_append_kv", "gva_absorb_query", "gva_decode_attention", "gva_combine"):
        assert n in names
    assert set(names) == set(gva.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = gva.lib()
    probe_header = os.path.join(ROOT, "include", "gva_probe.h")
    assert set(declared_functions(probe_header)) == set(gva.PROBE_EXPORTS)
    for name in declared_functions() + declared_functions(probe_header):
        assert hasattr(lib, name), name
    # every header under include/ is one of the two
    assert sorted(os.listdir(os.path.join(ROOT, "include"))) == ["gva.h", "gva_probe.h"]
    assert gva.gva_version() == 20000


def test_status_strings():
    assert gva.status_string(0) == "ok"
    assert "invalid" in gva.status_string(-1)
    assert "unsupported" in gva.status_string(-2)
    assert "HIP" in gva.status_string(-3)
    assert (gva.GVA_ERR_INVALID_ARG, gva.GVA_ERR_UNSUPPORTED, gva.GVA_ERR_HIP) == (-1, -2, -3)
    assert gva.status_string(99) == "unknown status"


def dims(**kw):
    base = dict(batch=2, n_heads=8, n_groups=2, d_v=128, d_c=128, d_r=16, t_max=64,
                dtype="bf16", rope_base=10000.0, scale=0.0)
    base.update(kw)
    return gva.make_dims(**base)


def decode_status(d, S=4, q=A, m=A, qa=None, qr=None, v=A, kr=A, lens=A, op=A, lp=A, vn=None, kn=None,
                  rows=0):
    return gva.lib().gva_decode_attention(ctypes.byref(d), q, m, qa, qr, v, kr, lens, vn, kn, S, rows,
                                          op, lp, None)


@pytest.mark.parametrize("kw", [
    dict(batch=0), dict(n_heads=0), dict(n_groups=0), dict(t_max=0),
    dict(n_heads=6, n_groups=4),           # H not a multiple of G
    dict(d_r=15),                          # odd positional width
    dict(d_r=-2), dict(d_v=0), dict(dtype=7),
    dict(scale=-1.0), dict(scale=float("nan")), dict(rope_base=0.0),
])
def test_bad_dims_rejected(kw):
    assert decode_status(dims(**kw)) == gva.GVA_ERR_INVALID_ARG


def test_bad_split_counts_rejected():
    d = dims()
    assert decode_status(d, S=0) == gva.GVA_ERR_INVALID_ARG
    assert decode_status(d, S=gva.GVA_MAX_SPLITS + 1) == gva.GVA_ERR_INVALID_ARG
    assert decode_status(d, rows=-32) == gva.GVA_ERR_INVALID_ARG          # split_rows < 0
    assert decode_status(d, rows=48) == gva.GVA_ERR_INVALID_ARG           # not whole 32-row tiles
    lib = gva.lib()
    assert lib.gva_combine(ctypes.byref(d), A, A, 0, A, None, None) == gva.GVA_ERR_INVALID_ARG


def test_null_and_misaligned_pointers_rejected():
    d = dims()
    assert decode_status(d, v=None) == gva.GVA_ERR_INVALID_ARG
    assert decode_status(d, kr=None) == gva.GVA_ERR_INVALID_ARG
    assert decode_status(d, lens=None) == gva.GVA_ERR_INVALID_ARG
    assert decode_status(d, op=None) == gva.GVA_ERR_INVALID_ARG
    assert decode_status(d, v=A + 2) == gva.GVA_ERR_INVALID_ARG
    assert decode_status(d, op=A + 4) == gva.GVA_ERR_INVALID_ARG
    # exactly one way to pass the query: raw (q, m) or absorbed (q_abs, q_rot)
    assert decode_status(d, q=None, m=None) == gva.GVA_ERR_INVALID_ARG
    assert decode_status(d, q=A, m=None) == gva.GVA_ERR_INVALID_ARG
    assert decode_status(d, qa=A, qr=A) == gva.GVA_ERR_INVALID_ARG
    assert decode_status(d, q=None, m=None, qa=A, qr=None) == gva.GVA_ERR_INVALID_ARG
    # the current token's row comes whole: value and positional key together
    assert decode_status(d, vn=None, kn=A) == gva.GVA_ERR_INVALID_ARG
    assert decode_status(d, vn=A, kn=None) == gva.GVA_ERR_INVALID_ARG
    assert decode_status(d, vn=A + 4, kn=A) == gva.GVA_ERR_INVALID_ARG


def test_unsupported_shapes_reported():
    assert decode_status(dims(d_v=96)) == gva.GVA_ERR_UNSUPPORTED           # bf16 d_v
    assert decode_status(dims(d_c=48)) == gva.GVA_ERR_UNSUPPORTED           # d_c % 32
    assert decode_status(dims(d_r=12)) == gva.GVA_ERR_UNSUPPORTED           # d_r % 8
    assert decode_status(dims(n_heads=32, n_groups=2)) == gva.GVA_ERR_UNSUPPORTED  # H/G = 16
    assert decode_status(dims(dtype="f32", d_v=512)) == gva.GVA_ERR_UNSUPPORTED
    assert decode_status(dims(d_r=66)) == gva.GVA_ERR_UNSUPPORTED           # > 32 RoPE pairs
    assert decode_status(dims(t_max=40)) == gva.GVA_ERR_UNSUPPORTED         # tiled layout: T % 16
    assert decode_status(dims(dtype="f32", d_r=6)) == gva.GVA_ERR_UNSUPPORTED  # fp32 pieces of 4
    # the fused bf16 prologue needs a content slice to absorb
    assert decode_status(dims(d_c=0)) == gva.GVA_ERR_UNSUPPORTED


def test_append_validation():
    lib = gva.lib()
    d = dims()
    # n_rows == 0 is a no-op that succeeds without touching the device
    assert lib.gva_append_kv(ctypes.byref(d), A, A, A, A, A, A, 0, None) == gva.GVA_OK
    assert lib.gva_append_kv(ctypes.byref(d), A, A, A, A, A, A, -1, None) == gva.GVA_ERR_INVALID_ARG
    assert lib.gva_append_kv(ctypes.byref(d), None, A, A, A, A, A, 3, None) == gva.GVA_ERR_INVALID_ARG
    assert lib.gva_append_kv(ctypes.byref(d), A + 8, A, A, A, A, A, 3, None) == gva.GVA_ERR_INVALID_ARG
    assert lib.gva_append_kv(ctypes.byref(d), A, None, A, A, A, A, 3, None) == gva.GVA_ERR_INVALID_ARG
    d2 = dims(d_v=4)  # 8-byte bf16 rows cannot be copied in 16-byte pieces
    assert lib.gva_append_kv(ctypes.byref(d2), A, A, A, A, A, A, 3, None) == gva.GVA_ERR_UNSUPPORTED


def test_absorb_validation():
    lib = gva.lib()
    d = dims()
    assert lib.gva_absorb_query(ctypes.byref(d), None, A, A, A, A, None) == gva.GVA_ERR_INVALID_ARG
    assert lib.gva_absorb_query(ctypes.byref(d), A, A, A, A, None, None) == gva.GVA_ERR_INVALID_ARG
    assert lib.gva_absorb_query(None, A, A, A, A, A, None) == gva.GVA_ERR_INVALID_ARG


def test_pick_splits_is_host_only_and_bounded():
    d = dims(batch=32, n_heads=32, n_groups=8, t_max=8192)
    assert gva.gva_pick_splits(d, 8192, 0, 256) == (1, 0)       # 256 streams fill 256 CUs
    assert gva.gva_pick_splits(d, 100, 0, 256) == (1, 0)        # short sequences: no split
    d3 = dims(batch=4, n_heads=32, n_groups=8, t_max=131072, d_r=32)
    assert gva.gva_pick_splits(d3, 131072, 0, 256) == (8, 0)    # few long streams
    d4 = dims(batch=64, n_heads=16, n_groups=2, t_max=32768)
    even, _ = gva.gva_pick_splits(d4, 32768, 64 * 32768, 256, chunked=False)
    spread, _ = gva.gva_pick_splits(d4, 32768, 64 * 6000, 256, chunked=False)
    assert spread == 2 * even                                   # widely spread lengths
    for S in (even, spread):
        assert 1 <= S <= gva.GVA_MAX_SPLITS
    # fewer streams than CUs: split once a stream holds 192 KiB of value
    # rows, then one workgroup per CU, no split under 32 KiB, at most 16
    d350 = dims(batch=8, n_heads=16, n_groups=4, t_max=8192, d_v=64, d_c=64)
    assert gva.gva_pick_splits(d350, 2048, 0, 256) == (8, 0)    # 256 KiB streams: 32 x 8 workgroups
    assert gva.gva_pick_splits(d350, 1024, 0, 256) == (1, 0)    # 128 KiB streams: no split
    assert gva.gva_pick_splits(d350, 1536, 0, 256) == (6, 0)    # 192 KiB: six splits of 32 KiB
    d1 = dims(batch=1, n_heads=32, n_groups=8, t_max=8192)
    assert gva.gva_pick_splits(d1, 8192, 0, 256) == (16, 0)     # 32 would fill the CUs: capped
    d16 = dims(batch=16, n_heads=32, n_groups=8, t_max=4096)
    assert gva.gva_pick_splits(d16, 4096, 0, 256) == (2, 0)     # 128 streams: two each
    # widely spread lengths whose longest stream is below 192 KiB: no split
    # (bounded chunks or even), as for uniform lengths
    assert gva.gva_pick_splits(d350, 1024, 8 * 300, 256) == (1, 0)
    assert gva.gva_pick_splits(d350, 1024, 8 * 300, 256, chunked=False) == (1, 0)
    # few streams (32 on 256 CUs): even splits, one workgroup per CU, also
    # for spread lengths
    assert gva.gva_pick_splits(d350, 4096, 8 * 1200, 256) == (8, 0)
    # fused only while the B * G * S workgroups are all resident (two per CU)
    assert gva.gva_prefer_fused(d, 2, 0, 256) and not gva.gva_prefer_fused(d, 3, 0, 256)
    assert gva.gva_prefer_fused(d3, 16, 0, 256) and not gva.gva_prefer_fused(d3, 17, 0, 256)
    # bounded chunks pad the splits to a multiple of 8
    assert gva.gva_prefer_fused(d3, 16, 64, 256) and not gva.gva_prefer_fused(d3, 9, 64, 128)
    assert not gva.gva_prefer_fused(d3, 0, 0, 256) and not gva.gva_prefer_fused(d3, 2, -32, 256)
    # bounded chunks of at least (H/G) d_c rows stay fused past the resident grid
    rag = dims(batch=64, n_heads=16, n_groups=2, t_max=32768)    # 8 heads x d_c 128 = 1024 map rows
    assert gva.gva_prefer_fused(rag, 16, 1024, 256) and gva.gva_prefer_fused(rag, 16, 1696, 256)
    assert not gva.gva_prefer_fused(rag, 16, 992, 256) and not gva.gva_prefer_fused(rag, 16, 0, 256)


def test_pick_splits_bounded_chunks_for_ragged_lengths():
    d4 = dims(batch=64, n_heads=16, n_groups=2, t_max=32768)
    S, rows = gva.gva_pick_splits(d4, 32768, 64 * 6000, 256)
    assert rows > 0 and rows % 32 == 0
    assert S == -(-32768 // rows) and S <= gva.GVA_MAX_SPLITS  # every row of the longest covered
    # none under 128 KiB of value rows; the chunks with rows (at most one
    # partial chunk per stream) fit two resident workgroups per CU, with
    # the shortest chunk that does
    assert rows * 128 * 2 >= 128 << 10
    stream_rows, streams = 64 * 6000 * 2, 64 * 2
    assert -(-stream_rows // rows) + streams <= 2 * 256
    assert rows - 32 < -(-stream_rows // (2 * 256 - streams))
    # uniform lengths keep even splits
    assert gva.gva_pick_splits(d4, 32768, 64 * 32768, 256)[1] == 0
    # no chunk shorter than the (H/G) d_c = 1024 map rows its absorption reads
    S7, rows7 = gva.gva_pick_splits(d4, 8192, 64 * 1400, 256)
    assert rows7 == 1024 and S7 == 8
    # more streams than half the resident workgroups: chunks sized for about
    # two per CU over the whole batch (the partial chunks can no longer all fit)
    d6 = dims(batch=256, n_heads=16, n_groups=2, t_max=32768)
    S6, rows6 = gva.gva_pick_splits(d6, 32768, 256 * 4000, 256)
    assert rows6 > 0 and S6 == -(-32768 // rows6)
    assert rows6 - 32 < -(-(256 * 4000 * 2) // 256) <= rows6
    # a very long, very ragged batch stays within GVA_MAX_SPLITS
    d5 = dims(batch=256, n_heads=8, n_groups=8, t_max=1 << 20, d_v=64)
    S5, rows5 = gva.gva_pick_splits(d5, 1 << 20, 256 * 1000, 256)
    assert 1 <= S5 <= gva.GVA_MAX_SPLITS and S5 * rows5 >= 1 << 20


def test_tiled_layout_matches_header_formula():
    import torch
    for dtype, P in ((torch.bfloat16, 8), (torch.float32, 4)):
        T, D = 48, 24
        x = torch.arange(T * D, dtype=torch.float32).reshape(T, D).to(dtype)
        y = gva.tiled(x).reshape(-1)
        for t in range(T):
            for i in range(D):
                off = (t // 16) * 16 * D + ((i // P) * 16 + t % 16) * P + i % P
                assert y[off] == x[t, i]
        assert torch.equal(gva.untiled(gva.tiled(x)), x)
    z = torch.randn(2, 3, 32, 16).to(torch.bfloat16)
    assert torch.equal(gva.untiled(gva.tiled(z)), z)


def gqa_status(d, q=A, stride=None, k=A, v=A, lens=A, S=2, op=A, lp=A, rows=0):
    stride = d.d_v + 16 if stride is None else stride
    return gva.lib().gva_gqa_decode_attention(ctypes.byref(d), q, stride, k, v, lens, S, rows, op, lp,
                                              None)


def test_gqa_validation():
    d = dims(n_heads=16, n_groups=2)
    assert gqa_status(dims(batch=0)) == gva.GVA_ERR_INVALID_ARG
    for kw in (dict(q=None), dict(k=None), dict(v=None), dict(lens=None), dict(op=None),
               dict(lp=None), dict(k=A + 2), dict(op=A + 4), dict(S=0),
               dict(S=gva.GVA_MAX_SPLITS + 1), dict(stride=64), dict(rows=-32), dict(rows=40)):
        assert gqa_status(d, **kw) == gva.GVA_ERR_INVALID_ARG, kw
    assert gqa_status(dims(dtype="f32")) == gva.GVA_ERR_UNSUPPORTED          # bf16 only
    assert gqa_status(dims(d_v=96), stride=96) == gva.GVA_ERR_UNSUPPORTED
    assert gqa_status(dims(n_heads=32, n_groups=2)) == gva.GVA_ERR_UNSUPPORTED   # H/G = 16
    assert gqa_status(d, stride=132) == gva.GVA_ERR_UNSUPPORTED             # 16-byte query rows
    assert gqa_status(dims(t_max=40)) == gva.GVA_ERR_UNSUPPORTED


def rope_status(d, q=A, m=A, v=A, lens=A, S=2, rows=0, op=A, lp=A):
    return gva.lib().gva_rope_decode_attention(ctypes.byref(d), q, m, v, lens, S, rows, op, lp, None)


def test_rope_decode_validation():
    d = dims(n_heads=8, n_groups=2, d_r=0)
    assert rope_status(dims(batch=0, d_r=0)) == gva.GVA_ERR_INVALID_ARG
    assert rope_status(dims(d_r=16)) == gva.GVA_ERR_INVALID_ARG              # no decoupled slice
    assert rope_status(dims(d_r=0, rope_base=0.0)) == gva.GVA_ERR_INVALID_ARG
    assert rope_status(dims(d_r=0, d_c=63)) == gva.GVA_ERR_INVALID_ARG       # whole pairs
    for kw in (dict(q=None), dict(m=None), dict(v=None), dict(lens=None), dict(op=None),
               dict(lp=None), dict(q=A + 2), dict(m=A + 8), dict(v=A + 4), dict(lens=A + 2),
               dict(S=0), dict(S=gva.GVA_MAX_SPLITS + 1), dict(rows=-32), dict(rows=40)):
        assert rope_status(d, **kw) == gva.GVA_ERR_INVALID_ARG, kw
    assert rope_status(dims(d_r=0, dtype="f32")) == gva.GVA_ERR_UNSUPPORTED   # bf16 only
    assert rope_status(dims(d_r=0, d_v=96)) == gva.GVA_ERR_UNSUPPORTED
    assert rope_status(dims(d_r=0, d_c=96)) == gva.GVA_ERR_UNSUPPORTED
    assert rope_status(dims(d_r=0, n_heads=32, n_groups=2)) == gva.GVA_ERR_UNSUPPORTED   # H/G = 16
    # W of 8 heads at d_v = d_c = 128 is 256 KiB: over the LDS budget
    assert rope_status(dims(d_r=0, n_heads=16, n_groups=2)) == gva.GVA_ERR_UNSUPPORTED
    assert rope_status(dims(d_r=0, t_max=40)) == gva.GVA_ERR_UNSUPPORTED


def prefill_status(d, N=4, qa=A, qr=A, v=A, kr=A, lens=A, o=A, lse=A):
    return gva.lib().gva_prefill_attention(ctypes.byref(d), N, qa, qr, v, kr, lens, o, lse, None)


def test_prefill_validation():
    d = dims(t_max=64)
    assert prefill_status(dims(batch=0)) == gva.GVA_ERR_INVALID_ARG
    for kw in (dict(N=0), dict(N=65), dict(qa=None), dict(qr=None), dict(v=None), dict(kr=None),
               dict(lens=None), dict(o=None), dict(lse=None), dict(qa=A + 4), dict(qr=A + 8),
               dict(v=A + 2), dict(kr=A + 8), dict(o=A + 4), dict(lens=A + 2)):
        assert prefill_status(d, **kw) == gva.GVA_ERR_INVALID_ARG, kw
    # d_r = 0: no positional operands needed
    assert prefill_status(dims(d_r=0, t_max=64, n_heads=32, n_groups=2), qr=None, kr=None) == \
        gva.GVA_ERR_UNSUPPORTED                                        # H/G = 16
    assert prefill_status(dims(t_max=64, dtype="f32")) == gva.GVA_ERR_UNSUPPORTED
    assert prefill_status(dims(t_max=64, d_v=96)) == gva.GVA_ERR_UNSUPPORTED
    assert prefill_status(dims(t_max=64, d_r=12)) == gva.GVA_ERR_UNSUPPORTED
    assert prefill_status(dims(t_max=40)) == gva.GVA_ERR_UNSUPPORTED
    lib = gva.lib()
    # the GQA baseline needs its key stream; the absorb needs 1 <= n_new <= T
    assert lib.gva_gqa_prefill_attention(ctypes.byref(d), 4, A, None, A, A, A, A, None) == \
        gva.GVA_ERR_INVALID_ARG
    assert lib.gva_gqa_prefill_attention(ctypes.byref(d), 4, A + 4, A, A, A, A, A, None) == \
        gva.GVA_ERR_INVALID_ARG
    assert lib.gva_prefill_absorb(ctypes.byref(d), 0, A, A, A, A, A, None) == gva.GVA_ERR_INVALID_ARG
    assert lib.gva_prefill_absorb(ctypes.byref(d), 65, A, A, A, A, A, None) == gva.GVA_ERR_INVALID_ARG
    assert lib.gva_prefill_absorb(ctypes.byref(d), 4, A, A, A, A, None, None) == gva.GVA_ERR_INVALID_ARG
    big = dims(batch=64, t_max=1 << 15)
    assert lib.gva_prefill_absorb(ctypes.byref(big), 1 << 15, A, A, A, A, A, None) == \
        gva.GVA_ERR_UNSUPPORTED                                        # 2^21 query rows


def test_probe_validation():
    lib = gva.lib()
    assert lib.gva_probe_read(None, 1 << 20, 8, A, None) == gva.GVA_ERR_INVALID_ARG
    assert lib.gva_probe_read(A, 8, 8, A, None) == gva.GVA_ERR_INVALID_ARG    # under one 16-byte piece
    assert lib.gva_probe_read(A, 1 << 20, 0, A, None) == gva.GVA_ERR_INVALID_ARG
    assert lib.gva_probe_read(A + 4, 1 << 20, 8, A, None) == gva.GVA_ERR_INVALID_ARG


def paged_status(d, pg, v=A, kr=A, bt=A, lens=A, S=2, rows=0, op=A, lp=A):
    return gva.lib().gva_paged_decode_attention(ctypes.byref(d), ctypes.byref(pg) if pg is not None else None,
                                                A, A, None, None, v, kr, bt, lens, None, None, S, rows, op,
                                                lp, None)


def test_paged_validation():
    d = dims(t_max=256)
    ok = gva.GvaPaging(64, 4, 10)
    for pg in (gva.GvaPaging(48, 4, 10),        # not whole 32-row tiles
               gva.GvaPaging(0, 4, 10), gva.GvaPaging(64, 0, 10), gva.GvaPaging(64, 4, 0),
               gva.GvaPaging(64, 3, 10)):       # capacity != t_max
        assert paged_status(d, pg) == gva.GVA_ERR_INVALID_ARG, (pg.page_rows, pg.max_pages, pg.n_pages)
    assert paged_status(d, None) == gva.GVA_ERR_INVALID_ARG
    assert paged_status(d, ok, bt=None) == gva.GVA_ERR_INVALID_ARG
    assert paged_status(d, ok, bt=A + 2) == gva.GVA_ERR_INVALID_ARG
    assert paged_status(d, ok, v=A + 2) == gva.GVA_ERR_INVALID_ARG
    assert paged_status(dims(t_max=256, dtype="f32"), ok) == gva.GVA_ERR_UNSUPPORTED
    big = dims(t_max=32 * (gva.GVA_MAX_PAGES + 1))
    assert paged_status(big, gva.GvaPaging(32, gva.GVA_MAX_PAGES + 1, 10)) == gva.GVA_ERR_UNSUPPORTED
    lib = gva.lib()
    assert lib.gva_paged_append_kv(ctypes.byref(d), ctypes.byref(ok), A, A, A, A, A, A, A, 0, None) == gva.GVA_OK
    assert lib.gva_paged_append_kv(ctypes.byref(d), ctypes.byref(gva.GvaPaging(64, 3, 10)), A, A, A, A, A, A,
                                   A, 2, None) == gva.GVA_ERR_INVALID_ARG
    assert lib.gva_paged_append_kv(ctypes.byref(d), ctypes.byref(ok), A, A, None, A, A, A, A, 2,
                                   None) == gva.GVA_ERR_INVALID_ARG


def test_page_plumbing_round_trip():
    import torch
    d = gva.make_dims(3, 8, 2, 64, 64, 16, 256, "bf16")
    pg = gva.make_paging(d, 64, 14)
    bt = torch.randperm(14, generator=torch.Generator().manual_seed(1))[:12].reshape(3, 4).to(torch.int32)
    v = torch.randn(3, 2, 256, 64).to(torch.bfloat16)
    kr = torch.randn(3, 256, 16).to(torch.bfloat16)
    vp, kp = gva.to_pages(gva.tiled(v), gva.tiled(kr), bt, pg)
    v2, k2 = gva.from_pages(vp, kp, bt, pg)
    assert torch.equal(gva.untiled(v2), v) and torch.equal(gva.untiled(k2), kr)
    # a page block is the tiled layout of that page's rows
    page = int(bt[1, 2])
    assert torch.equal(gva.untiled(vp[page]), v[1, :, 128:192])


def _ws_round(n):
    return (n + 255) // 256 * 256


def test_decode_workspace_size():
    # one split with the absorption fused: no workspace at all
    big = dims(batch=32, n_heads=32, n_groups=8, t_max=8192)
    assert gva.gva_decode_workspace_size(big, 1) == 0
    # several splits, absorption still fused (B G S <= 2 per CU on 256 CUs)
    S = 2
    assert gva.gva_prefer_fused(big, S, 0, 256)
    rows = 32 * 32
    assert gva.gva_decode_workspace_size(big, S) == _ws_round(rows * S * 128 * 4) + _ws_round(rows * S * 4)
    # ragged batch, bounded chunks shorter than a group's map rows (8 heads
    # x d_c = 1024): separate absorption (q~ and the rotated positional
    # query) plus the partials
    rag = dims(batch=64, n_heads=16, n_groups=2, t_max=32768)
    S, c = 16, 992
    assert not gva.gva_prefer_fused(rag, S, c, 256)
    rows = 64 * 16
    expect = (_ws_round(rows * 128 * 4) + _ws_round(rows * 16 * 4) + _ws_round(rows * S * 128 * 4)
              + _ws_round(rows * S * 4))
    assert gva.gva_decode_workspace_size(rag, S, c) == expect
    lib = gva.lib()
    n = ctypes.c_size_t(7)
    assert lib.gva_decode_workspace_size(ctypes.byref(rag), 0, 0, ctypes.byref(n)) == gva.GVA_ERR_INVALID_ARG
    assert lib.gva_decode_workspace_size(ctypes.byref(rag), 2, -32, ctypes.byref(n)) == gva.GVA_ERR_INVALID_ARG
    assert lib.gva_decode_workspace_size(ctypes.byref(rag), 2, 0, None) == gva.GVA_ERR_INVALID_ARG
    assert n.value == 7


def step_status(d, S=4, rows=0, q=A, m=A, ws=A, nbytes=1 << 30, o=A, lse=A, vn=None, kn=None):
    return gva.lib().gva_decode_step(ctypes.byref(d), q, m, A, A, A, vn, kn, S, rows, ws, nbytes, o, lse, None)


def test_decode_step_validation():
    rag = dims(batch=64, n_heads=16, n_groups=2, t_max=32768)
    need = gva.gva_decode_workspace_size(rag, 16, 1696)
    ok = dict(S=16, rows=1696)
    assert step_status(rag, ws=None, **ok) == gva.GVA_ERR_INVALID_ARG              # workspace needed
    assert step_status(rag, nbytes=need - 1, **ok) == gva.GVA_ERR_INVALID_ARG      # too short
    assert step_status(rag, ws=A + 128, **ok) == gva.GVA_ERR_INVALID_ARG           # not 256-byte aligned
    assert step_status(rag, q=None, **ok) == gva.GVA_ERR_INVALID_ARG               # raw query required
    assert step_status(rag, o=None, **ok) == gva.GVA_ERR_INVALID_ARG
    assert step_status(rag, lse=None, **ok) == gva.GVA_ERR_INVALID_ARG
    assert step_status(rag, S=0) == gva.GVA_ERR_INVALID_ARG
    assert step_status(rag, S=2, rows=48) == gva.GVA_ERR_INVALID_ARG                # not whole tiles
    assert step_status(rag, vn=None, kn=A, **ok) == gva.GVA_ERR_INVALID_ARG
    assert step_status(dims(d_v=96), S=1, ws=None) == gva.GVA_ERR_UNSUPPORTED
    assert step_status(dims(d_c=0), S=1, ws=None) == gva.GVA_ERR_UNSUPPORTED       # fused, nothing to absorb


def test_decode_step_static_validation():
    # checked on the host before any runtime call: a plan past the static
    # scratch buffer is refused with its own status
    lib = gva.lib()
    assert "static scratch" in gva.status_string(gva.GVA_ERR_SCRATCH)

    def st(d, S=4, rows=0, q=A, o=A, lse=A):
        return lib.gva_decode_step_static(ctypes.byref(d), q, A, A, A, A, None, None, S, rows, o, lse, None)

    huge = dims(batch=64, n_heads=64, n_groups=8, t_max=65536)
    assert gva.gva_decode_workspace_size(huge, 256) > gva.GVA_STATIC_SCRATCH_BYTES
    assert st(huge, S=256) == gva.GVA_ERR_SCRATCH
    rag = dims(batch=64, n_heads=16, n_groups=2, t_max=32768)
    assert 0 < gva.gva_decode_workspace_size(rag, 16, 1696) <= gva.GVA_STATIC_SCRATCH_BYTES
    assert st(rag, S=16, rows=1696, q=None) == gva.GVA_ERR_INVALID_ARG
    assert st(rag, S=16, rows=1696, lse=None) == gva.GVA_ERR_INVALID_ARG
    assert st(rag, S=0) == gva.GVA_ERR_INVALID_ARG
    assert st(dims(d_v=96), S=1) == gva.GVA_ERR_UNSUPPORTED
