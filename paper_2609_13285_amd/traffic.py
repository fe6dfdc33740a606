"""Cache-size and traffic accounting for the GVA decode step (host logic).

Cache counts follow Section 3.4 (eq. ngva): GVA keeps G value streams of
width d_h plus one shared positional key of width d_r per token, against
2*G*d_h for matched GQA; the ratio is 1/2 + d_r / (2 G d_h).

The algorithmic bytes of one decode launch are the bytes the method must
move at least once: every cached row of the value streams and of the shared
positional key up to each sequence's length, the maps M_h, the queries, and
the fp32 outputs.  Split partials and any re-read are implementation
overhead and are not counted.
"""

from __future__ import annotations

from typing import Iterable, Union

IntSeq = Union[Iterable[int], "torch.Tensor"]  # noqa: F821


def cache_scalars_gva(T: int, G: int, d_h: int, d_r: int) -> int:
    """Persistent scalars per layer and sequence, decoupled-RoPE GVA."""
    return T * G * d_h + T * d_r


def cache_scalars_gqa(T: int, G: int, d_h: int) -> int:
    """Persistent scalars per layer and sequence, grouped-query attention."""
    return 2 * T * G * d_h


def cache_ratio(G: int, d_h: int, d_r: int) -> float:
    """N_GVA / N_GQA = 1/2 + d_r / (2 G d_h)."""
    return 0.5 + d_r / (2.0 * G * d_h)


def _total_len(lens: IntSeq) -> int:
    try:
        return int(lens.to("cpu").long().clamp(min=0).sum())  # torch tensor
    except AttributeError:
        return int(sum(max(int(x), 0) for x in lens))


def stream_bytes(lens: IntSeq, G: int, d_v: int, d_r: int, elem: int) -> int:
    """Bytes of the value and positional-key streams over all cached rows."""
    return _total_len(lens) * (G * d_v + d_r) * elem


def decode_bytes(lens: IntSeq, B: int, H: int, G: int, d_v: int, d_c: int, d_r: int,
                 elem: int) -> int:
    """Algorithmic bytes of one fused absorb+attention launch.

    Streams + the maps M (H*d_v*d_c) + the queries (B*H*(d_c+d_r)).  The
    split outputs are overhead, so they are not counted here.
    """
    return (stream_bytes(lens, G, d_v, d_r, elem) + H * d_v * d_c * elem
            + B * H * (d_c + d_r) * elem)


def step_bytes(lens: IntSeq, B: int, H: int, G: int, d_v: int, d_c: int, d_r: int,
               elem: int, appended_rows: int) -> int:
    """Algorithmic bytes of one decode step: append + attention + fp32 output.

    The append reads and writes each new row once (value rows of all groups
    plus the positional key).
    """
    append = 2 * appended_rows * (G * d_v + d_r) * elem
    return decode_bytes(lens, B, H, G, d_v, d_c, d_r, elem) + append + B * H * d_v * 4


def launch_bytes(lens: IntSeq, B: int, H: int, G: int, d_v: int, d_c: int, d_r: int, elem: int,
                 appended_rows: int = 0, writes_output: bool = False) -> int:
    """Algorithmic bytes of one attention launch: the streams, M and q
    (decode_bytes), plus the current token's rows when the launch appends
    them (read once from the new rows, written once into the caches), plus
    the fp32 output when the launch writes it (one split: its partial is
    the output; with several, the combine writes it)."""
    append = 2 * appended_rows * (G * d_v + d_r) * elem
    out = B * H * d_v * 4 if writes_output else 0
    return decode_bytes(lens, B, H, G, d_v, d_c, d_r, elem) + append + out


def gqa_decode_bytes(lens: IntSeq, B: int, H: int, G: int, d_v: int, elem: int) -> int:
    """Algorithmic bytes of one matched-GQA decode launch (K and V streams)."""
    return _total_len(lens) * 2 * G * d_v * elem + B * H * d_v * elem


def rope_decode_flops(total_rows: int, H: int, d_v: int, d_c: int) -> int:
    """Algorithmic flops of one decode launch of GVA with ordinary RoPE
    (Section 3.2: the key map is not absorbable), over ``total_rows`` cached
    rows summed across the batch.  Per row and head: the key reconstruction
    v_t M_h (2 d_v d_c), the rotated score (2 d_c) and the weighted value
    sum (2 d_v).  Absorbed GVA needs only 2 d_v + 2 d_v per row and head."""
    return int(total_rows) * H * 2 * (d_v * d_c + d_c + d_v)


def prefill_flops(n_new: int, total_len: int, H: int, d_v: int, d_r: int) -> int:
    """Algorithmic flops of one causal prefill launch (absorbed form) for a
    sequence of ``total_len`` cached rows whose last ``n_new`` are the
    prompt: query p sees p+1 rows; per row and head the score costs
    2 (d_v + d_r) and the weighted value sum 2 d_v.  With d_r = 0 this is
    also the matched-GQA count (key width d_v)."""
    first = total_len - n_new
    seen = sum(max(0, first + i + 1) for i in range(n_new))
    return seen * H * 2 * (2 * d_v + d_r)
