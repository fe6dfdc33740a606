"""The ABI's split rule as test plumbing: the row range of every split of
every sequence, as gva_decode_attention defines it (include/gva.h), for
the tests that check each split's partial against the oracle run on that
split's rows.  Not part of the oracle: the paper has no splits; the rule is
the library's interface, restated here from its header."""

from __future__ import annotations

import torch


def split_bounds(lens: torch.Tensor, num_splits: int, tile: int = 32, split_rows: int = 0):
    """Row ranges [begin, end) of every split, per sequence: [S][B] each.

    Split s of a sequence with L rows covers [s*c, min(L, (s+1)*c)), except
    that the last split ends at L.  c = split_rows when it is positive,
    else c = tile * ceil(ceil(L / S) / tile).  Trailing splits may be empty.
    """
    L = lens.to(torch.int64).clamp(min=0)
    if split_rows > 0:
        chunk = torch.full_like(L, int(split_rows))
    else:
        per = (L + num_splits - 1) // num_splits
        chunk = ((per + tile - 1) // tile) * tile
    begins, ends = [], []
    for s in range(num_splits):
        b = torch.minimum(chunk * s, L)
        e = L if s == num_splits - 1 else torch.minimum(chunk * (s + 1), L)
        begins.append(b.to(torch.int32))
        ends.append(e.to(torch.int32))
    return begins, ends
