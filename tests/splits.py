"""The ABI's split rule as test plumbing: the row range of every split of
every sequence, as gva_decode_attention defines it (include/gva.h), for
the tests that check each split's partial against the oracle run on that
split's rows.  Not part of the oracle: the paper has no splits; the rule is
the library's interface, restated here from its header."""

from __future__ import annotations

import torch


def split_bounds(lens: torch.Tensor, num_splits: int, tile: int = 32, split_rows: int = 0):
    """Row ranges [begin, end) of every split, per sequence: [S][B] each.

    The first n splits of a sequence with L rows share them evenly: split s
    covers [s*c, min(L, (s+1)*c)) with c = tile * ceil(ceil(L / n) / tile),
    and splits from n on are empty.  n = S for even splits (split_rows = 0);
    with split_rows > 0 (bounded chunks) n = ceil(L / split_rows), clamped
    to [1, S].
    """
    L = lens.to(torch.int64).clamp(min=0)
    if split_rows > 0:
        n = ((L + split_rows - 1) // split_rows).clamp(min=1, max=num_splits)
    else:
        n = torch.full_like(L, num_splits)
    per = (L + n - 1) // n
    chunk = ((per + tile - 1) // tile) * tile
    begins, ends = [], []
    for s in range(num_splits):
        begins.append(torch.minimum(chunk * s, L).to(torch.int32))
        ends.append(torch.minimum(chunk * (s + 1), L).to(torch.int32))
    return begins, ends
