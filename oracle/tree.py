"""Brute-force cached-prefix lengths (TEST INFRASTRUCTURE: only the tests, the smoke
check and the benchmark's CPU baseline use this package).

With no capacity limit a chunked prefix tree holds every full chunk of every
request inserted so far, each under its exact predecessor chunks (Sec. 4.2). A new
request therefore reuses exactly the longest run of leading whole chunks that it
shares with some earlier request. This computes that run directly, by comparing
the request with every earlier one, without building a tree.
"""
from __future__ import annotations

from typing import Sequence

import numpy as np


def shared_leading_chunks(a: Sequence[int], b: Sequence[int], chunk: int) -> int:
    """Number of leading whole chunks on which two token sequences agree."""
    a = np.asarray(a)
    b = np.asarray(b)
    n = 0
    while (n + 1) * chunk <= len(a) and (n + 1) * chunk <= len(b):
        if not np.array_equal(a[n * chunk:(n + 1) * chunk], b[n * chunk:(n + 1) * chunk]):
            break
        n += 1
    return n


def cached_prefix_tokens(request: Sequence[int], earlier: Sequence[Sequence[int]], chunk: int,
                         block: int) -> int:
    """Tokens of `request` whose KV an unbounded chunk tree filled with `earlier`
    holds, cut to a block boundary and leaving at least one token to compute."""
    best = max((shared_leading_chunks(request, e, chunk) for e in earlier), default=0)
    hit = best * chunk
    if hit >= len(request):
        hit = (len(request) - 1) // block * block
    return hit - hit % block
