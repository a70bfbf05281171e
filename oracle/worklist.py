"""Reference definition of the work list (test infrastructure).

The (head, token) pairs are laid out head-major in one index space of length
H*T and cut into ranges of C tokens; every (user, head) pair with tokens is cut
at the range boundaries into segments, listed in (head, user, range) order.
Item = (b, h, t0, t1, range, split, pair_first, 0), see sa_build_worklist.
Plain Python; shares nothing with the library.
"""
from typing import List, Sequence, Tuple


def worklist(offsets: Sequence[int], T: int, H: int, C: int) -> List[Tuple[int, ...]]:
    B = len(offsets) - 1
    items = []
    for h in range(H):
        for b in range(B):
            lo, hi = int(offsets[b]), int(offsets[b + 1])
            if hi <= lo:
                continue
            first = len(items)
            g_lo, g_hi = h * T + lo, h * T + hi          # half-open range in the flat space
            segs = []
            g = g_lo
            while g < g_hi:
                r = g // C
                end = min(g_hi, (r + 1) * C)
                segs.append((r, g - h * T, end - h * T))
                g = end
            split = 1 if len(segs) > 1 else 0
            for r, t0, t1 in segs:
                items.append((b, h, t0, t1, r, split, first, 0))
    return items


def coverage_ok(items, offsets, H) -> bool:
    """Every token of every user, for every head, appears in exactly one item."""
    B = len(offsets) - 1
    seen = {}
    for (b, h, t0, t1, r, split, first, _) in items:
        for t in range(t0, t1):
            key = (h, t)
            if key in seen:
                return False
            seen[key] = b
    for h in range(H):
        for b in range(B):
            for t in range(int(offsets[b]), int(offsets[b + 1])):
                if seen.get((h, t)) != b:
                    return False
    return True
