"""Oracle: coverage metrics of a prefetch decision.

Test infrastructure only.

Paper passages followed: Sec. IV-B, full coverage K_r subset of K_p^(delta) (Eq. 2)
and the oracle budget delta* = min{delta : K_r \\ K_p^(delta) empty} (Eq. 3); Sec. V-C,
overlap accuracy between the prefetched and the routed experts, read as the fraction
of routed experts that were prefetched, |K_r intersect K_p| / k.
"""
from __future__ import annotations


def delta_star(ranked, K_r, k):
    """Eq. 3 by enumeration: the smallest delta whose ranked prefix holds all of K_r."""
    need = set(int(e) for e in K_r if e >= 0)
    N = len(ranked)
    for delta in range(N - k + 1):
        if need <= set(int(e) for e in ranked[:k + delta]):
            return delta
    raise ValueError("routed set not contained in the ranked list")


def overlap(K_r, K_p, k):
    r = set(int(e) for e in K_r if e >= 0)
    p = set(int(e) for e in K_p if e >= 0)
    return len(r & p) / k


def full_coverage(K_r, K_p):
    r = set(int(e) for e in K_r if e >= 0)
    p = set(int(e) for e in K_p if e >= 0)
    return r <= p
