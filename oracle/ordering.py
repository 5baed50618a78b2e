"""Reference for the ordering objective that shapes each request's cached depth.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper Sec. 3.3, Eq. 1: for an order O of the retrieved set D and a tree T of
recently served orders, l(O, T) is the length of the longest leading run of O
that follows a cached root-to-node path; the best order maximises it over all
permutations, and documents after the reused run keep their retrieval rank.
With recency as the residency estimate (Sec. 3.4), a node is cached when it lies
on one of the orders served within the recent window, so the cached
root-to-node paths are exactly the prefixes of those orders.
"""
from __future__ import annotations

import itertools


def reusable_prefix_depth(order, cached_orders) -> int:
    """l(O, T) with T given as the list of cached served orders."""
    best = 0
    for p in cached_orders:
        n = 0
        while n < len(p) and n < len(order) and p[n] == order[n]:
            n += 1
        best = max(best, n)
    return best


def exhaustive_best_depth(docs, cached_orders) -> int:
    """max over all permutations O of D of l(O, T) (the k! search)."""
    return max(reusable_prefix_depth(o, cached_orders) for o in itertools.permutations(docs))


def canonical_best_order(docs, cached_orders):
    """One argmax of Eq. 1 whose tail keeps retrieval rank: among permutations
    reaching the best depth, the reused run that comes first when runs are
    compared by the retrieval ranks of their documents, then the rest in rank
    order."""
    best = exhaustive_best_depth(docs, cached_orders)
    rank = {d: i for i, d in enumerate(docs)}
    runs = set()
    for p in cached_orders:
        if len(p) >= best and set(p[:best]) <= set(docs):
            runs.add(tuple(p[:best]))
    run = min(runs, key=lambda r: [rank[d] for d in r]) if best else ()
    rest = [d for d in docs if d not in run]
    return list(run) + rest, best
