"""Reference for evidence ordering: the objective that shapes each request's
cached depth, the greedy walk, the baseline orders, and residency feedback.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper Sec. 3.3, Eq. 1: for an order O of the retrieved set D and a tree T of
recently served orders, l(O, T) is the length of the longest leading run of O
that follows a cached root-to-node path; the best order maximises it over all
permutations, and documents after the reused run keep their retrieval rank.
Sec. 3.4: recency stands in for residency, so a node is cached when an order
served within the recent window passes through it; the feedback option marks
a path stale when the engine shows it was not resident.

The tree is modelled here by its definition, not as a trie: the list of served
orders with their service times, plus the stale marks. A root-to-node path p
(a tuple of documents) exists when some served order starts with p; it is
cached when the latest such order was served within the last `window`
insertions and p was not marked stale at or after that time.
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


class TreeModel:
    """The knowledge tree of Sec. 3.2 held as its served orders (see above)."""

    def __init__(self, window: int):
        self.window = int(window)
        self.clock = 0
        self.served = []        # (time, order tuple), in service order
        self.stale = {}         # path tuple -> time of the latest stale mark

    def insert(self, order) -> None:
        """Record an order after its request was served (time = new clock)."""
        self.clock += 1
        self.served.append((self.clock, tuple(order)))

    def last_served(self, path):
        """Latest service time of an order starting with `path`, or None."""
        path = tuple(path)
        t = None
        for when, o in self.served:
            if o[:len(path)] == path and len(o) >= len(path):
                t = when
        return t

    def is_cached(self, path) -> bool:
        t = self.last_served(path)
        if t is None or t <= self.clock - self.window:
            return False
        mark = self.stale.get(tuple(path))
        return mark is None or mark < t

    def mark_stale(self, order, observed_depth: int) -> None:
        """Feedback (Sec. 3.4): the engine reused only `observed_depth`
        documents of `order`, so every deeper node of it is stale from now."""
        order = tuple(order)
        for j in range(observed_depth + 1, len(order) + 1):
            if self.last_served(order[:j]) is None:
                break
            self.stale[order[:j]] = self.clock

    def doc_last_served(self, d):
        """Latest service time of document d within the window, or None."""
        t = None
        for when, o in self.served:
            if d in o:
                t = when
        return t if t is not None and t > self.clock - self.window else None


def walk_depth(order, is_cached) -> int:
    """l(O, T): how many leading documents of O follow cached nodes, each node
    of the run cached (the walk from the root stops at the first that is not)."""
    n = 0
    while n < len(order) and is_cached(tuple(order[:n + 1])):
        n += 1
    return n


def greedy_order(docs, is_cached):
    """The greedy order of Sec. 3.3 (Algorithm 1), stated by what it selects:
    the reused run r_1, r_2, ... is built one level at a time, r_j being the
    document of lowest retrieval rank among those not yet placed whose node
    below (r_1 .. r_{j-1}) is cached; the run ends at the first level with no
    such document, and the unplaced documents follow in retrieval rank.

    Returns (order, depth, probes). probes is the number of child lookups a
    scan in retrieval rank makes to find those choices: at a level that places
    document d, one per unplaced document of rank up to d's; at the level that
    finds nothing (when documents remain), one per unplaced document."""
    rank = {d: i for i, d in enumerate(docs)}
    run = ()
    probes = 0
    while True:
        unplaced = [d for d in docs if d not in run]
        candidates = [d for d in unplaced if is_cached(run + (d,))]
        if not candidates:
            probes += len(unplaced)
            break
        pick = min(candidates, key=rank.__getitem__)
        probes += sum(1 for d in unplaced if rank[d] <= rank[pick])
        run = run + (pick,)
    return list(run) + [d for d in docs if d not in run], len(run), probes


def exhaustive_order(docs, is_cached):
    """Eq. 1 by enumerating all k! permutations: the deepest reusable run;
    among equally deep runs, the one whose documents' retrieval ranks come
    first lexicographically; the rest in retrieval rank. Returns (order, depth)."""
    rank = {d: i for i, d in enumerate(docs)}
    best_depth, best_run = 0, ()
    for o in itertools.permutations(docs):
        n = walk_depth(o, is_cached)
        run = tuple(o[:n])
        if n > best_depth or (n == best_depth and [rank[d] for d in run] < [rank[d] for d in best_run]):
            best_depth, best_run = n, run
    return list(best_run) + [d for d in docs if d not in best_run], best_depth


def retrieval_order(docs):
    """The retriever's rank order, unchanged (the APC+Retrieval baseline)."""
    return list(docs)


def sorted_order(docs):
    """Lexicographic sorting of document IDs (the APC+Sorted baseline, Sec. 4
    strategies). Documents carry fixed-width IDs, so this is ascending ID."""
    return sorted(docs)


def recency_order(docs, tree: TreeModel):
    """The recency heuristic of Table `baselines`: documents served within the
    window first, most recently served first (ties in retrieval rank), then
    the others in retrieval rank."""
    rank = {d: i for i, d in enumerate(docs)}
    seen = [(tree.doc_last_served(d), d) for d in docs]
    recent = sorted([x for x in seen if x[0] is not None], key=lambda x: (-x[0], rank[x[1]]))
    return [d for _, d in recent] + [d for t, d in seen if t is None]
