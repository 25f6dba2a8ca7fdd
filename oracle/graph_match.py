"""TEST INFRASTRUCTURE ONLY -- oracle of the topology-aware subgraph matching
(Section 4.2, Algorithm "Topology-Aware Subgraph Matching").

Graphs are DAGs of operators: nodes 0..n-1, edges (tensors) u -> v; node 0
is the single source (the graph input) and node n-1 the single sink (its
output); every node lies on a path from the source to the sink.  Eq holds
pairs (a, b): the output tensor of node a of graph 1 is equivalent to the
output of node b of graph 2.

Readings of the printed algorithm (its loop bound and recursive call are
garbled in the extracted text):
  * d dominates v when every path from the source to v passes through d;
    the dominator path is the chain of the sink's dominators, source first;
  * the cut points are the pairs of Eq on the two dominator paths, plus the
    two sources and the two sinks (equivalent by hypothesis), reduced to a
    longest chain rising in both paths (ties: the lexicographically smallest
    chain of path positions);
  * the region between consecutive cuts c and c' is every node c dominates
    minus the nodes c' strictly dominates (so c and c' belong to it), and the
    regions of the two graphs at the same step are matched;
  * a pair with no interior cut is a finest match; otherwise every pair of
    regions is matched again, recursively, with Eq restricted to it.
The result lists the finest matched pairs as ((entry1, exit1), (entry2,
exit2)), in path order.  Dominators are found from their definition: d
dominates v exactly when v cannot be reached from the source once d is
removed.
"""
from __future__ import annotations


def _reach(n, succ, src, removed, allowed):
    seen = {src}
    stack = [src]
    while stack:
        u = stack.pop()
        for v in succ[u]:
            if v in allowed and v != removed and v not in seen:
                seen.add(v)
                stack.append(v)
    return seen


def dominators(nodes, succ, source):
    """dom[v] = the set of nodes dominating v (v included), within `nodes`."""
    allowed = set(nodes)
    full = _reach(None, succ, source, None, allowed)
    dom = {v: {v, source} for v in nodes}
    for d in nodes:
        if d == source:
            continue
        reach = _reach(None, succ, source, d, allowed)
        for v in full:
            if v != d and v not in reach:
                dom[v].add(d)
    return dom


def dominator_path(nodes, succ, source, sink):
    dom = dominators(nodes, succ, source)
    return sorted(dom[sink], key=lambda d: len(dom[d])), dom


def _chain(p1, p2, eq):
    """Longest chain of pairs rising in both paths (source and sink pairs kept)."""
    i1 = {v: i for i, v in enumerate(p1)}
    i2 = {v: i for i, v in enumerate(p2)}
    pts = sorted({(i1[a], i2[b]) for a, b in eq if a in i1 and b in i2} |
                 {(0, 0), (len(p1) - 1, len(p2) - 1)})
    best = {}  # best chain ending at each point, compared by (length, -lexicographic)
    for k, (x, y) in enumerate(pts):
        cand = [(x, y)]
        for (px, py) in pts[:k]:
            if px < x and py < y:
                c = best[(px, py)] + [(x, y)]
                if len(c) > len(cand) or (len(c) == len(cand) and c < cand):
                    cand = c
        best[(x, y)] = cand
    chain = best[(len(p1) - 1, len(p2) - 1)]
    assert chain[0] == (0, 0)
    return [(p1[x], p2[y]) for x, y in chain]


def _region(nodes, dom, c, c_next):
    return [v for v in nodes if c in dom[v] and not (c_next in dom[v] and v != c_next)]


def match(n1, edges1, n2, edges2, eq):
    succ1 = {v: [] for v in range(n1)}
    for u, v in edges1:
        succ1[u].append(v)
    succ2 = {v: [] for v in range(n2)}
    for u, v in edges2:
        succ2[u].append(v)
    out = []

    def rec(nodes1, s1, e1, nodes2, s2, e2, eqs):
        p1, dom1 = dominator_path(nodes1, succ1, s1, e1)
        p2, dom2 = dominator_path(nodes2, succ2, s2, e2)
        cuts = _chain(p1, p2, eqs)
        if len(cuts) <= 2:
            out.append(((s1, e1), (s2, e2)))
            return
        for (a1, a2), (b1, b2) in zip(cuts, cuts[1:]):
            r1 = _region(nodes1, dom1, a1, b1)
            r2 = _region(nodes2, dom2, a2, b2)
            s1set, s2set = set(r1), set(r2)
            sub = [(a, b) for a, b in eqs if a in s1set and b in s2set]
            rec(r1, a1, b1, r2, a2, b2, sub)

    rec(list(range(n1)), 0, n1 - 1, list(range(n2)), 0, n2 - 1,
        [(int(a), int(b)) for a, b in eq])
    return out
