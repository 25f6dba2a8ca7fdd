"""Pins of the subgraph-matching oracle (Section 4.2's topology-aware
matching): dominators of hand-drawn graphs, and matchings worked out by hand,
among them the attention / feed-forward example of the paper's figure."""
from oracle import graph_match as G


def _succ(n, edges):
    s = {v: [] for v in range(n)}
    for u, v in edges:
        s[u].append(v)
    return s


def test_dominators_of_a_diamond_and_a_chain():
    # 0 -> 1 -> 3, 0 -> 2 -> 3, 3 -> 4
    edges = [(0, 1), (0, 2), (1, 3), (2, 3), (3, 4)]
    dom = G.dominators(list(range(5)), _succ(5, edges), 0)
    assert dom == {0: {0}, 1: {0, 1}, 2: {0, 2}, 3: {0, 3}, 4: {0, 3, 4}}
    path, _ = G.dominator_path(list(range(5)), _succ(5, edges), 0, 4)
    assert path == [0, 3, 4]


def test_paper_figure_attention_then_feed_forward():
    # App A: in(0) -> Q(1), K(2), V(3) -> Attn(4) -> Mul(5) -> Add(6) -> out(7)
    a_edges = [(0, 1), (0, 2), (0, 3), (1, 4), (2, 4), (3, 4), (4, 5), (4, 6), (5, 6), (6, 7)]
    # App B: in(0) -> QKV(1) -> Split(2) -> Attn(3) -> Linear(4) -> out(5)
    b_edges = [(0, 1), (1, 2), (2, 3), (3, 4), (4, 5)]
    # equivalent tensors: the inputs, the attention outputs, the block outputs
    eq = [(0, 0), (4, 3), (6, 4), (7, 5)]
    got = G.match(8, a_edges, 6, b_edges, eq)
    # cuts in, Attn, Add/Linear, out: three finest pairs, in path order
    assert got == [((0, 4), (0, 3)), ((4, 6), (3, 4)), ((6, 7), (4, 5))]


def test_no_interior_equivalence_gives_one_pair():
    a = [(0, 1), (1, 2), (2, 3)]
    b = [(0, 1), (0, 2), (1, 3), (2, 3)]
    assert G.match(4, a, 4, b, []) == [((0, 3), (0, 3))]


def test_crossing_pairs_keep_a_longest_rising_chain():
    # two chains 0-1-2-3-4; pairs (1,3) and (3,1) cross; (2,2) is compatible with both
    chain = [(0, 1), (1, 2), (2, 3), (3, 4)]
    got = G.match(5, chain, 5, chain, [(1, 3), (3, 1), (2, 2)])
    # longest chains: (0,0)-(1,3)?-... ; rising chains through (2,2) have 3 cuts + ends
    # candidates of length 3 interior-free: [(0,0),(2,2),(4,4)], [(0,0),(1,3),(4,4)],
    # [(0,0),(3,1),(4,4)]; the lexicographically smallest position chain is (1,3)
    # -> positions (0,0),(1,3),(4,4)
    assert got == [((0, 1), (0, 3)), ((1, 4), (3, 4))]


def test_several_cuts_and_branches():
    # graph 1: 0 -> {1, 2} -> 3 -> 4 -> {5, 6} -> 7 -> 8
    a = [(0, 1), (0, 2), (1, 3), (2, 3), (3, 4), (4, 5), (4, 6), (5, 7), (6, 7), (7, 8)]
    # graph 2: 0 -> 1 -> 2 -> {3, 4} -> 5 -> 6
    b = [(0, 1), (1, 2), (2, 3), (2, 4), (3, 5), (4, 5), (5, 6)]
    # cuts: 3~1, 4~2, 7~5 (node 1 of graph 1 is off the dominator path: ignored)
    got = G.match(9, a, 7, b, [(3, 1), (4, 2), (7, 5), (1, 3)])
    assert got == [((0, 3), (0, 1)), ((3, 4), (1, 2)), ((4, 7), (2, 5)), ((7, 8), (5, 6))]
