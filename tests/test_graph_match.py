"""Section 4.2's topology-aware subgraph matching in the library (host code,
through the C ABI) against the oracle: planted block structures, decoy pairs
off the dominator paths, crossing pairs, and the input checks."""
import numpy as np
import pytest

import synth
from oracle import graph_match as G


def _lib_match(c):
    import paper_2512_08365_amd as mag
    return mag.match_subgraphs(c["n1"], c["edges1"], c["n2"], c["edges2"], c["eq"])


@pytest.mark.parametrize("seed", range(12))
def test_planted_blocks_are_the_finest_pairs(seed):
    # without decoys every block boundary is a cut and the blocks are the pairs
    c = synth.graph_pair(seed, blocks=3 + seed % 6, width=2 + seed % 3, decoys=0)
    got = _lib_match(c)
    assert got == G.match(c["n1"], c["edges1"], c["n2"], c["edges2"], c["eq"])
    b1, b2 = c["bounds1"], c["bounds2"]
    assert got == [((b1[k], b1[k + 1]), (b2[k], b2[k + 1])) for k in range(len(b1) - 1)]


@pytest.mark.parametrize("seed", range(12))
def test_decoy_pairs_against_the_oracle(seed):
    # interior pairs count only where both lie on the dominator paths (blocks
    # of width 1 put their interior operators there)
    c = synth.graph_pair(50 + seed, blocks=4 + seed % 5, width=1 + seed % 4, decoys=8)
    assert _lib_match(c) == G.match(c["n1"], c["edges1"], c["n2"], c["edges2"], c["eq"])


@pytest.mark.parametrize("seed", range(12))
def test_crossing_pairs_against_the_oracle(seed):
    c = synth.graph_pair(100 + seed, blocks=6, width=3, crossing=1 + seed % 3)
    assert _lib_match(c) == G.match(c["n1"], c["edges1"], c["n2"], c["edges2"], c["eq"])


def test_large_graphs():
    # about 2,000 operators per graph (a few hundred blocks)
    c = synth.graph_pair(7, blocks=300, width=4, decoys=200, crossing=20)
    got = _lib_match(c)
    want = G.match(c["n1"], c["edges1"], c["n2"], c["edges2"], c["eq"])
    assert got == want and len(got) > 200


def test_input_checks():
    import paper_2512_08365_amd as mag
    from paper_2512_08365_amd import _native as N
    chain = [(0, 1), (1, 2)]
    with pytest.raises(mag.MagnetonError) as e:
        mag.match_subgraphs(3, [(0, 1), (1, 2), (2, 1)], 3, chain, [])  # a cycle
    assert e.value.code == N.MAG_E_GRAPH
    with pytest.raises(mag.MagnetonError) as e:
        mag.match_subgraphs(4, chain + [(0, 3)], 3, chain, [])  # node 2 off the 0 -> 3 paths
    assert e.value.code == N.MAG_E_GRAPH
    with pytest.raises(mag.MagnetonError) as e:
        mag.match_subgraphs(3, [(0, 5)], 3, chain, [])
    assert e.value.code == N.MAG_E_SIZE
    with pytest.raises(mag.MagnetonError) as e:
        mag.match_subgraphs(3, chain, 3, chain, [(0, 7)])
    assert e.value.code == N.MAG_E_SIZE
    with pytest.raises(mag.MagnetonError):
        mag.match_subgraphs(1, [], 3, chain, [])
