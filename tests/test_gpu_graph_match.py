"""The subgraph matching (host code behind mag_match_subgraphs) run on the GPU
host with the same library build as the GPU tests, against the oracle: the
CPU suite covers it in full (test_graph_match.py); this keeps its parity in
the GPU run's record as well."""
import pytest

import synth
from oracle import graph_match as G

pytestmark = pytest.mark.gpu


def _check(c):
    import paper_2512_08365_amd as mag
    got = mag.match_subgraphs(c["n1"], c["edges1"], c["n2"], c["edges2"], c["eq"])
    assert got == G.match(c["n1"], c["edges1"], c["n2"], c["edges2"], c["eq"])
    return got


@pytest.mark.parametrize("seed", range(3))
def test_planted_decoy_and_crossing_pairs(seed):
    b = _check(synth.graph_pair(seed, blocks=3 + seed, width=2 + seed, decoys=0))
    assert len(b) == 3 + seed  # one pair per planted block
    _check(synth.graph_pair(50 + seed, blocks=4 + seed, width=1 + seed, decoys=8))
    _check(synth.graph_pair(100 + seed, blocks=6, width=3, crossing=1 + seed))


def test_large_graph_pair():
    got = _check(synth.graph_pair(7, blocks=300, width=4, decoys=200, crossing=20))
    assert len(got) > 200
