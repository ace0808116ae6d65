"""GPU parity of the backward (padoc_tree_attn_bwd) against the fp64
backward oracle, through the C ABI, on seeded bf16 trees."""
import numpy as np
import pytest

import padoc_synth as syn
from _cases import backward_case

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("heads", [(4, 1), (16, 2), (28, 4)])
@pytest.mark.parametrize("d", [64, 128])
def test_backward_random_trees(heads, d):
    """Depth <= 5, segments up to 90 tokens (several 64-key tiles and 128-key
    runs, ragged tails), forks anywhere, some segments with fewer queries
    than tokens."""
    Hq, Hkv = heads
    for seed in range(2):
        nodes = syn.random_tree(300 + 10 * seed + d + Hq, n_pages=2, max_depth=5, max_len=90,
                                q_mode="all" if seed == 0 else "some", max_nodes=14)
        if sum(n.q_len for n in nodes) == 0:
            continue
        backward_case(nodes, Hq, Hkv, d, seed)


def test_backward_page_split_columns():
    """A page whose prefix keys are seen by more than 1024 query columns, so
    their runs are split over several items that add into the same rows."""
    rng = np.random.default_rng(9)
    N = 30
    f = np.sort(rng.integers(0, 97, N))
    L = rng.integers(1, 60, N)
    page = syn.Page(300, 300, 96, 96, tuple(syn.Branch(int(a), int(b), int(b)) for a, b in zip(f, L)))
    errs, plan = backward_case([page], 16, 2, 128, 7)
    ex = plan.export()
    assert (ex["bwd"]["col0"] > 0).any(), "expected split key runs"


def test_backward_edge_cases():
    # single tokens, forks 0 and full, q_len 0 segments, a 200-token root
    nodes = [(-1, 0, 1, 1), (0, 0, 1, 1), (0, 1, 3, 0), (2, 3, 2, 2), (2, 0, 1, 1), (-1, 0, 200, 7),
             (5, 200, 1, 1), (5, 0, 65, 65), (7, 64, 64, 64), (7, 65, 1, 0)]
    for heads in [(1, 1), (8, 1), (12, 3)]:
        backward_case(nodes, heads[0], heads[1], 128, 3)
        backward_case(nodes, heads[0], heads[1], 64, 5)
