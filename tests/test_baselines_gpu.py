"""The paper's attention backends as measured beside the tree kernel (App. C:
dense SDPA over the materialised ancestor mask, and tree-varlen -- one causal
problem per branch over the gathered [prefix, stream[:fork], branch] keys,
bottom-right aligned), built from PyTorch-ROCm operations in the benchmark.
Each must compute the same function as the oracle: their outputs are compared
with the fp64 oracle at the bf16 tolerances on a paper-shaped tree."""
import math

import numpy as np
import pytest
import torch

import bench
import oracle
from oracle import dense as od
import padoc_synth as syn
import paper_2608_06146_amd as pa
from _cases import TOL

pytestmark = pytest.mark.gpu


def _pages():
    rng = np.random.default_rng(21)
    pages = []
    for _ in range(2):
        P, S, N = int(rng.integers(300, 700)), int(rng.integers(40, 120)), int(rng.integers(6, 14))
        f = np.sort(rng.integers(1, S + 1, N))
        L = np.clip(np.rint(rng.lognormal(math.log(40), 0.5, N)), 4, 200).astype(int)
        pages.append(syn.Page(P, P, S, S, tuple(syn.Branch(int(a), int(b), int(b)) for a, b in zip(f, L))))
    return pages


def test_forward_baselines_match_oracle():
    pages = _pages()
    segs = pa.segments_from_pages(pages, 0)
    nodes = od.page_nodes(pages)
    T = syn.count_tokens(pages)
    Hq, Hkv, d = 16, 2, 128
    q = syn.draw_normal((T, Hq, d), 3, 1, "bf16", device="cuda")
    k = syn.draw_normal((T, Hkv, d), 3, 2, "bf16", device="cuda")
    v = syn.draw_normal((T, Hkv, d), 3, 3, "bf16", device="cuda")
    plan = pa.TreePlan(segs, Hq, Hkv, d, "bf16", 0, num_kv_rows=T, num_q_rows=T)
    o_tree, _ = pa.tree_attn_fwd(q, k, v, plan)
    torch.cuda.synchronize()
    timing, outs = bench.forward_baselines(torch, np, segs, q, k, v, o_tree, Hq, Hkv, d, 1)
    O, _ = oracle.tree_attention(nodes, q, k, v, 1.0 / math.sqrt(d), Hq, Hkv)
    mx, mn = TOL["bf16"]
    for name in ("dense_sdpa", "tree_varlen"):
        x = outs[name].to("cpu", torch.float64).numpy()
        assert np.isfinite(x).all(), name
        e = np.abs(x - O)
        print(f"{name} ({timing[name].get('method', 'SDPA, dense mask')}): max-abs {e.max():.3e} "
              f"mean-abs {e.mean():.3e}", flush=True)
        assert e.max() <= mx and e.mean() <= mn, (name, e.max(), e.mean())
