"""padoc_branch_decode_no_alloc (the decode step on the library's fixed
per-GPU workspace) against padoc_branch_decode on the same plans and inputs:
two calls in a row, the second with a smaller tree, each bit-identical to the
workspace entry point and within the bf16 bounds of the oracle."""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import dense as od
import padoc_synth as syn
import paper_2608_06146_amd as pa
from _cases import compare, fill_pool

pytestmark = pytest.mark.gpu


def _case(pages, Hq, Hkv, d, seed, n_pool):
    segs = pa.segments_from_pages(pages, 16)
    nodes = od.page_nodes(pages)
    T, nq = syn.count_tokens(pages), syn.count_queries(pages)
    q = syn.draw_normal((nq, Hq, d), seed, 1, "bf16", device="cuda")
    k = syn.draw_normal((T, Hkv, d), seed, 2, "bf16", device="cuda")
    v = syn.draw_normal((T, Hkv, d), seed, 3, "bf16", device="cuda")
    kc, vc, ids = fill_pool(nodes, k, v, n_pool, seed)
    bt = torch.as_tensor(ids, device="cuda")
    plan = pa.TreePlan(segs, Hq, Hkv, d, "bf16", 16, num_kv_rows=n_pool, num_q_rows=nq, block_table_host=ids)
    return nodes, plan, q, kc, vc, bt, ids


def test_no_alloc_decode_matches_workspace_entry_point():
    big = syn.make_workload("single_page_decode").pages
    rng = np.random.default_rng(4)
    small = [syn.Page(180, 0, 30, 1, tuple(syn.Branch(int(f), int(L), 1) for f, L in
                                           zip(np.sort(rng.integers(1, 30, 5)), rng.integers(1, 90, 5))))]
    for i, (pages, n_pool) in enumerate(((big, 400), (small, 60))):
        nodes, plan, q, kc, vc, bt, ids = _case(pages, 16, 2, 128, 40 + i, n_pool)
        assert plan.workspace_bytes <= pa.NO_ALLOC_WORKSPACE_BYTES
        print(f"[case] no-alloc call {i}: {q.shape[0]} queries, workspace {plan.workspace_bytes} bytes", flush=True)
        o_ref, l_ref = pa.branch_decode(q, kc, vc, bt, plan)
        o = torch.full_like(o_ref, float("nan"))
        lse = torch.full_like(l_ref, float("nan"))
        pa.branch_decode_no_alloc(q, kc, vc, bt, plan, o, lse)
        torch.cuda.synchronize()
        assert torch.equal(o, o_ref) and torch.equal(lse, l_ref), f"call {i}: differs from padoc_branch_decode"
        O, L = oracle.tree_attention_paged(nodes, q, kc, vc, ids, 1.0 / math.sqrt(128), 16, 2, 16)
        compare(f"no-alloc call {i}", o, lse, O, L, "bf16")
