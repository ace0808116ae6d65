"""Pins of the CPU oracle to things other than itself (no GPU needed).

Each test names the passage of the paper it follows.  A plausible slip in the
oracle -- a dropped ancestor term, an off-by-one fork, a missing scale, the
wrong log base, a transposed operand, the wrong GQA map -- fails at least one:

* P1  chain tree == causal attention computed by torch's SDPA (library routine)
* P2  every node == its root-to-node path run alone through causal SDPA
      (the tree-varlen identity of App. C), brute force over all tiny trees
* P3  perturbation invariance of siblings / future stream / other pages
* P4  softmax rows sum to one, exact zeros off the mask
* P5  closed forms with Q = 0 (LSE = ln n_visible, O = mean of visible V)
* P6  one-hot V recovers the probability matrix; its support is the mask
* P7  the visibility rule equals the logical fused mask of the masked
      parallel decoding algorithm (App. E), bit for bit
* P8  paged (decode) form == packed form on the same values
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import dense as ot
import padoc_synth as syn

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _sdpa(q, k, v, scale, causal=False, mask=None):
    """torch SDPA in fp64 on the CPU; q [n, d] (queries are the last n keys
    when causal, i.e. bottom-right alignment), k/v [m, d]."""
    qq = torch.as_tensor(q, dtype=torch.float64)[None, None]
    kk = torch.as_tensor(k, dtype=torch.float64)[None, None]
    vv = torch.as_tensor(v, dtype=torch.float64)[None, None]
    n, m = qq.shape[2], kk.shape[2]
    if causal:
        mask = torch.ones(n, m, dtype=torch.bool).tril(diagonal=m - n)
    if mask is not None:
        mask = torch.as_tensor(mask)
    out = F.scaled_dot_product_attention(qq, kk, vv, attn_mask=mask, scale=scale)
    return out[0, 0].numpy()


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


# ---------------------------------------------------------------- structure

def test_tiny_page_structure_matches_hand_derivation():
    """App. C packed sample for the tiny page; counts from the Sec. 3.2 rule."""
    gold = json.load(open(os.path.join(GOLD, "tiny_page_structure.json")))
    wl = syn.make_workload("tiny_fp32_forward")
    nodes = ot.page_nodes(wl.pages)
    kv_off, q_off = ot.canonical_layout(nodes, 0)
    for s, g in enumerate(gold["segments"]):
        assert nodes[s] == (g["parent"], g["fork"], g["len"], g["q_len"])
        assert kv_off[s] == g["kv_off"] and q_off[s] == g["q_off"]
    bt_off, _ = ot.canonical_layout(nodes, 16)
    assert list(bt_off) == gold["paged_block_offsets_block16"]
    assert ot.visible_pair_count(nodes) == gold["visible_pairs"]["total"]
    _, _, mask = ot.dense_mask(nodes, 0)
    per_row = mask.sum(1)
    assert per_row[:256].sum() == gold["visible_pairs"]["prefix"]
    assert per_row[256:320].sum() == gold["visible_pairs"]["stream"]
    for k in range(4):
        assert per_row[320 + 32 * k: 352 + 32 * k].sum() == gold["visible_pairs"]["branches"][k]
    assert mask.sum() == gold["visible_pairs"]["total"]
    assert gold["causal_pairs_same_length"] == 448 * 449 // 2


def test_attention_mask_rows_equal_elementwise_mask():
    """The mask rows tree_attention builds (segment slices) equal the
    element-by-element rule of dense_mask: one-hot V exposes the support."""
    for seed in range(30):
        nodes = [(a.parent, a.fork, a.length, a.length) for a in syn.random_tree(seed, n_pages=2)]
        T = sum(n[2] for n in nodes)
        q = _rand((T, 1, 3), seed)
        k = _rand((T, 1, 3), seed + 1)
        O, _ = oracle.tree_attention(nodes, q, k, np.eye(T)[:, None, :], 0.5, 1, 1)
        support = O[:, 0, :] > 0
        roots = ot.page_of(nodes)
        kv_off, _ = ot.canonical_layout(nodes, 0)
        for root in set(int(r) for r in roots):
            seg, pos, mask = ot.dense_mask(nodes, root)
            rows = np.array([kv_off[s] + p for s, p in zip(seg, pos)])
            np.testing.assert_array_equal(support[np.ix_(rows, rows)], mask)
            others = np.setdiff1d(np.arange(T), rows)
            assert not support[np.ix_(rows, others)].any()


def test_closed_form_visible_counts_for_page_trees():
    """n_vis = p+1 (prefix), P+p+1 (stream), P+f_k+p+1 (branch)."""
    pg = syn.Page(5, 5, 4, 4, (syn.Branch(0, 3, 3), syn.Branch(2, 2, 2), syn.Branch(4, 1, 1)))
    nodes = ot.page_nodes([pg])
    _, _, mask = ot.dense_mask(nodes, 0)
    n = mask.sum(1)
    exp = [p + 1 for p in range(5)] + [5 + p + 1 for p in range(4)]
    for b in pg.branches:
        exp += [5 + b.fork + p + 1 for p in range(b.length)]
    np.testing.assert_array_equal(n, exp)


# ---------------------------------------------------------------- P1

@pytest.mark.parametrize("G", [1, 4])
def test_P1_chain_equals_causal_sdpa(G):
    """A single-branch tree with f = S is one causal sequence (App. C)."""
    P, S, L, d, Hkv = 7, 5, 6, 16, 2
    pg = syn.Page(P, P, S, S, (syn.Branch(S, L, L),))
    nodes = ot.page_nodes([pg])
    T = P + S + L
    Hq = G * Hkv
    q, k, v = _rand((T, Hq, d), 1), _rand((T, Hkv, d), 2), _rand((T, Hkv, d), 3)
    O, LSE = oracle.tree_attention(nodes, q, k, v, 0.3, Hq, Hkv)
    for h in range(Hq):
        ref = _sdpa(q[:, h], k[:, h // G], v[:, h // G], 0.3, causal=True)
        np.testing.assert_allclose(O[:, h], ref, rtol=0, atol=1e-12)
    # K/V repeated per group (MHA) gives the same result: pins the GQA map
    kr, vr = np.repeat(k, G, axis=1), np.repeat(v, G, axis=1)
    O2, LSE2 = oracle.tree_attention(nodes, q, kr, vr, 0.3, Hq, Hq)
    np.testing.assert_allclose(O, O2, atol=1e-12)
    np.testing.assert_allclose(LSE, LSE2, atol=1e-12)


def test_P1_interleaved_gqa_map_differs():
    """Negative control: the interleaved head map h % Hkv gives another answer."""
    P, S, d, Hkv, G = 6, 3, 8, 2, 2
    nodes = ot.page_nodes([syn.Page(P, P, S, S, ())])
    T, Hq = P + S, Hkv * G
    q, k, v = _rand((T, Hq, d), 4), _rand((T, Hkv, d), 5), _rand((T, Hkv, d), 6)
    O, _ = oracle.tree_attention(nodes, q, k, v, 0.5, Hq, Hkv)
    ref_inter = np.stack([_sdpa(q[:, h], k[:, h % Hkv], v[:, h % Hkv], 0.5, causal=True)
                          for h in range(Hq)], 1)
    assert not np.allclose(O, ref_inter, atol=1e-6)


def test_masked_attention_equals_sdpa_with_bool_mask():
    rng = np.random.default_rng(7)
    for _ in range(20):
        n, m, d = rng.integers(1, 9), rng.integers(1, 12), 8
        mask = rng.random((n, m)) < 0.5
        mask[np.arange(n), rng.integers(0, m, n)] = True
        q, k, v = rng.standard_normal((n, d)), rng.standard_normal((m, d)), rng.standard_normal((m, d))
        o, lse = oracle.masked_attention(q, k, v, mask, 0.7)
        np.testing.assert_allclose(o, _sdpa(q, k, v, 0.7, mask=mask), atol=1e-12)
        # LSE: scipy's logsumexp over the visible scaled scores
        from scipy.special import logsumexp
        s = 0.7 * q @ k.T
        ref = np.array([logsumexp(s[i][mask[i]]) for i in range(n)])
        np.testing.assert_allclose(lse, ref, atol=1e-12)


def test_lse_single_visible_key_closed_form():
    """The first prefix token sees only itself: LSE = scale * q . k exactly."""
    nodes = ot.page_nodes([syn.Page(3, 3, 2, 2, ())])
    q, k, v = _rand((5, 2, 4), 8), _rand((5, 1, 4), 9), _rand((5, 1, 4), 10)
    O, LSE = oracle.tree_attention(nodes, q, k, v, 0.25, 2, 1)
    for h in range(2):
        assert LSE[0, h] == pytest.approx(0.25 * float(q[0, h] @ k[0, 0]), abs=1e-14)
        np.testing.assert_allclose(O[0, h], v[0, 0], atol=1e-14)


# ---------------------------------------------------------------- P2

def _path_check(nodes, d=4, Hq=2, Hkv=1, seed=0):
    T = sum(n[2] for n in nodes)
    nq = sum(n[3] for n in nodes)
    kv_off, q_off = ot.canonical_layout(nodes, 0)
    q, k, v = _rand((nq, Hq, d), seed), _rand((T, Hkv, d), seed + 1), _rand((T, Hkv, d), seed + 2)
    O, LSE = oracle.tree_attention(nodes, q, k, v, 0.5, Hq, Hkv)
    G = Hq // Hkv
    for s, (_, _, n, ql) in enumerate(nodes):
        if ql == 0:
            continue
        rows = []
        for t, f in ot.ancestors(nodes, s):
            rows += list(range(kv_off[t], kv_off[t] + f))
        rows += list(range(kv_off[s], kv_off[s] + n))
        qs = slice(q_off[s], q_off[s] + ql)
        for h in range(Hq):
            ref = _sdpa(q[qs, h], k[rows, h // G], v[rows, h // G], 0.5, causal=True)
            np.testing.assert_allclose(O[qs, h], ref, rtol=0, atol=1e-12)


def test_P2_path_decomposition_brute_force_two_branches():
    """All trees with P in 1..3, S in 1..4, N in 0..2, f in 0..S, L in 1..3."""
    count = 0
    for P in range(1, 4):
        for S in range(1, 5):
            for N in range(0, 3):
                for fs in itertools.product(range(0, S + 1), repeat=N):
                    for Ls in itertools.product(range(1, 4), repeat=N):
                        if N == 2 and (P, S) not in ((1, 1), (3, 4), (2, 3)):
                            continue
                        br = tuple(syn.Branch(f, L, L) for f, L in zip(fs, Ls))
                        _path_check(ot.page_nodes([syn.Page(P, P, S, S, br)]), seed=count)
                        count += 1
    assert count > 300


def test_P2_path_decomposition_three_branches_sampled():
    rng = np.random.default_rng(11)
    for i in range(60):
        P, S = int(rng.integers(1, 4)), int(rng.integers(1, 5))
        br = tuple(syn.Branch(int(rng.integers(0, S + 1)), int(rng.integers(1, 4)), 0) for _ in range(3))
        br = tuple(syn.Branch(b.fork, b.length, int(rng.integers(0, b.length + 1))) for b in br)
        _path_check(ot.page_nodes([syn.Page(P, int(rng.integers(0, P + 1)), S, int(rng.integers(0, S + 1)), br)]), seed=i)


def test_P2_random_deep_trees():
    """Depth up to 5 (the descriptor allows any depth with parent < self)."""
    for seed in range(25):
        nodes = [(a.parent, a.fork, a.length, a.q_len)
                 for a in syn.random_tree(seed, n_pages=2, max_depth=5, q_mode="some")]
        _path_check(nodes, Hq=4, Hkv=2, seed=seed)


# ---------------------------------------------------------------- P3

def test_P3_perturbation_invariance():
    """A content branch observes neither siblings nor later layout tokens nor
    another page (Sec. 3.3; App. E): perturbing them leaves its rows bit-identical."""
    pages = [syn.Page(4, 4, 6, 6, (syn.Branch(2, 3, 3), syn.Branch(4, 3, 3), syn.Branch(4, 2, 2))),
             syn.Page(3, 3, 2, 2, (syn.Branch(1, 2, 2),))]
    nodes = ot.page_nodes(pages)
    kv_off, q_off = ot.canonical_layout(nodes, 0)
    T, nq, d = sum(n[2] for n in nodes), sum(n[3] for n in nodes), 8
    q, k, v = _rand((nq, 2, d), 20), _rand((T, 1, d), 21), _rand((T, 1, d), 22)
    O0, L0 = oracle.tree_attention(nodes, q, k, v, 0.4, 2, 1)
    b1 = 2  # first branch of page 0: fork 2, 3 tokens
    mine = slice(q_off[b1], q_off[b1] + 3)
    perturb_rows = []
    perturb_rows += list(range(kv_off[3], kv_off[3] + 3))                 # sibling
    perturb_rows += list(range(kv_off[4], kv_off[4] + 2))                 # sibling
    perturb_rows += list(range(kv_off[1] + 2, kv_off[1] + 6))             # stream tokens >= f
    perturb_rows += list(range(kv_off[5], T))                             # other page
    k2, v2 = k.copy(), v.copy()
    k2[perturb_rows] += 3.0
    v2[perturb_rows] -= 5.0
    O1, L1 = oracle.tree_attention(nodes, q, k2, v2, 0.4, 2, 1)
    np.testing.assert_array_equal(O0[mine], O1[mine])
    np.testing.assert_array_equal(L0[mine], L1[mine])
    # own future tokens: the branch's first query must not see its 2nd/3rd token
    k3 = k.copy()
    k3[kv_off[b1] + 1: kv_off[b1] + 3] += 1.0
    O2, _ = oracle.tree_attention(nodes, q, k3, v, 0.4, 2, 1)
    np.testing.assert_array_equal(O0[q_off[b1]], O2[q_off[b1]])
    # control: perturbing a visible stream token does change the output
    k4 = k.copy()
    k4[kv_off[1] + 1] += 1.0
    O3, _ = oracle.tree_attention(nodes, q, k4, v, 0.4, 2, 1)
    assert not np.array_equal(O0[mine], O3[mine])


# ---------------------------------------------------------------- P4, P6

def test_P4_P6_probabilities_and_support():
    for seed in range(10):
        nodes = [(a.parent, a.fork, a.length, a.q_len) for a in syn.random_tree(seed, n_pages=2)]
        T = sum(n[2] for n in nodes)
        nq = sum(n[3] for n in nodes)
        kv_off, q_off = ot.canonical_layout(nodes, 0)
        q = _rand((nq, 1, 6), seed)
        k = _rand((T, 1, 6), seed + 100)
        v = np.eye(T)[:, None, :]                   # one-hot V: row j = e_j
        O, LSE, Pm = oracle.tree_attention(nodes, q, k, v, 0.8, 1, 1, return_probs=True)
        np.testing.assert_allclose(Pm.sum(-1), 1.0, atol=1e-12)         # P4
        np.testing.assert_allclose(O[:, 0, :], Pm[:, 0, :], atol=1e-15)  # P6
        # expected support straight from the visibility rule
        exp = np.zeros((nq, T), dtype=bool)
        for s, (_, _, n, ql) in enumerate(nodes):
            for i in range(ql):
                p = n - ql + i
                for t, c in ot.visible_counts(nodes, s, p).items():
                    exp[q_off[s] + i, kv_off[t]: kv_off[t] + c] = True
        np.testing.assert_array_equal(O[:, 0, :] > 0, exp)
        assert np.all(Pm[:, 0, :][~exp] == 0.0)


# ---------------------------------------------------------------- P5

def test_P5_zero_query_closed_form():
    pg = syn.Page(6, 6, 5, 5, (syn.Branch(1, 4, 4), syn.Branch(5, 2, 2)))
    nodes = ot.page_nodes([pg])
    T = 6 + 5 + 6
    q = np.zeros((T, 3, 4))
    v = _rand((T, 1, 4), 30)
    k = _rand((T, 1, 4), 31)
    O, LSE = oracle.tree_attention(nodes, q, k, v, 1.3, 3, 1)
    nvis = [p + 1 for p in range(6)] + [6 + p + 1 for p in range(5)]
    nvis += [6 + 1 + p + 1 for p in range(4)] + [6 + 5 + p + 1 for p in range(2)]
    np.testing.assert_allclose(LSE, np.log(np.array(nvis, float))[:, None].repeat(3, 1), atol=1e-13)
    # O = mean of the visible V rows, visible sets written out by hand
    def rows_of(r):
        if r < 6:
            return list(range(r + 1))
        if r < 11:
            return list(range(6)) + list(range(6, r + 1))
        if r < 15:
            return list(range(6)) + [6] + list(range(11, r + 1))
        return list(range(6)) + list(range(6, 11)) + list(range(15, r + 1))
    for r in range(T):
        np.testing.assert_allclose(O[r, 0], v[rows_of(r), 0].mean(0), atol=1e-13)


# ---------------------------------------------------------------- P7

def _run_alg1(seed, P=3, steps=14):
    rng = np.random.default_rng(seed)

    def decide(step, c, is_layout):
        u = rng.random()
        if is_layout:
            if step >= steps - 1 or u < 0.08:
                return "eos"
            return "fork" if u < 0.45 else "continue"
        return "eos" if u < 0.25 else "continue"

    return ot.simulate_masked_parallel_decoding(P, decide, max_steps=steps + 20)


@pytest.mark.parametrize("seed", range(12))
def test_P7_visibility_equals_masked_parallel_decoding(seed):
    P = 3
    tags, queries, forks = _run_alg1(seed, P)
    counts = {}
    for c, i in tags:
        counts[c] = max(counts.get(c, 0), i + 1)
    children = sorted(c for c in counts if c > 0)
    nodes = [(-1, 0, P, 0), (0, P, counts.get(0, 0), counts.get(0, 0))]
    seg_of = {-1: 0, 0: 1}
    for c in children:
        seg_of[c] = len(nodes)
        nodes.append((1, forks[c], counts[c], counts[c]))
    kv_off, _ = ot.canonical_layout(nodes, 0)
    seg, pos, mask = ot.dense_mask(nodes, 0)
    packed_row = {(int(s), int(p)): a for a, (s, p) in enumerate(zip(seg, pos))}
    assert len(queries) > 0
    for c, i, row in queries:
        q = packed_row[(seg_of[c], i)]
        want = set()
        for l, (cc, ii) in enumerate(tags[:row.size]):
            if row[l]:
                want.add(packed_row[(seg_of[cc], ii)])
        got = set(np.nonzero(mask[q])[0].tolist())
        assert got == want, (c, i)


def test_P7_fork_offset_counts_pre_boundary_tokens():
    """A child forked when the layout stream has cached f tokens sees exactly
    stream tokens [0, f): the boundary output itself is appended later."""
    script = {(0, 0): "continue", (1, 0): "fork", (2, 0): "continue", (3, 0): "eos"}

    def decide(step, c, is_layout):
        return script.get((step, c), "eos" if step >= 3 else "continue")

    tags, queries, forks = ot.simulate_masked_parallel_decoding(2, decide, max_steps=10)
    assert forks[1] == 2                     # two layout tokens cached at the fork
    first_child = [row for c, i, row in queries if c == 1 and i == 0][0]
    seen = [tags[l] for l in range(first_child.size) if first_child[l]]
    assert seen == [(-1, 0), (-1, 1), (0, 0), (0, 1), (1, 0)]


# ---------------------------------------------------------------- P8

def test_P8_paged_equals_packed():
    rng = np.random.default_rng(40)
    for seed in range(6):
        nodes = [(a.parent, a.fork, a.length, a.q_len)
                 for a in syn.random_tree(seed, n_pages=2, max_len=40, q_mode="tail")]
        T = sum(n[2] for n in nodes)
        nq = sum(n[3] for n in nodes)
        if nq == 0:
            continue
        Hkv, d = 2, 8
        k, v = _rand((T, Hkv, d), seed), _rand((T, Hkv, d), seed + 1)
        q = _rand((nq, 4, d), seed + 2)
        O_p, L_p = oracle.tree_attention(nodes, q, k, v, 0.3, 4, Hkv)
        bt_off, _ = ot.canonical_layout(nodes, 16)
        nb = int(sum(-(-n[2] // 16) for n in nodes))
        pool_n = nb + 7
        ids = syn.draw_block_ids(nb, pool_n, seed)
        pool_k = np.full((pool_n, Hkv, d // 8, 16, 8), np.nan)  # K blocks are chunk-major
        pool_v = np.full((pool_n, Hkv, d, 16), np.nan)      # V blocks are d-major
        blk, slot = ot.paged_slots(nodes, ids, 16)
        pool_k[blk, :, :, ot.chunk_slot(slot), :] = k.reshape(len(slot), Hkv, d // 8, 8)
        pool_v[blk, :, :, slot] = v
        O_d, L_d = oracle.tree_attention_paged(nodes, q, pool_k, pool_v, ids, 0.3, 4, Hkv, 16)
        np.testing.assert_allclose(O_d, O_p, atol=1e-12)
        np.testing.assert_allclose(L_d, L_p, atol=1e-12)
        assert np.isfinite(O_d).all()


def test_chunk_major_k_layout():
    """Chunk-major paged K blocks: the slot table written out, its own
    inverse, the two 128-byte line groups, and a gather read element by
    element from a pool whose values encode their own position."""
    s = ot.chunk_slot(np.arange(16))
    assert list(s) == [0, 1, 2, 3, 8, 9, 10, 11, 4, 5, 6, 7, 12, 13, 14, 15]
    assert list(ot.chunk_slot(s)) == list(range(16))
    assert set(np.arange(16)[s < 8]) == {0, 1, 2, 3, 8, 9, 10, 11}
    nodes = [(-1, 0, 37, 0), (0, 20, 9, 1)]
    Hkv, d = 2, 16
    nb = 3 + 1
    ids = np.array([5, 2, 7, 0], dtype=np.int32)
    pool = np.zeros((8, Hkv, d // 8, 16, 8))
    for b in range(8):
        for h in range(Hkv):
            for c in range(d // 8):
                for sl in range(16):
                    for e in range(8):
                        pool[b, h, c, sl, e] = b * 1e6 + h * 1e4 + c * 1e3 + sl * 10 + e
    got = ot.gather_paged(nodes, pool, ids, 16, layout="chunked")
    assert got.shape == (37 + 9, Hkv, d)
    bt_off, _ = ot.canonical_layout(nodes, 16)
    row = 0
    for seg, (_, _, ln, _) in enumerate(nodes):
        for j in range(ln):
            b = ids[bt_off[seg] + j // 16]
            t = j % 16
            for h in range(Hkv):
                for dim in range(d):
                    c, e = divmod(dim, 8)
                    assert got[row, h, dim] == b * 1e6 + h * 1e4 + c * 1e3 + int(ot.chunk_slot(t)) * 10 + e
            row += 1


# ---------------------------------------------------------------- P9 decoding depths

def test_P9_depths_of_a_worked_page():
    """Sec. 3.1 by hand: layout 12 tokens; branches (fork 3, 20 tokens),
    (fork 7, 2), (fork 12, 5).  Sequential: 12 + 20 + 2 + 5 = 39 steps;
    critical path: max(12, 3 + 20, 7 + 2, 12 + 5) = 23."""
    nodes = [(-1, 0, 50, 0), (0, 50, 12, 12), (1, 3, 20, 20), (1, 7, 2, 2), (1, 12, 5, 5)]
    assert ot.decoding_depths(nodes) == {0: (39, 23)}
    # a branch of a branch starts after its parent's fork tokens: 3 + 4 + 9
    nodes.append((2, 4, 9, 9))
    assert ot.decoding_depths(nodes) == {0: (48, 23)}
    nodes.append((5, 9, 3, 3))      # 3 + 4 + 9 + 3 = 19
    nodes.append((2, 20, 8, 8))     # 3 + 20 + 8 = 31
    assert ot.decoding_depths(nodes) == {0: (59, 31)}


@pytest.mark.parametrize("seed", range(10))
def test_P9_depths_equal_alg1_step_counts(seed):
    """The replay of masked parallel decoding takes exactly D_crit steps and
    decodes exactly D_seq tokens, on the tree its events produce."""
    P = 4
    tags, queries, forks = _run_alg1(seed, P)
    counts = {}
    for c, i in tags:
        counts[c] = max(counts.get(c, 0), i + 1)
    nodes = [(-1, 0, P, 0), (0, P, counts.get(0, 0), counts.get(0, 0))]
    for c in sorted(k for k in counts if k > 0):
        nodes.append((1, forks[c], counts[c], counts[c]))
    # step of each query: the mask row grows by the live count each step
    sizes = sorted(set(row.size for _, _, row in queries))
    steps = len(sizes)
    d_seq, d_crit = ot.decoding_depths(nodes)[0]
    assert d_seq == len(queries)
    assert d_crit == steps


# ---------------------------------------------------------------- P10 remaining paths, budgeted steps

def _worked_page():
    return [(-1, 0, 50, 0), (0, 50, 12, 12), (1, 3, 20, 20), (1, 7, 2, 2), (1, 12, 5, 5),
            (2, 4, 9, 9), (5, 9, 3, 3), (2, 20, 8, 8)]


def test_P10_remaining_paths_of_the_worked_page():
    """The worked page of P9 by hand.  From the start every segment's path
    is counted from its own start: layout max(12, 3+20+8, 3+4+9+3, 7+2,
    12+5) = 31 (= D_crit); branch 2: max(20, 4+9+3, 20+8) = 28; branch 5:
    9+3 = 12.  After the layout has produced 5 tokens and branch 2 one
    (branch 3 not yet: it starts at 7): layout max(12-5, 7-5+2, 12-5+5) =
    12; branch 2: max(19, 4-1+12, 20-1+8) = 27; the page: max(12, 27) = 27
    (the started segments 1 and 2)."""
    nodes = _worked_page()
    assert ot.remaining_paths(nodes).tolist() == [31, 31, 28, 2, 5, 12, 3, 8]
    prog = [0, 5, 1, 0, 0, 0, 0, 0]
    assert ot.remaining_paths(nodes, prog).tolist() == [27, 12, 27, 2, 5, 12, 3, 8]


@pytest.mark.parametrize("seed", range(8))
def test_P10_root_path_is_the_critical_path(seed):
    """From the start, each root's remaining path is its page's D_crit."""
    nodes = [(a.parent, a.fork, a.length, a.q_len)
             for a in syn.random_tree(seed, n_pages=2, max_len=6, max_depth=4)]
    dep = ot.decoding_depths(nodes)
    rem = ot.remaining_paths(nodes)
    for r, (_, crit) in dep.items():
        assert rem[r] == crit


def _brute_force_min_steps(nodes, max_rows):
    """Fewest steps to decode the tree with at most max_rows segments
    advancing per step, by breadth-first search over progress states
    (tiny trees only)."""
    import itertools
    n = len(nodes)
    dec = [s for s in range(n) if nodes[s][0] >= 0]
    start = tuple(0 for _ in range(n))
    frontier, seen, steps = {start}, {start}, 0
    while True:
        if any(all(st[s] == nodes[s][2] for s in dec) for st in frontier):
            return steps
        nxt = set()
        for st in frontier:
            started = ot._started(nodes, list(st))
            cand = [s for s in dec if started[s] and st[s] < nodes[s][2]]
            for k in range(1, min(max_rows, len(cand)) + 1):
                for pick in itertools.combinations(cand, k):
                    t = list(st)
                    for s in pick:
                        t[s] += 1
                    t = tuple(t)
                    if t not in seen:
                        seen.add(t)
                        nxt.add(t)
        frontier, steps = nxt, steps + 1


@pytest.mark.parametrize("seed", range(6))
def test_P10_budgeted_steps_bounds(seed):
    """Every schedule advances at most max_rows segments a step, decodes
    every token exactly once, and takes at least max(D_crit, D_seq /
    max_rows) steps; with room for every started segment both orders take
    exactly D_crit steps."""
    nodes = [(a.parent, a.fork, a.length, a.q_len)
             for a in syn.random_tree(seed + 3, n_pages=2, max_len=7, max_depth=4, max_children=3)]
    dep = ot.decoding_depths(nodes)
    d_seq = sum(v[0] for v in dep.values())
    d_crit = max(v[1] for v in dep.values())
    for B in (1, 2, 3, 1000):
        for by_pr in (False, True):
            steps = ot.budgeted_decoding(nodes, B, by_pr)
            assert all(len(x) <= B for x in steps)
            count = {}
            for x in steps:
                for s in x:
                    count[s] = count.get(s, 0) + 1
            assert all(count.get(s, 0) == nodes[s][2] for s in range(len(nodes)) if nodes[s][0] >= 0)
            assert len(steps) >= max(d_crit, -(-d_seq // B))
            if B == 1000:
                assert len(steps) == d_crit


@pytest.mark.parametrize("seed", range(6))
def test_P10_critical_path_first_is_optimal_on_independent_streams(seed):
    """Streams that fork nothing (chains below a root): taking the longest
    remaining path first is optimal -- checked against an exhaustive search
    of every schedule on small cases -- and oldest first is not always."""
    rng = np.random.default_rng(seed)
    n = int(rng.integers(3, 5))
    nodes = [(-1, 0, 4, 0)] + [(0, 4, int(x), int(x)) for x in rng.integers(1, 5, size=n)]
    for B in (1, 2):
        best = _brute_force_min_steps(nodes, B)
        assert len(ot.budgeted_decoding(nodes, B, True)) == best
        assert len(ot.budgeted_decoding(nodes, B, False)) >= best
    # a case where the order matters: short streams opened first
    nodes = [(-1, 0, 4, 0), (0, 4, 1, 1), (0, 4, 1, 1), (0, 4, 4, 4)]
    assert len(ot.budgeted_decoding(nodes, 2, True)) == _brute_force_min_steps(nodes, 2) == 4
    assert len(ot.budgeted_decoding(nodes, 2, False)) == 5
