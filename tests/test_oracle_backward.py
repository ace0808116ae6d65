"""Pins of the backward oracle to things other than itself (no GPU needed).

The backward oracle (``oracle.backward``) writes out the closed-form gradient
of masked softmax attention over the tree's ancestor mask (App. E, the Attn
equation; App. C, the tree-varlen relation it is trained with).  A plausible
slip -- a dropped D term, a missing scale, dK and dQ swapped, a transposed
product, GQA gradients not summed over the group, a shared prefix counted for
one branch only -- fails at least one of:

* B1  finite differences of the (pinned) forward oracle's loss sum(dO * O)
* B2  torch autograd through each segment's root-to-segment path run alone
      through causal SDPA (the tree-varlen identity of App. C), with the
      gradients of shared rows summed by the gather's own transpose
* B3  exact invariants: per KV head, sum_j dK_j = 0 (softmax gradients sum to
      zero over each row's keys) and sum_j dV_j = sum of dO over the group's
      query rows (probabilities sum to one)
* B4  the stored-output form: D from a given O equals the exact form when O
      is the exact forward output, and a perturbation dO_i . delta of the
      stored O_i shifts dQ_i by exactly -c * delta_D * sum_j P_ij k_j
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import dense as ot
import padoc_synth as syn


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def _problem(nodes, Hq, Hkv, d, seed):
    ko, qo = ot.canonical_layout(nodes, 0)
    T = int(sum(n[2] for n in nodes))
    nq = int(sum(n[3] for n in nodes))
    q = _rand((nq, Hq, d), seed)
    k = _rand((T, Hkv, d), seed + 1)
    v = _rand((T, Hkv, d), seed + 2)
    do = _rand((nq, Hq, d), seed + 3)
    return ko, qo, q, k, v, do


def _tiny_nodes():
    # one page: prefix 5, stream 4, branches forking at 1 and 3 (lengths 3, 2)
    return ot.page_nodes([syn.Page(5, 5, 4, 4, (syn.Branch(1, 3, 3), syn.Branch(3, 2, 2)))])


def test_B1_finite_differences():
    nodes = _tiny_nodes()
    Hq, Hkv, d, scale = 4, 2, 8, 0.37
    ko, qo, q, k, v, do = _problem(nodes, Hq, Hkv, d, 5)

    def loss(qq, kk, vv):
        o, _ = ot.tree_attention(nodes, qq, kk, vv, scale, Hq, Hkv, kv_off=ko, q_off=qo)
        return float(np.sum(o * do))

    dq, dk, dv = oracle.tree_attention_backward(nodes, q, k, v, do, scale, Hq, Hkv, kv_off=ko, q_off=qo)
    rng = np.random.default_rng(0)
    eps = 1e-5
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        for _ in range(25):
            idx = tuple(int(rng.integers(0, n)) for n in x.shape)
            xp, xm = x.copy(), x.copy()
            xp[idx] += eps
            xm[idx] -= eps
            args_p = {"q": (xp, k, v), "k": (q, xp, v), "v": (q, k, xp)}[name]
            args_m = {"q": (xm, k, v), "k": (q, xm, v), "v": (q, k, xm)}[name]
            fd = (loss(*args_p) - loss(*args_m)) / (2 * eps)
            assert abs(fd - g[idx]) <= 1e-7 + 1e-6 * abs(fd), (name, idx, fd, g[idx])


def _autograd_by_paths(nodes, q, k, v, do, scale, Hq, Hkv, ko, qo):
    """Gradients of sum(dO * O) where each segment's queries attend causally
    over their root-to-segment path (ancestor prefixes up to the fork, then
    the own segment), gathered from the packed K/V rows."""
    G = Hq // Hkv
    qt = torch.tensor(q, dtype=torch.float64, requires_grad=True)
    kt = torch.tensor(k, dtype=torch.float64, requires_grad=True)
    vt = torch.tensor(v, dtype=torch.float64, requires_grad=True)
    dot = torch.tensor(do, dtype=torch.float64)
    total = torch.zeros((), dtype=torch.float64)
    for s, (_, _, n, ql) in enumerate(nodes):
        if ql == 0:
            continue
        rows = []
        for t, f in reversed(ot.ancestors(nodes, s)):  # root first
            rows += [int(ko[t]) + j for j in range(f)]
        rows += [int(ko[s]) + j for j in range(n)]
        idx = torch.tensor(rows)
        qrows = torch.arange(int(qo[s]), int(qo[s]) + ql)
        m = len(rows)
        causal = torch.ones(ql, m, dtype=torch.bool).tril(diagonal=m - ql)
        for h in range(Hq):
            g = h // G
            qq = qt[qrows, h, :][None, None]
            kk = kt[idx, g, :][None, None]
            vv = vt[idx, g, :][None, None]
            o = F.scaled_dot_product_attention(qq, kk, vv, attn_mask=causal, scale=scale)[0, 0]
            total = total + (o * dot[qrows, h, :]).sum()
    total.backward()
    return qt.grad.numpy(), kt.grad.numpy(), vt.grad.numpy()


@pytest.mark.parametrize("Hq,Hkv", [(1, 1), (4, 2), (6, 2)])
def test_B2_autograd_through_paths(Hq, Hkv):
    nodes = _tiny_nodes()
    d, scale = 8, 0.29
    ko, qo, q, k, v, do = _problem(nodes, Hq, Hkv, d, 11 + Hq)
    got = oracle.tree_attention_backward(nodes, q, k, v, do, scale, Hq, Hkv, kv_off=ko, q_off=qo)
    ref = _autograd_by_paths(nodes, q, k, v, do, scale, Hq, Hkv, ko, qo)
    for a, b in zip(got, ref):
        np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-12)


def test_B2_random_deep_trees_with_partial_queries():
    """Depth up to 4, two pages, some segments with fewer queries than tokens."""
    for seed in range(8):
        nodes = [(a.parent, a.fork, a.length, a.q_len)
                 for a in syn.random_tree(seed, n_pages=2, max_depth=4, q_mode="some")]
        if sum(n[3] for n in nodes) == 0:
            continue
        ko, qo, q, k, v, do = _problem(nodes, 4, 2, 8, seed)
        got = oracle.tree_attention_backward(nodes, q, k, v, do, 0.31, 4, 2, kv_off=ko, q_off=qo)
        ref = _autograd_by_paths(nodes, q, k, v, do, 0.31, 4, 2, ko, qo)
        for a, b in zip(got, ref):
            np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-12)


def test_B3_gradient_invariants():
    nodes = ot.page_nodes([syn.Page(12, 12, 6, 6, (syn.Branch(2, 5, 5), syn.Branch(6, 4, 4), syn.Branch(6, 7, 7)))])
    Hq, Hkv, d = 6, 2, 16
    ko, qo, q, k, v, do = _problem(nodes, Hq, Hkv, d, 3)
    dq, dk, dv = oracle.tree_attention_backward(nodes, q, k, v, do, 0.25, Hq, Hkv, kv_off=ko, q_off=qo)
    G = Hq // Hkv
    for g in range(Hkv):
        np.testing.assert_allclose(dk[:, g, :].sum(axis=0), 0.0, atol=1e-11)
        np.testing.assert_allclose(dv[:, g, :].sum(axis=0), do[:, g * G:(g + 1) * G, :].sum(axis=(0, 1)),
                                   rtol=1e-12, atol=1e-11)


def test_B4_stored_output_form():
    nodes = _tiny_nodes()
    Hq, Hkv, d, scale = 4, 2, 8, 0.37
    ko, qo, q, k, v, do = _problem(nodes, Hq, Hkv, d, 21)
    O, _ = ot.tree_attention(nodes, q, k, v, scale, Hq, Hkv, kv_off=ko, q_off=qo)
    exact = oracle.tree_attention_backward(nodes, q, k, v, do, scale, Hq, Hkv, kv_off=ko, q_off=qo)
    stored = oracle.tree_attention_backward(nodes, q, k, v, do, scale, Hq, Hkv, kv_off=ko, q_off=qo, o=O)
    for a, b in zip(exact, stored):
        np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-12)
    # perturb one stored row: dQ of that row moves by -c * dD * (P k) (P k = O
    # computed with K in place of V), other rows' dQ stay
    row, h = 3, 1
    delta = _rand((d,), 77) * 1e-3
    O2 = O.copy()
    O2[row, h] += delta
    dq2, _, dv2 = oracle.tree_attention_backward(nodes, q, k, v, do, scale, Hq, Hkv, kv_off=ko, q_off=qo, o=O2)
    dD = float(do[row, h] @ delta)
    Pk, _ = ot.tree_attention(nodes, q, k, k, scale, Hq, Hkv, kv_off=ko, q_off=qo)
    want = exact[0].copy()
    want[row, h] -= scale * dD * Pk[row, h]
    np.testing.assert_allclose(dq2, want, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dv2, exact[2], rtol=1e-12, atol=1e-12)
