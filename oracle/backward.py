"""Plain fp64 CPU oracle for the backward of packed tree attention.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  The product library
never calls it and shares no code with it.

What it computes
----------------
The paper trains with its tree-varlen attention backend (App. C, tree-varlen
relation; Table of backend step times), so training needs the gradient of the
packed tree forward (App. E, the Attn equation with the ancestor mask A_M) with
respect to Q, K and V.  The gradient of masked softmax attention has a plain
closed form, written out here per query row i over its visible keys j
(scale ``c``, upstream gradient ``dO``):

* ``P_ij = exp(c q_i.k_j - LSE_i)`` (the forward's probabilities),
* ``dV_j = sum_i P_ij dO_i``,
* ``dP_ij = dO_i . v_j``,
* ``D_i = sum_j P_ij dP_ij`` (= ``dO_i . O_i``),
* ``dS_ij = P_ij (dP_ij - D_i)``,
* ``dQ_i = c sum_j dS_ij k_j``, ``dK_j = c sum_i dS_ij q_i``.

Masked pairs enter no sum.  ``D_i`` equals ``dO_i . O_i``; a backward that
receives the forward's stored output (rounded to the forward's dtype)
computes D from that stored O, so both functions take an optional ``o``: when
given, ``D_i = dO_i . o_i`` (fp64 sum of the given values), else the exact
``sum_j P_ij dP_ij``.  With grouped heads (query head h reads KV head
``h // G``), dK and dV of a KV head sum over its G query heads; a key shared by
several segments (a page prefix, a layout stream) sums over every query of
every descendant that sees it.  Everything is fp64 (bf16 inputs are exact in
fp64).
"""
from __future__ import annotations

from typing import Optional

import numpy as np

from .dense import _as_nodes, _f64, ancestors, canonical_layout, masked_attention, page_of

__all__ = ["masked_attention_backward", "tree_attention_backward"]


def masked_attention_backward(q, k, v, mask, scale: float, dout, o=None):
    """Gradient of one head of masked softmax attention, fp64.

    ``q [nq, d]``, ``k, v [nk, d]``, ``mask [nq, nk]`` (True = visible),
    ``dout [nq, dv]``, optional stored output ``o [nq, dv]`` for D.  Returns
    ``(dq, dk, dv)`` by the closed form in the module docstring."""
    q, k, v, dout = _f64(q), _f64(k), _f64(v), _f64(dout)
    _, _, p = masked_attention(q, k, v, mask, scale, return_probs=True)
    dv = p.T @ dout
    dp = dout @ v.T
    if o is None:
        dd = np.sum(p * dp, axis=1, keepdims=True)
    else:
        dd = np.sum(dout * _f64(o), axis=1, keepdims=True)
    ds = np.where(mask, p * (dp - dd), 0.0)
    dq = scale * (ds @ k)
    dk = scale * (ds.T @ q)
    return dq, dk, dv


def tree_attention_backward(nodes, q, k, v, dout, scale: float, num_heads_q: int, num_heads_kv: int,
                            kv_off=None, q_off=None, o=None):
    """Backward of packed tree attention by definition.

    Layouts as in :func:`oracle.dense.tree_attention`: ``q, dout [n_q, Hq, d]``,
    ``k, v [T, Hkv, d]``.  Returns fp64 ``(dQ [n_q, Hq, d], dK [T, Hkv, d],
    dV [T, Hkv, d])``; K/V rows no query sees get zero gradient.  ``o [n_q,
    Hq, d]``, when given, is the stored forward output D is computed from."""
    nodes = _as_nodes(nodes)
    if num_heads_q % num_heads_kv:
        raise ValueError("Hq must be a multiple of Hkv")
    G = num_heads_q // num_heads_kv
    q64, k64, v64, do64 = _f64(q), _f64(k), _f64(v), _f64(dout)
    o64 = None if o is None else _f64(o)
    if kv_off is None or q_off is None:
        ko, qo = canonical_layout(nodes, 0)
        kv_off = ko if kv_off is None else kv_off
        q_off = qo if q_off is None else q_off
    dQ = np.zeros_like(q64)
    dK = np.zeros_like(k64)
    dV = np.zeros_like(v64)
    roots = page_of(nodes)
    for root in sorted(set(int(r) for r in roots)):
        segs = [i for i in range(len(nodes)) if roots[i] == root]
        starts, total = {}, 0
        for i in segs:
            starts[i] = total
            total += nodes[i][2]
        kv_rows = np.concatenate([kv_off[i] + np.arange(nodes[i][2], dtype=np.int64) for i in segs]) \
            if total else np.zeros(0, np.int64)
        qs, qp, qr = [], [], []
        for s in segs:
            n, ql = nodes[s][2], nodes[s][3]
            for p in range(n - ql, n):
                qs.append(s)
                qp.append(p)
                qr.append(int(q_off[s] + p - (n - ql)))
        if not qr:
            continue
        qr = np.array(qr)
        mask = np.zeros((len(qr), total), dtype=bool)
        for a, (s, p) in enumerate(zip(qs, qp)):
            mask[a, starts[s]: starts[s] + p + 1] = True
            for t, f in ancestors(nodes, s):
                mask[a, starts[t]: starts[t] + f] = True
        for h in range(num_heads_q):
            g = h // G
            dq, dk, dv = masked_attention_backward(q64[qr, h, :], k64[kv_rows, g, :], v64[kv_rows, g, :], mask,
                                                   scale, do64[qr, h, :],
                                                   None if o64 is None else o64[qr, h, :])
            dQ[qr, h, :] = dq
            dK[kv_rows, g, :] += dk
            dV[kv_rows, g, :] += dv
    return dQ, dK, dV
