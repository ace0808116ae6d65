"""Shared helpers of the GPU parity tests: build a case from seeded inputs,
run it through the C ABI (via the thin binding) and through the oracle, and
compare with the tolerances of the hot path:

* fp32 outputs: max-abs error <= 1e-5 (O and LSE)
* bf16 outputs: max-abs error <= 1.5e-2 and mean-abs error <= 2e-3 (O and LSE)
"""
from __future__ import annotations

import math
from typing import List, Optional, Sequence

import numpy as np
import torch

import oracle
from oracle import dense as od
import padoc_synth as syn
import paper_2608_06146_amd as pa

TOL = {"f32": (1e-5, 1e-5), "bf16": (1.5e-2, 2e-3)}


def nodes_of(segs) -> List[tuple]:
    return [(int(s["parent"]), int(s["fork"]), int(s["len"]), int(s["q_len"])) for s in segs]


def compare(name, o_gpu, lse_gpu, O_ref, LSE_ref, dtype, rows=None):
    """Element-wise comparison against the oracle; returns (max, mean) errors."""
    o = o_gpu.detach().to("cpu", torch.float64).numpy()
    l = lse_gpu.detach().to("cpu", torch.float64).numpy()
    if rows is not None:
        rows = np.asarray(sorted(rows))
        o, l, O_ref, LSE_ref = o[rows], l[rows], O_ref[rows], LSE_ref[rows]
    assert np.isfinite(o).all(), f"{name}: non-finite output"
    assert np.isfinite(l).all(), f"{name}: non-finite LSE"
    eo = np.abs(o - O_ref)
    el = np.abs(l - LSE_ref)
    mx, mn = TOL[dtype]
    assert eo.max() <= mx, f"{name}: O max-abs {eo.max():.3e} > {mx}"
    assert el.max() <= mx, f"{name}: LSE max-abs {el.max():.3e} > {mx}"
    if dtype == "bf16":
        assert eo.mean() <= mn, f"{name}: O mean-abs {eo.mean():.3e} > {mn}"
        assert el.mean() <= mn, f"{name}: LSE mean-abs {el.mean():.3e} > {mn}"
    return float(eo.max()), float(eo.mean()), float(el.max())


def forward_case(pages_or_nodes, Hq, Hkv, d, dtype, seed, prescale=False, kv_off=None, q_off=None,
                 kv_rows=None, check=True, rows=None, device="cuda"):
    """Packed forward on seeded inputs.  The tree comes from pages (paper
    form) or generic nodes; the library lays it out (canonical packed order)
    unless the test passes explicit offsets, and the oracle uses its own
    layout, so a layout slip on either side shows up as a mismatch."""
    if len(pages_or_nodes) and isinstance(pages_or_nodes[0], syn.Page):
        segs = pa.segments_from_pages(pages_or_nodes, 0)
        nodes = od.page_nodes(pages_or_nodes)
    else:
        nodes = [tuple(n) if isinstance(n, tuple) else (n.parent, n.fork, n.length, n.q_len) for n in pages_or_nodes]
        segs = pa.segments_layout(nodes, 0)
    if kv_off is not None:
        segs["kv_off"] = kv_off
        segs["q_off"] = q_off
        ref_kv, ref_q = np.asarray(kv_off), np.asarray(q_off)
    else:
        ref_kv, ref_q = od.canonical_layout(nodes, 0)
    T = int(kv_rows if kv_rows is not None else sum(n[2] for n in nodes))
    nq = int(max([int(a + n[3]) for a, n in zip(ref_q, nodes)] + [0]))
    ps = (1.0 / math.sqrt(d)) if prescale else None
    q = syn.draw_normal((nq, Hq, d), seed, 1, dtype, device=device, prescale=ps)
    k = syn.draw_normal((T, Hkv, d), seed, 2, dtype, device=device, prescale=ps)
    v = syn.draw_normal((T, Hkv, d), seed, 3, dtype, device=device, prescale=ps)
    plan = pa.TreePlan(segs, Hq, Hkv, d, dtype, 0, num_kv_rows=T, num_q_rows=nq)
    print(f"[case] forward T={T} nq={nq} Hq={Hq} Hkv={Hkv} d={d} {dtype} seed={seed} work={len(plan.export()['work'])}",
          flush=True)
    o, lse = pa.tree_attn_fwd(q, k, v, plan)
    torch.cuda.synchronize()
    if not check:
        return o, lse, plan, (q, k, v)
    O_ref, LSE_ref = oracle.tree_attention(nodes, q, k, v, 1.0 / math.sqrt(d), Hq, Hkv,
                                           kv_off=ref_kv, q_off=ref_q, rows=rows)
    errs = compare(f"forward seed={seed}", o, lse, O_ref, LSE_ref, dtype, rows=rows)
    return o, lse, plan, errs


def fill_pool(nodes, k_packed, v_packed, n_pool, seed, device="cuda", sentinel=float("nan")):
    """Paged caches (K chunk-major [n_pool, Hkv, d/8, 16, 8], V d-major
    [n_pool, Hkv, d, 16]) holding the packed K/V at the block ids drawn by the
    generator; every other slot holds `sentinel`."""
    nb = int(sum(-(-n[2] // 16) for n in nodes))
    ids = syn.draw_block_ids(nb, n_pool, seed)
    Hkv, d = k_packed.shape[1], k_packed.shape[2]
    kc = torch.full((n_pool, Hkv, d // 8, 16, 8), sentinel, dtype=k_packed.dtype, device=device)
    vc = torch.full((n_pool, Hkv, d, 16), sentinel, dtype=v_packed.dtype, device=device)
    blk, slot = od.paged_slots(nodes, ids, 16)
    bi = torch.as_tensor(blk, device=device)
    si = torch.as_tensor(slot, device=device)
    ci = torch.as_tensor(od.chunk_slot(slot), device=device)
    kc[bi, :, :, ci, :] = k_packed.to(device).reshape(len(slot), Hkv, d // 8, 8)
    vc[bi, :, :, si] = v_packed.to(device)
    return kc, vc, ids


def decode_case(pages_or_nodes, Hq, Hkv, d, dtype, seed, pool_extra=7, check=True, rows=None,
                max_chunk_keys=0, device="cuda"):
    """Decode step over a paged cache: structure from pages (paper form) or
    generic nodes, canonical paged layout."""
    if len(pages_or_nodes) and isinstance(pages_or_nodes[0], syn.Page):
        segs = pa.segments_from_pages(pages_or_nodes, 16)
        nodes = od.page_nodes(pages_or_nodes)
    else:
        nodes = [tuple(n) if isinstance(n, tuple) else (n.parent, n.fork, n.length, n.q_len) for n in pages_or_nodes]
        segs = pa.segments_layout(nodes, 16)
    T = int(sum(n[2] for n in nodes))
    nq = int(sum(n[3] for n in nodes))
    nb = int(sum(-(-n[2] // 16) for n in nodes))
    n_pool = nb + pool_extra
    q = syn.draw_normal((nq, Hq, d), seed, 1, dtype, device=device)
    k = syn.draw_normal((T, Hkv, d), seed, 2, dtype, device=device)
    v = syn.draw_normal((T, Hkv, d), seed, 3, dtype, device=device)
    kc, vc, ids = fill_pool(nodes, k, v, n_pool, seed, device=device)
    bt = torch.as_tensor(ids, device=device)
    plan = pa.TreePlan(segs, Hq, Hkv, d, dtype, 16, num_kv_rows=n_pool, num_q_rows=nq, block_table_host=ids,
                       max_chunk_keys=max_chunk_keys)
    print(f"[case] decode T={T} nq={nq} blocks={nb} Hq={Hq} Hkv={Hkv} d={d} {dtype} seed={seed} "
          f"work={len(plan.export()['work'])}", flush=True)
    o, lse = pa.branch_decode(q, kc, vc, bt, plan)
    torch.cuda.synchronize()
    if not check:
        return o, lse, plan, (q, kc, vc, bt, ids)
    O_ref, LSE_ref = oracle.tree_attention_paged(nodes, q, kc, vc, ids, 1.0 / math.sqrt(d), Hq, Hkv, 16, rows=rows)
    errs = compare(f"decode seed={seed}", o, lse, O_ref, LSE_ref, dtype, rows=rows)
    return o, lse, plan, errs
