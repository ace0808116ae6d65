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
                max_chunk_keys=0, device="cuda", target_workgroups=0):
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
                       max_chunk_keys=max_chunk_keys, target_workgroups=target_workgroups)
    print(f"[case] decode T={T} nq={nq} blocks={nb} Hq={Hq} Hkv={Hkv} d={d} {dtype} seed={seed} "
          f"work={len(plan.export()['work'])}", flush=True)
    o, lse = pa.branch_decode(q, kc, vc, bt, plan)
    torch.cuda.synchronize()
    if not check:
        return o, lse, plan, (q, kc, vc, bt, ids)
    O_ref, LSE_ref = oracle.tree_attention_paged(nodes, q, kc, vc, ids, 1.0 / math.sqrt(d), Hq, Hkv, 16, rows=rows)
    errs = compare(f"decode seed={seed}", o, lse, O_ref, LSE_ref, dtype, rows=rows)
    return o, lse, plan, errs


# Backward tolerance.  Gradients have no unit scale (a prefix key's dK sums
# over every query below it), so the stated bf16 bounds (max 1.5e-2, mean
# 2e-3) are applied in units of the gradient's scale: for the max, the larger
# of the tensor's RMS and the RMS of the element's own row (a key seen by
# every query of a page sums thousands of terms, each carrying the half-ulp
# bf16 rounding of its P or dS operand, so its error grows with its own
# magnitude), plus one bf16 ulp of the element's value (2^-8 |g|: the output
# is rounded to nearest-even after fp32 accumulation); for the mean, the
# tensor's RMS.
BWD_TOL = (1.5e-2, 2e-3)
BWD_ULP = 2.0 ** -8


def backward_case(pages_or_nodes, Hq, Hkv, d, seed, device="cuda", check=True):
    """Packed forward then backward on seeded bf16 inputs, against the fp64
    backward oracle on the same values (dO drawn like the inputs)."""
    if len(pages_or_nodes) and isinstance(pages_or_nodes[0], syn.Page):
        segs = pa.segments_from_pages(pages_or_nodes, 0)
        nodes = od.page_nodes(pages_or_nodes)
    else:
        nodes = [tuple(n) if isinstance(n, tuple) else (n.parent, n.fork, n.length, n.q_len) for n in pages_or_nodes]
        segs = pa.segments_layout(nodes, 0)
    ref_kv, ref_q = od.canonical_layout(nodes, 0)
    T = int(sum(n[2] for n in nodes))
    nq = int(sum(n[3] for n in nodes))
    q = syn.draw_normal((nq, Hq, d), seed, 1, "bf16", device=device)
    k = syn.draw_normal((T, Hkv, d), seed, 2, "bf16", device=device)
    v = syn.draw_normal((T, Hkv, d), seed, 3, "bf16", device=device)
    do = syn.draw_normal((nq, Hq, d), seed, 4, "bf16", device=device)
    plan = pa.TreePlan(segs, Hq, Hkv, d, "bf16", 0, num_kv_rows=T, num_q_rows=nq)
    ex = plan.export()
    print(f"[case] backward T={T} nq={nq} Hq={Hq} Hkv={Hkv} d={d} seed={seed} work={len(ex['work'])} "
          f"bwd={len(ex['bwd'])}", flush=True)
    scale = 1.0 / math.sqrt(d)
    if not check:
        o, lse = pa.tree_attn_fwd(q, k, v, plan)
        return pa.tree_attn_bwd(q, k, v, o, lse, do, plan), plan
    # Both sides get the same stored forward output: the oracle's O rounded
    # to bf16 (what a bf16 forward stores) and its LSE in fp32; D = dO . O is
    # then formed from the same values on both sides.
    O_ref, LSE_ref = oracle.tree_attention(nodes, q, k, v, scale, Hq, Hkv, kv_off=ref_kv, q_off=ref_q)
    o = torch.tensor(O_ref, dtype=torch.float64).to(torch.bfloat16).to(device)
    lse = torch.tensor(LSE_ref, dtype=torch.float64).to(torch.float32).to(device)
    dq, dk, dv = pa.tree_attn_bwd(q, k, v, o, lse, do, plan)
    torch.cuda.synchronize()
    ref = oracle.tree_attention_backward(nodes, q, k, v, do, scale, Hq, Hkv, kv_off=ref_kv, q_off=ref_q, o=o)
    errs = {}
    for name, g, r in zip(("dq", "dk", "dv"), (dq, dk, dv), ref):
        x = g.detach().to("cpu", torch.float64).numpy()
        assert np.isfinite(x).all(), f"{name}: non-finite gradient"
        s = float(np.sqrt(np.mean(r * r))) if r.size else 1.0
        s = s if s > 0 else 1.0
        err = np.abs(x - r)
        s_el = np.maximum(s, np.sqrt(np.mean(r * r, axis=2, keepdims=True)))
        e_max = float(np.max(np.maximum(err - BWD_ULP * np.abs(r), 0.0) / s_el)) if r.size else 0.0
        e_mean = float(err.mean() / s) if r.size else 0.0
        errs[name] = (e_max, e_mean, s)
        print(f"  {name}: rms {s:.3e} (max-err - ulp)/scale {e_max:.3e} mean-err/rms {e_mean:.3e}", flush=True)
        assert e_max <= BWD_TOL[0], f"{name}: (max-abs - ulp)/scale {e_max:.3e} > {BWD_TOL[0]}"
        assert e_mean <= BWD_TOL[1], f"{name}: mean-abs/rms {e_mean:.3e} > {BWD_TOL[1]}"
    return errs, plan
