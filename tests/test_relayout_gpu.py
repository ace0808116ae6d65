"""Row-layout paged caches ([num_blocks, Hkv, 16, d], each token's row
contiguous) rewritten into the library's paged layouts by
padoc_cache_from_rows: every element lands where the oracle's reader of the
library layout (chunk-major K with bits 2 and 3 of the slot exchanged,
d-major V) looks for it, bit-exactly, and a decode step over the rewritten
cache equals the oracle's attention over the row-layout cache.  Errors are
raised before anything is enqueued."""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import dense as od
import padoc_synth as syn
import paper_2608_06146_amd as pa
from _cases import compare

pytestmark = pytest.mark.gpu


def _rows(nb, hkv, d, dtype, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    x = torch.randn((nb, hkv, 16, d), generator=g, device="cuda", dtype=torch.float32)
    return x.to(torch.bfloat16 if dtype == "bf16" else torch.float32)


@pytest.mark.parametrize("dtype,d,hkv", [("bf16", 128, 2), ("bf16", 64, 4), ("f32", 64, 1), ("f32", 128, 3)])
def test_cache_from_rows_layout(dtype, d, hkv):
    nb = 37
    kr, vr = _rows(nb, hkv, d, dtype, 1), _rows(nb, hkv, d, dtype, 2)
    print(f"[case] relayout {dtype} d={d} Hkv={hkv} blocks={nb}", flush=True)
    kc, vc = pa.cache_from_rows(kr, vr)
    torch.cuda.synchronize()
    K, V = kr.cpu().to(torch.float64).numpy(), vr.cpu().to(torch.float64).numpy()
    KC, VC = kc.cpu().to(torch.float64).numpy(), vc.cpu().to(torch.float64).numpy()
    t = np.arange(16)
    # the library layouts as the oracle reads them
    got_k = KC[:, :, :, od.chunk_slot(t), :]                      # [nb, hkv, d/8, 16, 8]
    got_k = np.moveaxis(got_k, 3, 2).reshape(nb, hkv, 16, d)     # [nb, hkv, 16 slots, d]
    got_v = np.moveaxis(VC, 3, 2)                                 # [nb, hkv, 16, d]
    assert np.array_equal(got_k, K)
    assert np.array_equal(got_v, V)


def test_cache_from_rows_decode_matches_oracle():
    """Decode on the rewritten caches against the oracle's attention over the
    row-layout caches (gathered by the oracle's own row-layout reader)."""
    rng = np.random.default_rng(3)
    S = 96
    f = np.sort(rng.integers(1, S, size=6))
    L = rng.integers(5, 90, size=6)
    pages = [syn.Page(300, 0, S, 1, tuple(syn.Branch(int(a), int(b), 1) for a, b in zip(f, L)))]
    nodes = od.page_nodes(pages)
    segs = pa.segments_from_pages(pages, 16)
    Hq, Hkv, d = 16, 2, 128
    nb = int(sum(-(-n[2] // 16) for n in nodes))
    n_pool = nb + 9
    ids = syn.draw_block_ids(nb, n_pool, 5)
    kr, vr = _rows(n_pool, Hkv, d, "bf16", 7), _rows(n_pool, Hkv, d, "bf16", 8)
    nq = int(sum(n[3] for n in nodes))
    q = syn.draw_normal((nq, Hq, d), 4, 1, "bf16", device="cuda")
    kc, vc = pa.cache_from_rows(kr, vr)
    plan = pa.TreePlan(segs, Hq, Hkv, d, "bf16", 16, num_kv_rows=n_pool, num_q_rows=nq, block_table_host=ids)
    o, lse = pa.branch_decode(q, kc, vc, torch.as_tensor(ids, device="cuda"), plan)
    torch.cuda.synchronize()
    K = od.gather_paged(nodes, kr, ids, 16, layout="rows")
    V = od.gather_paged(nodes, vr, ids, 16, layout="rows")
    kv_off, q_off = od.canonical_layout(nodes, 0)
    O, Lse = oracle.tree_attention(nodes, q, K, V, 1.0 / math.sqrt(d), Hq, Hkv, kv_off=kv_off, q_off=q_off)
    compare("relayout decode", o, lse, O, Lse, "bf16")


def test_cache_from_rows_errors():
    kr = torch.zeros((2, 1, 16, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ValueError):
        pa.cache_from_rows(kr, torch.zeros((2, 1, 16, 64), dtype=torch.float32, device="cuda"))
    with pytest.raises(ValueError):
        pa.cache_from_rows(kr[:, :, :8].contiguous(), kr[:, :, :8].contiguous())
    from paper_2608_06146_amd import _lib
    import ctypes as C
    lib = _lib.lib()
    p = C.c_void_p(kr.data_ptr())
    assert lib.padoc_cache_from_rows(p, p, p, p, 2, 1, 64, _lib.BF16, None) == _lib.ERR_ARG     # in place
    assert lib.padoc_cache_from_rows(p, p, None, None, 2, 1, 96, _lib.BF16, None) == _lib.ERR_SHAPE
    assert lib.padoc_cache_from_rows(None, None, None, None, 0, 1, 64, _lib.BF16, None) == _lib.OK  # nothing to do
