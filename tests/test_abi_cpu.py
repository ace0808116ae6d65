"""C-ABI tests that need no GPU: exports, tree construction and schedules
held bit-exactly to the oracle's independent derivation, and error paths.

The schedule checks follow the visibility rule (Sec. 3.2 ancestor sets, App.
C tree-varlen relation): every visible (query, key) pair must be covered by
exactly one scheduled range of exactly one work item per KV head (forward) or
one combined partial (decode); no scheduled key tile may be fully masked; a
tile classified "full" must be fully visible to every token of its item.
"""
import ctypes as C
import os
import re
import threading

import numpy as np
import pytest

from oracle import dense as od
import padoc_synth as syn
import paper_2608_06146_amd as pa
from paper_2608_06146_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_symbol():
    hdr = open(os.path.join(ROOT, "include", "padoc_attn.h")).read()
    names = set(re.findall(r"^\s*(?:padoc_status|void|const char\*)\s+(padoc_\w+)\s*\(", hdr, re.M))
    assert len(names) >= 11, names
    L = _lib.lib()
    for n in sorted(names):
        assert hasattr(L, n), f"{n} declared in padoc_attn.h but not exported"
    assert set(_lib.EXPORTED) == names
    assert pa.version().startswith("padoc_attn")


def test_struct_layouts_match_header():
    assert C.sizeof(_lib.Segment) == 32 and pa.SEGMENT_DTYPE.itemsize == 32
    assert _lib.WORK_DTYPE.itemsize == 48 and _lib.RANGE_DTYPE.itemsize == 32


# ---------------------------------------------------------------- tree -> segments

@pytest.mark.parametrize("name", list(syn.CONFIGS))
@pytest.mark.parametrize("block", [0, 16])
def test_segments_from_pages_match_oracle(name, block):
    wl = syn.make_workload(name)
    segs = pa.segments_from_pages(wl.pages, block)
    nodes = od.page_nodes(wl.pages)
    kv, q = od.canonical_layout(nodes, block)
    assert len(segs) == len(nodes)
    for s, n, a, b in zip(segs, nodes, kv, q):
        assert (int(s["parent"]), int(s["fork"]), int(s["len"]), int(s["q_len"])) == n
        assert int(s["kv_off"]) == a and int(s["q_off"]) == b


def test_segments_layout_matches_oracle_random_trees():
    for seed in range(40):
        nodes = [(n.parent, n.fork, n.length, n.q_len) for n in syn.random_tree(seed, q_mode="some")]
        for block in (0, 16):
            segs = pa.segments_layout(nodes, block)
            kv, q = od.canonical_layout(nodes, block)
            np.testing.assert_array_equal(segs["kv_off"], kv)
            np.testing.assert_array_equal(segs["q_off"], q)


# ---------------------------------------------------------------- schedules

def _token_of_row(nodes, q_off):
    out = {}
    for s, (_, _, n, ql) in enumerate(nodes):
        for i in range(ql):
            out[int(q_off[s] + i)] = (s, n - ql + i)
    return out


def _visible_keys(nodes, s, p):
    return {(t, j) for t, c in od.visible_counts(nodes, s, p).items() for j in range(c)}


def _item_coverage(ex, w, G):
    """{token index i -> multiset of (segment, key)} covered by work item w,
    plus the tile classes checked against the item's own limits."""
    toks = ex["toks"][w["tok_begin"]: w["tok_begin"] + w["ntok"]]
    cover = {i: [] for i in range(w["ntok"])}
    for r in range(w["rng_begin"], w["rng_begin"] + w["rng_count"]):
        R = ex["ranges"][r]
        lims = (np.full(w["ntok"], R["n_keys"]) if R["lim_off"] < 0
                else ex["lims"][R["lim_off"]: R["lim_off"] + w["ntok"]])
        assert lims.max() == R["n_keys"] and lims.min() == R["min_lim"]
        for i in range(w["ntok"]):
            cover[i] += [(int(R["seg"]), int(R["key_begin"]) + j) for j in range(int(lims[i]))]
        KT = ex["tile_keys"]
        nkt = -(-int(R["n_keys"]) // KT)
        cls = ex["tile_class"][ex["tile_class_off"][r]: ex["tile_class_off"][r] + nkt]
        for kt in range(nkt):
            seen = np.clip(lims - kt * KT, 0, KT)
            assert seen.max() > 0, "scheduled key tile is fully masked"
            full = bool((seen == KT).all())
            assert cls[kt] == (1 if full else 2)
    return toks, cover


def _check_forward(segs, G, Hkv):
    nodes = [(int(s["parent"]), int(s["fork"]), int(s["len"]), int(s["q_len"])) for s in segs]
    plan = pa.TreePlan(segs, G * Hkv, Hkv, 128, "bf16", 0, num_kv_rows=int(sum(n[2] for n in nodes)))
    ex = plan.export()
    assert ex["kind"] == 0
    row_tok = _token_of_row(nodes, segs["q_off"])
    seen = {g: {} for g in range(Hkv)}
    for w in ex["work"]:
        assert w["ntok"] * G <= ex["tile_cols"] and w["col0"] == 0 and w["ncol"] == w["ntok"] * G
        toks, cover = _item_coverage(ex, w, G)
        for i, row in enumerate(toks):
            assert int(row) not in seen[int(w["kvh"])], "query row scheduled twice for one KV head"
            seen[int(w["kvh"])][int(row)] = True
            s, p = row_tok[int(row)]
            assert len(cover[i]) == len(set(cover[i])), "a key is covered twice"
            assert set(cover[i]) == _visible_keys(nodes, s, p)
    for g in range(Hkv):
        assert set(seen[g]) == set(row_tok), "some query row is not scheduled"
    # work items are ordered costliest first
    assert (np.diff(ex["work"]["cost"]) <= 0).all()


def test_forward_schedule_tiny_page():
    wl = syn.make_workload("tiny_fp32_forward")
    _check_forward(pa.segments_from_pages(wl.pages, 0), 4, 1)


@pytest.mark.parametrize("G,Hkv", [(1, 1), (4, 1), (8, 2), (7, 4)])
def test_forward_schedule_random_trees(G, Hkv):
    for seed in range(8):
        nodes = [(n.parent, n.fork, n.length, n.q_len)
                 for n in syn.random_tree(seed, max_len=90, q_mode="some", max_nodes=16)]
        _check_forward(pa.segments_layout(nodes, 0), G, Hkv)


def test_forward_schedule_scaled_pages():
    rng = np.random.default_rng(3)
    pages = []
    for _ in range(2):
        P, S, N = int(rng.integers(100, 700)), int(rng.integers(20, 150)), int(rng.integers(3, 30))
        f = np.sort(rng.integers(1, S + 1, N))
        L = np.clip(np.rint(rng.lognormal(np.log(20), 0.5, N)), 4, 100).astype(int)
        pages.append(syn.Page(P, P, S, S, tuple(syn.Branch(int(a), int(b), int(b)) for a, b in zip(f, L))))
    _check_forward(pa.segments_from_pages(pages, 0), 8, 2)


def _check_decode(segs, G, Hkv, chunk=0, read_once=False):
    nodes = [(int(s["parent"]), int(s["fork"]), int(s["len"]), int(s["q_len"])) for s in segs]
    nb = int(sum(-(-n[2] // 16) for n in nodes))
    plan = pa.TreePlan(segs, G * Hkv, Hkv, 128, "bf16", 16, num_kv_rows=nb, block_table_len=nb,
                       max_chunk_keys=chunk)
    ex = plan.export()
    assert ex["kind"] == 1
    row_tok = _token_of_row(nodes, segs["q_off"])
    slot_cover = {}
    cols_of = {}
    for idx, w in enumerate(ex["work"]):
        width = 256 if idx < ex["n_work_shared"] else 16
        assert 0 < w["ncol"] <= width and w["col0"] % width == 0
        assert w["col0"] + w["ncol"] <= w["ntok"] * G
        cols_of.setdefault(int(w["out_base"]), []).extend(range(w["col0"], w["col0"] + w["ncol"]))
        toks, cover = _item_coverage(ex, w, G)
        if idx < ex["n_work_shared"]:  # a tile item stages the ids of at most 128 64-key tiles
            rr = ex["ranges"][w["rng_begin"]: w["rng_begin"] + w["rng_count"]]
            assert sum(-(-int(n) // 64) for n in rr["n_keys"]) <= 128
        for r in range(w["rng_begin"], w["rng_begin"] + w["rng_count"]):
            R = ex["ranges"][r]
            assert R["key_begin"] % 16 == 0
            assert R["kv_start"] == segs["kv_off"][R["seg"]] + R["key_begin"] // 16
            if chunk:
                assert R["n_keys"] <= chunk
        for i in range(w["ntok"]):
            slot_cover[int(w["out_base"]) + i * G] = (int(toks[i]), int(w["kvh"]), cover[i])
        dr = w["direct"]
        if dr[0] >= 0:  # a private item carrying its one range and its Q row
            R = ex["ranges"][w["rng_begin"]]
            assert idx >= ex["n_work_shared"] and w["rng_count"] == 1 and w["ntok"] == 1
            assert (dr[0], dr[1]) == (R["kv_start"], R["n_keys"]) and R["lim_off"] < 0
            assert dr[2] == ex["toks"][w["tok_begin"]]
        else:
            assert (dr[0], dr[1], dr[2]) == (-1, 0, 0)
    for base, cols in cols_of.items():
        assert sorted(cols) == list(range(len(cols))), "task columns not covered exactly once"
    n_q = int(sum(n[3] for n in nodes))
    assert len(ex["comb_ptr"]) == n_q * Hkv + 1
    for row, (s, p) in row_tok.items():
        for g in range(Hkv):
            ents = ex["comb_slot"][ex["comb_ptr"][row * Hkv + g]: ex["comb_ptr"][row * Hkv + g + 1]]
            keys = []
            for e in ents:
                r2, g2, cov = slot_cover[int(e)]
                assert r2 == row and g2 == g and len(cov) > 0
                keys += cov
            assert len(keys) == len(set(keys)), "a key is combined twice"
            assert set(keys) == _visible_keys(nodes, s, p)
    # the combine kernel visits exactly the rows that have entries (every
    # query row sees at least its own token)
    nonempty = {rk for rk in range(n_q * Hkv) if ex["comb_ptr"][rk + 1] > ex["comb_ptr"][rk]}
    assert nonempty == set(range(n_q * Hkv))
    assert list(ex["comb_rows"]) == sorted(nonempty)
    # slots the combine does not read belong to tokens that see no key there
    used = set(int(e) for e in ex["comb_slot"])
    for slot, (_, _, cov) in slot_cover.items():
        assert (slot in used) == (len(cov) > 0)
    if read_once:
        # every key is streamed by exactly one task per KV head (siblings
        # share the task's tiles)
        owner = {}
        for i, w in enumerate(ex["work"]):
            for r in range(w["rng_begin"], w["rng_begin"] + w["rng_count"]):
                R = ex["ranges"][r]
                for j in range(int(R["n_keys"])):
                    key = (int(w["kvh"]), int(R["seg"]), int(R["key_begin"]) + j)
                    assert owner.setdefault(key, int(w["out_base"])) == int(w["out_base"])
    return ex


@pytest.mark.parametrize("chunk", [0, 64, 128, 320])
def test_decode_schedule_random_trees(chunk):
    for seed in range(8):
        nodes = [(n.parent, n.fork, n.length, n.q_len)
                 for n in syn.random_tree(seed, max_len=150, q_mode="tail", max_nodes=16)]
        if sum(n[3] for n in nodes) == 0:
            continue
        _check_decode(pa.segments_layout(nodes, 16), 8, 2, chunk)


def test_decode_schedule_single_page_workload():
    wl = syn.make_workload("single_page_decode")
    _check_decode(pa.segments_from_pages(wl.pages, 16), 8, 2, read_once=True)
    _check_decode(pa.segments_from_pages(wl.pages, 16), 8, 2, chunk=128, read_once=True)


def test_decode_schedule_mixed_step_structure():
    """Scaled-down mixed step (q_len 1 and 8 streams, G = 7)."""
    br = tuple([syn.Branch(f, 40 + 3 * f, 1) for f in range(1, 40, 3)] + [syn.Branch(f, 8, 8) for f in (40, 41, 45)])
    pages = [syn.Page(500, 0, 50, 1, br)]
    _check_decode(pa.segments_from_pages(pages, 16), 7, 4)


def test_concurrent_decode_read_once():
    """64 pages x 24 branches: every cached key is streamed by exactly one
    work item per KV head (the page's 25 streams share one 200-column tile
    item for the prefix and stream), and every cached key is streamed."""
    wl = syn.make_workload("concurrent_decode_64pages")
    segs = pa.segments_from_pages(wl.pages, 16)
    nb = int(sum(-(-int(s["len"]) // 16) for s in segs))
    plan = pa.TreePlan(segs, 16, 2, 128, "bf16", 16, num_kv_rows=nb, block_table_len=nb)
    ex = plan.export()
    for g in range(2):
        owner = [np.full(int(sg["len"]), -1, dtype=np.int64) for sg in segs]
        for i, w in enumerate(ex["work"]):
            if w["kvh"] != g:
                continue
            for r in range(w["rng_begin"], w["rng_begin"] + w["rng_count"]):
                R = ex["ranges"][r]
                o = owner[int(R["seg"])][int(R["key_begin"]): int(R["key_begin"]) + int(R["n_keys"])]
                assert ((o == -1) | (o == i)).all(), "a key is streamed by two work items"
                o[:] = i
        assert all((o >= 0).all() for o in owner), "a cached key is never streamed"


# ---------------------------------------------------------------- errors

def _desc(segs, **kw):
    args = dict(num_heads_q=4, num_heads_kv=1, head_dim=64, dtype="bf16", block_size=0,
                num_kv_rows=int(sum(int(s["len"]) for s in segs)))
    args.update(kw)
    return args


def _err(segs, **kw):
    with pytest.raises(pa.PadocError) as e:
        pa.TreePlan(segs, **_desc(segs, **kw))
    return e.value.status


def _segs(rows):
    a = np.zeros(len(rows), dtype=pa.SEGMENT_DTYPE)
    for i, r in enumerate(rows):
        a[i] = r
    return a


def test_plan_errors():
    good = _segs([(-1, 0, 10, 10, 0, 0), (0, 10, 5, 5, 10, 10)])
    pa.TreePlan(good, **_desc(good))
    assert _err(_segs([(-1, 0, 10, 10, 0, 0), (1, 0, 5, 5, 10, 10)])) == _lib.ERR_TREE      # parent >= own
    assert _err(_segs([(-1, 0, 10, 10, 0, 0), (0, 11, 5, 5, 10, 10)])) == _lib.ERR_TREE     # fork > len(parent)
    assert _err(_segs([(-1, 0, 10, 10, 0, 0), (0, -1, 5, 5, 10, 10)])) == _lib.ERR_TREE     # negative fork
    assert _err(_segs([(-1, 3, 10, 10, 0, 0)])) == _lib.ERR_TREE                            # root with fork
    assert _err(_segs([(-1, 0, 10, 11, 0, 0)])) == _lib.ERR_TREE                            # q_len > len
    assert _err(good, num_heads_q=6, num_heads_kv=4) == _lib.ERR_SHAPE                      # Hq % Hkv
    assert _err(good, head_dim=96) == _lib.ERR_SHAPE
    assert _err(good, num_heads_q=130, num_heads_kv=2) == _lib.ERR_SHAPE                    # G > 64
    assert _err(good, num_kv_rows=14) == _lib.ERR_BOUNDS                                    # K/V rows
    assert _err(good, num_q_rows=12) == _lib.ERR_BOUNDS                                     # Q rows
    assert _err(_segs([(-1, 0, 10, 10, 0, 0), (0, 10, 5, 5, 10, 8)])) == _lib.ERR_BOUNDS    # overlapping q rows
    assert _err(good, softmax_scale=-1.0) == _lib.ERR_ARG
    assert _err(good, softmax_scale=float("inf")) == _lib.ERR_ARG
    assert _err(good, block_size=8) == _lib.ERR_ARG
    assert _err(good, max_chunk_keys=100) == _lib.ERR_ARG
    assert _err(good, max_chunk_keys=8192 + 64) == _lib.ERR_ARG                            # chunk > 8192 keys
    pa.TreePlan(good, **_desc(good, max_chunk_keys=8192))
    # paged: block table too short, block id outside the pool
    pg = _segs([(-1, 0, 20, 0, 0, 0), (0, 20, 5, 1, 2, 0)])
    pa.TreePlan(pg, **_desc(pg, block_size=16, num_kv_rows=8, block_table_host=np.arange(3)))
    assert _err(pg, block_size=16, num_kv_rows=8, block_table_len=2) == _lib.ERR_BOUNDS
    assert _err(pg, block_size=16, num_kv_rows=8, block_table_host=np.array([0, 1, 8])) == _lib.ERR_BOUNDS
    assert _err(pg, block_size=16, num_kv_rows=8, block_table_host=np.array([0, -1, 2])) == _lib.ERR_BOUNDS


def test_plan_error_dtype_and_null_pointers():
    L = _lib.lib()
    h = C.c_void_p()
    assert L.padoc_plan_create(None, C.byref(h)) == _lib.ERR_ARG
    assert "desc is null" in L.padoc_last_error().decode()
    seg = _segs([(-1, 0, 4, 4, 0, 0)])
    d = _lib.TreeDesc(1, seg.ctypes.data, 4, 1, 64, 0.125, 7, 0, 4, 4, None, 0, 0, 0)
    assert L.padoc_plan_create(C.byref(d), C.byref(h)) == _lib.ERR_DTYPE
    d = _lib.TreeDesc(1, None, 4, 1, 64, 0.125, 1, 0, 4, 4, None, 0, 0, 0)
    assert L.padoc_plan_create(C.byref(d), C.byref(h)) == _lib.ERR_ARG
    n = C.c_int32()
    assert L.padoc_tree_from_pages(None, 1, 0, None, 0, C.byref(n)) == _lib.ERR_ARG


def test_launch_errors_return_before_any_device_call():
    """Argument and workspace errors are reported before anything is
    enqueued (these calls never reach HIP, so they run without a GPU)."""
    L = _lib.lib()
    segs = _segs([(-1, 0, 10, 10, 0, 0)])
    plan = pa.TreePlan(segs, **_desc(segs))
    fake = C.c_void_p(1 << 20)
    ws_ok = plan.workspace_bytes
    assert L.padoc_tree_attn_fwd(plan.handle, fake, fake, fake, fake, fake, fake, ws_ok - 1, None) == _lib.ERR_WORKSPACE
    assert "smaller" in L.padoc_last_error().decode()
    assert L.padoc_tree_attn_fwd(plan.handle, None, fake, fake, fake, fake, fake, ws_ok, None) == _lib.ERR_ARG
    assert L.padoc_tree_attn_fwd(plan.handle, fake, fake, fake, fake, fake, None, ws_ok, None) == _lib.ERR_WORKSPACE
    assert L.padoc_tree_attn_fwd(plan.handle, fake, fake, fake, fake, fake, C.c_void_p((1 << 20) + 16), ws_ok,
                                 None) == _lib.ERR_WORKSPACE  # misaligned workspace
    assert L.padoc_branch_decode(plan.handle, fake, fake, fake, fake, fake, fake, fake, ws_ok, None) == _lib.ERR_MODE
    assert L.padoc_tree_attn_fwd(None, fake, fake, fake, fake, fake, fake, ws_ok, None) == _lib.ERR_ARG
    pg = _segs([(-1, 0, 20, 1, 0, 0)])
    dplan = pa.TreePlan(pg, **_desc(pg, block_size=16, num_kv_rows=4, block_table_len=2))
    wsd = dplan.workspace_bytes
    assert L.padoc_tree_attn_fwd(dplan.handle, fake, fake, fake, fake, fake, fake, wsd, None) == _lib.ERR_MODE
    assert L.padoc_branch_decode(dplan.handle, fake, fake, fake, None, fake, fake, fake, wsd, None) == _lib.ERR_ARG
    assert L.padoc_set_kernel_events(fake, None) == _lib.ERR_ARG
    # schedule upload and resident decode: argument and state errors
    assert L.padoc_plan_upload(plan.handle, fake, ws_ok, None) == _lib.ERR_MODE  # forward plan
    assert L.padoc_plan_upload(dplan.handle, None, wsd, None) == _lib.ERR_WORKSPACE
    assert L.padoc_plan_upload(dplan.handle, fake, wsd - 1, None) == _lib.ERR_WORKSPACE
    assert L.padoc_plan_upload(None, fake, wsd, None) == _lib.ERR_ARG
    assert L.padoc_branch_decode_resident(plan.handle, fake, fake, fake, fake, fake, fake, fake, ws_ok,
                                          None) == _lib.ERR_MODE  # forward plan
    # never uploaded: refused before any launch
    assert L.padoc_branch_decode_resident(dplan.handle, fake, fake, fake, fake, fake, fake, fake, wsd,
                                          None) == _lib.ERR_MODE
    assert "padoc_plan_upload" in L.padoc_last_error().decode()
    assert L.padoc_branch_decode_resident(dplan.handle, fake, fake, fake, None, fake, fake, fake, wsd,
                                          None) == _lib.ERR_ARG


def test_last_error_is_thread_local():
    segs = _segs([(-1, 0, 10, 11, 0, 0)])
    with pytest.raises(pa.PadocError):
        pa.TreePlan(segs, **_desc(segs))
    msg = {}

    def other():
        msg["v"] = _lib.lib().padoc_last_error().decode()

    t = threading.Thread(target=other)
    t.start()
    t.join()
    assert msg["v"] == ""
    assert "q_len" in _lib.lib().padoc_last_error().decode()


# ---------------------------------------------------------------- generator

def test_workloads_regenerate_bit_exactly():
    for name in syn.CONFIGS:
        a, b = syn.make_workload(name), syn.make_workload(name)
        assert a.pages == b.pages


def test_workload_shapes():
    wl = syn.make_workload("single_page_decode")
    assert syn.count_queries(wl.pages) == 17
    wl = syn.make_workload("packed_forward_8pages")
    assert 30_000 < syn.count_tokens(wl.pages) < 60_000 and len(wl.pages) == 8
    wl = syn.make_workload("concurrent_decode_64pages")
    assert syn.count_queries(wl.pages) == 1600
    wl = syn.make_workload("dense_page_mixed_step")
    assert syn.count_queries(wl.pages) == 353
    for name in syn.CONFIGS:
        for p in syn.make_workload(name).pages:
            for b in p.branches:
                assert 0 <= b.fork <= p.stream_len and 0 <= b.q_len <= b.length
                if syn.make_workload(name).kind == "decode":
                    assert b.fork < p.stream_len   # the stream's newest token is not visible to branches


def test_block_ids_distinct_and_in_range():
    ids = syn.draw_block_ids(5000, 1 << 24, 3)
    assert len(set(ids.tolist())) == 5000 and ids.min() >= 0 and ids.max() < (1 << 24)
    ids = syn.draw_block_ids(100, 150, 3)
    assert len(set(ids.tolist())) == 100 and ids.max() < 150


def _check_backward(nodes, G, Hkv):
    """Backward key-major items cover every visible (key row, query row,
    head) exactly once: no pair is missed (a gradient term lost) or added
    twice (counted twice in the sum)."""
    segs = pa.segments_layout(nodes, 0)
    T = int(sum(n[2] for n in nodes))
    nq = int(sum(n[3] for n in nodes))
    plan = pa.TreePlan(segs, G * Hkv, Hkv, 128, "bf16", 0, num_kv_rows=T, num_q_rows=nq)
    ex = plan.export()
    row_tok = _token_of_row(nodes, segs["q_off"])
    want = {}
    for row, (s, p) in row_tok.items():
        for (t, j) in _visible_keys(nodes, s, p):
            krow = int(segs["kv_off"][t]) + j
            for g in range(Hkv):
                for h in range(G):
                    want[(krow, g, row, g * G + h)] = 1
    got = {}
    for b in ex["bwd"]:
        assert 0 < b["n_keys"] <= 128 and 0 < b["ncol"] and b["col0"] % 32 == 0
        assert b["col0"] + b["ncol"] <= b["ntok"] * G
        assert b["cost"] == -(-b["ncol"] // 32)
        for c in range(b["col0"], b["col0"] + b["ncol"]):
            t, h = divmod(c, G)
            row = int(ex["btoks"][b["tok_begin"] + t])
            lim = int(ex["blims"][b["lim_begin"] + t])
            assert 0 < lim <= b["n_keys"]
            for j in range(lim):
                key = (int(b["key_row0"]) + j, int(b["kvh"]), row, int(b["kvh"]) * G + h)
                got[key] = got.get(key, 0) + 1
    assert got == want
    costs = list(ex["bwd"]["cost"])
    assert costs == sorted(costs, reverse=True)
    return ex


@pytest.mark.parametrize("G,Hkv", [(1, 1), (8, 2), (7, 4)])
def test_backward_schedule_random_trees(G, Hkv):
    for seed in range(3):
        nodes = [(a.parent, a.fork, a.length, a.q_len)
                 for a in syn.random_tree(seed + 40, n_pages=2, max_depth=4, max_len=70, q_mode="some", max_nodes=10)]
        _check_backward(nodes, G, Hkv)


def test_backward_schedule_split_runs():
    # 500 queries x G=8 see the prefix: 4000 columns = 125 blocks, more than
    # the 64-block minimum piece -> two equal pieces per key run
    nodes = [(-1, 0, 130, 0), (0, 130, 300, 300), (1, 50, 120, 120), (1, 100, 80, 80)]
    ex = _check_backward(nodes, 8, 1)
    pre = ex["bwd"][ex["bwd"]["key_row0"] < 130]
    assert (pre["col0"] == 2016).any() and (pre["ncol"] == 2016).any()


def test_backward_workspace_and_modes():
    nodes = [(-1, 0, 10, 10)]
    segs = pa.segments_layout(nodes, 0)
    plan = pa.TreePlan(segs, 2, 1, 64, "bf16", 0, num_kv_rows=10, num_q_rows=10)
    nb = plan.backward_workspace_bytes()
    assert nb >= 10 * 2 * 4 + 2 * 10 * 1 * 64 * 4 and nb % 256 == 0
    f32 = pa.TreePlan(segs, 2, 1, 64, "f32", 0, num_kv_rows=10, num_q_rows=10)
    with pytest.raises(_lib.PadocError) as e:
        f32.backward_workspace_bytes()
    assert e.value.status == _lib.ERR_DTYPE


# ---------------------------------------------------------------- decoding depths

def test_tree_depths_match_oracle():
    cases = [[(a.parent, a.fork, a.length, a.q_len) for a in syn.random_tree(seed, n_pages=3, max_depth=5,
                                                                              max_len=30)] for seed in range(20)]
    for name in ("concurrent_decode_64pages", "packed_forward_8pages", "dense_page_mixed_step"):
        cases.append(od.page_nodes(syn.make_workload(name, 0).pages))
    for nodes in cases:
        segs = pa.segments_layout(nodes, 0)
        roots, d_seq, d_crit = pa.tree_depths(segs)
        want = od.decoding_depths(nodes)
        assert sorted(want) == roots.tolist()
        for r, a, b in zip(roots, d_seq, d_crit):
            assert (int(a), int(b)) == want[int(r)]


def test_tree_depths_errors():
    L = _lib.lib()
    bad = _segs([(0, 0, 3, 0, 0, 0)])                 # parent not earlier
    z = np.zeros(1, np.int64)
    assert L.padoc_tree_depths(bad.ctypes.data, 1, z.ctypes.data, z.ctypes.data) == _lib.ERR_TREE
    bad = _segs([(-1, 0, 3, 0, 0, 0), (0, 4, 2, 0, 3, 0)])   # fork beyond the parent
    z = np.zeros(2, np.int64)
    assert L.padoc_tree_depths(bad.ctypes.data, 2, z.ctypes.data, z.ctypes.data) == _lib.ERR_TREE
    assert L.padoc_tree_depths(None, -1, None, None) == _lib.ERR_ARG


def test_no_alloc_decode_rejects_oversized_plans():
    """A plan whose workspace exceeds the fixed per-GPU array is refused
    before anything touches a device (host-side check, no GPU needed)."""
    import ctypes as C
    import padoc_synth as syn
    wl = syn.make_workload("concurrent_decode_64pages")
    pages = wl.pages * 4
    segs = pa.segments_from_pages(pages, 16)
    nb, nq = syn.count_blocks(pages), syn.count_queries(pages)
    plan = pa.TreePlan(segs, 16, 2, 128, "bf16", 16, num_kv_rows=nb, num_q_rows=nq, block_table_len=nb)
    assert plan.workspace_bytes > pa.NO_ALLOC_WORKSPACE_BYTES
    fake = C.c_void_p(1 << 20)   # never dereferenced: the size check comes first
    st = pa._lib.lib().padoc_branch_decode_no_alloc(plan.handle, fake, fake, fake, fake, fake, fake, None)
    assert st == pa._lib.ERR_WORKSPACE
    assert "at most" in pa._lib.lib().padoc_last_error().decode()
