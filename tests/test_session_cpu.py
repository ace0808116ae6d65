"""Decode session host logic (no GPU): the Alg.-1 step loop, block pool and
block-table bookkeeping, the per-step schedule, and error handling.

* Every query of every step sees exactly the cache positions the oracle's
  replay of the fused mask (App. E, masked parallel decoding) selects.
* Blocks in use are distinct, inside the pool, and with the free ones make
  up the pool; every kept stream's table region holds its blocks; each new
  row's (block, slot) is its stream's position in its blocks; the step's
  patches, applied to the device table as the previous steps left it,
  reproduce every entry the step's tree reads.
* The step's schedule equals a plan built from scratch for the same tree.
* Closing every stream returns every block.
"""
import numpy as np
import pytest

import paper_2608_06146_amd as pa
from paper_2608_06146_amd import _lib

from _session import Alg1Run, make_decide, oracle_rows, session_visible_tags


def _check_blocks(sess, view, dev_table):
    seg = view["seg"]
    bt = view["block_table"]
    used = []
    for g in seg:
        nb = -(-int(g["len"]) // 16)
        ent = bt[int(g["kv_off"]): int(g["kv_off"]) + nb]
        assert (ent >= 0).all() and (ent < sess.num_blocks).all()
        used += ent.tolist()
        if view["prepared"]:
            assert (dev_table[int(g["kv_off"]): int(g["kv_off"]) + nb] == ent).all(), "patches miss an entry"
    assert len(used) == len(set(used)), "a block is used twice"
    assert len(used) + view["free_blocks"] == sess.num_blocks


def _check_new_slots(view, n_new):
    seg = view["seg"]
    bt = view["block_table"]
    for i, sid in enumerate(view["row_id"]):
        s = int(np.nonzero(view["seg_id"] == sid)[0][0])
        g = seg[s]
        L = int(g["len"])
        rows = view["new_slot"][view["new_off"][i]: view["new_off"][i + 1]]
        assert len(rows) == n_new[i]
        for j, (b, t) in enumerate(rows):
            pos = L - n_new[i] + j
            assert b == bt[int(g["kv_off"]) + pos // 16] and t == pos % 16


def _check_schedule_matches_fresh_plan(sess, view):
    ex = view["schedule"]
    segs = view["seg"]
    fresh = pa.TreePlan(segs, sess.num_heads_q, sess.num_heads_kv, sess.head_dim, sess.dtype, 16,
                        num_kv_rows=sess.num_blocks, num_q_rows=int(view["q_off"][-1]),
                        block_table_len=sess.block_table_capacity).export()
    for k in ("work", "ranges", "lims", "toks", "comb_ptr", "comb_slot", "comb_rows"):
        assert np.array_equal(ex[k], fresh[k]), k
    assert ex["n_work_shared"] == fresh["n_work_shared"]


@pytest.mark.parametrize("seed", range(6))
def test_alg1_replay_visibility_and_blocks(seed):
    rng = np.random.default_rng(seed)
    n_pages = 3
    prefix = [int(x) for x in rng.integers(1, 40, size=n_pages)]
    steps = 24
    decides = [make_decide(seed, pg, steps) for pg in range(n_pages)]
    sess = pa.DecodeSession(8, 2, 64, num_blocks=400, block_table_capacity=2048)
    run = Alg1Run(sess, prefix, decides)
    dev = np.full(sess.block_table_capacity, -7, dtype=np.int32)   # the device table as patched so far

    def do_step(n_new, n_query, schedule=False):
        sess.prepare(n_new, n_query)
        v = sess.view(schedule=schedule)
        for e, b in v["patch"]:
            dev[e] = b
        _check_blocks(sess, v, dev)
        _check_new_slots(v, n_new if n_new is not None else np.ones(len(v["row_id"]), np.int32))
        if schedule:
            _check_schedule_matches_fresh_plan(sess, v)
        sess.commit()
        return v

    n_new, n_q = run.prefill_rows()
    do_step(n_new, n_q)
    run.after_prefill()
    want = oracle_rows(prefix, decides, max_steps=steps + 12)
    n_checked = 0
    while sess.n_open:
        v = do_step(None, None, schedule=(run.step_no % 5 == 0))
        for r, (pg, c, i) in enumerate(run.rows(v["row_id"])):
            tags, rows = want[pg]
            row = rows[(c, i)]
            oracle_tags = {(pg,) + tags[l] for l in range(row.size) if row[l]}
            assert session_visible_tags(v, run, r) == oracle_tags, (pg, c, i)
            n_checked += 1
        run.events(v["row_id"])
    assert n_checked > 30
    # every page retired: all blocks back, nothing kept
    v = sess.view()
    assert v["free_blocks"] == sess.num_blocks and len(v["seg"]) == 0


def test_multi_token_steps_and_deep_trees():
    """Residual prefill (several new tokens, some queried), streams forked
    off content streams, parents closed before their children."""
    rng = np.random.default_rng(11)
    sess = pa.DecodeSession(4, 1, 64, num_blocks=300, block_table_capacity=1024)
    r = sess.open(-1, 0)
    dev = np.full(sess.block_table_capacity, -7, dtype=np.int32)
    lens = {r: 0}
    parent = {r: -1}
    for step in range(30):
        v0 = sess.view()
        ids = [int(x) for x in v0["row_id"]]
        n_new = rng.integers(0, 6, size=len(ids)).astype(np.int32)
        n_q = np.array([rng.integers(0, n + 1) for n in n_new], dtype=np.int32)
        sess.prepare(n_new, n_q)
        v = sess.view(schedule=True)
        for e, b in v["patch"]:
            dev[e] = b
        _check_blocks(sess, v, dev)
        _check_new_slots(v, n_new)
        _check_schedule_matches_fresh_plan(sess, v)
        assert list(v["q_off"]) == [0] + list(np.cumsum(n_q))
        sess.commit()
        for i, sid in enumerate(ids):
            lens[sid] += int(n_new[i])
        # events: fork a child of a random open stream at a random offset,
        # close a random open stream
        ids = [int(x) for x in sess.view()["row_id"]]
        if ids and rng.random() < 0.6:
            p = int(rng.choice(ids))
            c = sess.open(p, int(rng.integers(0, lens[p] + 1)))
            lens[c] = 0
            parent[c] = p
        if len(ids) > 2 and rng.random() < 0.3:
            sess.close(int(rng.choice(ids)))
    for sid in [int(x) for x in sess.view()["row_id"]]:
        sess.close(sid)
    assert sess.view()["free_blocks"] == sess.num_blocks


def test_region_moves_and_reuse():
    """A stream outgrowing its region moves (patches carry all its blocks);
    released regions and blocks are reused."""
    sess = pa.DecodeSession(2, 1, 64, num_blocks=40, block_table_capacity=64)
    a = sess.open(-1, 0)
    sess.prepare(np.array([64], np.int32), np.array([0], np.int32))     # 4 blocks: region of 4
    v = sess.view()
    assert len(v["patch"]) == 4 and int(v["seg"]["kv_off"][0]) == 0
    sess.commit()
    sess.prepare(np.array([1], np.int32), np.array([1], np.int32))      # 5 blocks: moves to a region of 8
    v = sess.view()
    assert int(v["seg"]["kv_off"][0]) == 4 and len(v["patch"]) == 5
    assert (v["block_table"][:4] == -1).all()
    sess.commit()
    b = sess.open(-1, 0)
    sess.prepare(np.array([0, 20], np.int32), np.array([0, 1], np.int32))  # b takes the freed region at 0
    v = sess.view()
    assert int(v["seg"]["kv_off"][1]) == 0
    sess.commit()
    sess.close(a)
    assert sess.view()["free_blocks"] == 40 - 2
    sess.close(b)
    assert sess.view()["free_blocks"] == 40


def test_pool_and_table_exhaustion_leave_state_unchanged():
    sess = pa.DecodeSession(2, 1, 64, num_blocks=6, block_table_capacity=16)
    a = sess.open(-1, 0)
    with pytest.raises(pa.PadocError) as e:
        sess.prepare(np.array([7 * 16], np.int32), np.array([0], np.int32))
    assert e.value.status == _lib.ERR_BOUNDS
    v = sess.view()
    assert v["free_blocks"] == 6 and int(v["seg"]["len"][0]) == 0 and not v["prepared"]
    sess.prepare(np.array([6 * 16], np.int32), np.array([1], np.int32))   # fits exactly
    sess.commit()
    # table: region of 8 in use; a second stream of 9 blocks' region (16) does not fit
    sess2 = pa.DecodeSession(2, 1, 64, num_blocks=100, block_table_capacity=16)
    x = sess2.open(-1, 0)
    y = sess2.open(-1, 0)
    sess2.prepare(np.array([16 * 8, 16], np.int32), np.array([0, 0], np.int32))
    sess2.commit()
    with pytest.raises(pa.PadocError) as e:
        sess2.prepare(np.array([0, 16 * 8], np.int32), np.array([0, 0], np.int32))
    assert e.value.status == _lib.ERR_BOUNDS
    v = sess2.view()
    assert list(v["seg"]["len"]) == [128, 16] and v["free_blocks"] == 100 - 9
    assert x == 0 and y == 1


def test_session_errors():
    L = _lib.lib()
    sess = pa.DecodeSession(4, 2, 64, num_blocks=16)
    with pytest.raises(pa.PadocError) as e:
        sess.open(3, 0)                       # no such parent
    assert e.value.status == _lib.ERR_ARG
    with pytest.raises(pa.PadocError) as e:
        sess.open(-1, 2)                      # a root has fork 0
    assert e.value.status == _lib.ERR_TREE
    r = sess.open(-1, 0)
    with pytest.raises(pa.PadocError) as e:
        sess.open(r, 1)                       # fork beyond the parent's length
    assert e.value.status == _lib.ERR_TREE
    with pytest.raises(pa.PadocError) as e:
        sess.prepare(np.array([1], np.int32), np.array([2], np.int32))
    assert e.value.status == _lib.ERR_ARG
    with pytest.raises(pa.PadocError) as e:
        sess.commit()
    assert e.value.status == _lib.ERR_MODE
    sess.prepare()
    for call in (lambda: sess.prepare(), lambda: sess.open(r, 0), lambda: sess.close(r)):
        with pytest.raises(pa.PadocError) as e:
            call()
        assert e.value.status == _lib.ERR_MODE
    # host-only session: launch is refused before any device call
    st = L.padoc_session_launch(sess.handle, None, None, None, None, None, None, 0, None)
    assert st == _lib.ERR_ARG
    sess.commit()
    sess.close(r)
    with pytest.raises(pa.PadocError) as e:
        sess.close(r)
    assert e.value.status == _lib.ERR_ARG
    with pytest.raises(pa.PadocError) as e:
        sess.open(r, 0)                       # released
    assert e.value.status == _lib.ERR_ARG
    with pytest.raises(pa.PadocError) as e:
        pa.DecodeSession(4, 3, 64, num_blocks=16)   # Hq not a multiple of Hkv
    assert e.value.status == _lib.ERR_SHAPE


def test_steps_with_no_open_stream_and_closed_parents():
    """A step with no open stream is empty; a closed stream with an open
    child keeps its blocks and takes new children."""
    sess = pa.DecodeSession(4, 2, 64, num_blocks=32)
    n_kv, n_q, ws = sess.prepare()
    assert (n_kv, n_q) == (0, 0) and len(sess.view()["seg"]) == 0
    sess.commit()
    r = sess.open(-1, 0)
    sess.prepare(np.array([20], np.int32), np.array([0], np.int32))
    sess.commit()
    a = sess.open(r, 20)
    sess.close(r)
    b = sess.open(r, 7)                      # a closed but kept parent takes a child
    sess.prepare()
    v = sess.view()
    assert list(v["seg"]["parent"]) == [-1, 0, 0] and list(v["seg"]["fork"]) == [0, 20, 7]
    assert list(v["seg"]["q_len"]) == [0, 1, 1]
    sess.commit()
    sess.close(a)
    sess.close(b)
    v = sess.view()
    assert len(v["seg"]) == 0 and v["free_blocks"] == 32


# ---------------------------------------------------------------- remaining paths and budgeted steps

def _segs_of(nodes):
    seg = np.zeros(len(nodes), dtype=pa.SEGMENT_DTYPE)
    seg["parent"] = [x[0] for x in nodes]
    seg["fork"] = [x[1] for x in nodes]
    seg["len"] = [x[2] for x in nodes]
    return seg


def _random_states(nodes, rng, count):
    """Reachable progress states: random started segments advance."""
    from oracle import dense as od
    prog = [0] * len(nodes)
    out = [list(prog)]
    for _ in range(count):
        st = od._started(nodes, prog)
        cand = [s for s in range(len(nodes)) if nodes[s][0] >= 0 and st[s] and prog[s] < nodes[s][2]]
        if not cand:
            break
        for s in cand:
            if rng.random() < 0.6:
                prog[s] += 1
        out.append(list(prog))
    return out


@pytest.mark.parametrize("seed", range(10))
def test_tree_remaining_matches_oracle(seed):
    import padoc_synth as syn
    from oracle import dense as od
    nodes = [(a.parent, a.fork, a.length, a.q_len)
             for a in syn.random_tree(seed, n_pages=3, max_len=6, max_depth=5, max_children=3)]
    segs = _segs_of(nodes)
    rng = np.random.default_rng(seed)
    for prog in _random_states(nodes, rng, 12):
        got = pa.tree_remaining(segs, prog)
        want = od.remaining_paths(nodes, prog)
        assert got.tolist() == want.tolist(), prog
    _, _, crit = pa.tree_depths(segs)
    roots = [s for s in range(len(nodes)) if nodes[s][0] < 0]
    assert pa.tree_remaining(segs)[roots].tolist() == crit.tolist()


def test_tree_remaining_errors():
    nodes = [(-1, 0, 5, 0), (0, 5, 4, 0), (1, 2, 3, 0)]
    segs = _segs_of(nodes)
    with pytest.raises(pa.PadocError):
        pa.tree_remaining(segs, [0, 5, 0])      # progress past the length
    with pytest.raises(pa.PadocError):
        pa.tree_remaining(segs, [0, 1, 1])      # child progressed before its fork
    with pytest.raises(pa.PadocError):
        pa.tree_remaining(segs, [0, -1, 0])
    bad = segs.copy()
    bad["fork"][2] = 9                          # fork past the parent's length
    with pytest.raises(pa.PadocError):
        pa.tree_remaining(bad)
    assert pa.tree_remaining(segs, [0, 2, 1]).tolist() == [2, 2, 2]


def test_session_select_orders():
    s = pa.DecodeSession(4, 2, 64, 64, "bf16")
    r = s.open(-1, 0)
    s.prepare(np.array([4], np.int32), np.array([0], np.int32))
    s.commit()
    ids = [s.open(r, 4) for _ in range(5)]
    s.close(r)
    n_new, n_q = s.select(0)
    assert n_new.tolist() == [1] * 5 and n_q.tolist() == [1] * 5
    n_new, _ = s.select(2)
    assert n_new.tolist() == [1, 1, 0, 0, 0]            # the oldest
    n_new, n_q = s.select(3, [5, 9, 5, 9, 1])
    assert n_new.tolist() == [1, 1, 0, 1, 0]            # 9, 9, then the older 5
    assert n_q.tolist() == n_new.tolist()
    assert len(ids) == 5
    s.destroy()


@pytest.mark.parametrize("seed", range(8))
def test_budgeted_replay_matches_oracle(seed):
    """The session driven by padoc_session_select (oldest first, or with
    padoc_tree_remaining as priorities) advances, step by step, exactly the
    segments of the oracle's budgeted decoding."""
    import bench
    import padoc_synth as syn
    from oracle import dense as od
    nodes = [(a.parent, a.fork, a.length, a.q_len)
             for a in syn.random_tree(seed + 40, n_pages=2, max_len=7, max_depth=4, max_children=3)]
    if not any(x[0] >= 0 for x in nodes):
        pytest.skip("no decoded segment")
    for B in (1, 2, 3, 0):
        for by_pr in (False, True):
            s = pa.DecodeSession(4, 2, 64, 4096, "bf16")
            R = bench.BudgetedReplay(pa, np, s, nodes, B, by_pr)
            while not R.done():
                R.step()
            want = od.budgeted_decoding(nodes, B, by_pr)
            assert R.steps == want, (B, by_pr)
            s.destroy()
