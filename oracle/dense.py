"""Plain fp64 CPU oracle for PaDoc's ancestor-masked tree attention.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  The product library
never calls it, and it shares no code with the product (no kernels, headers,
tables or helpers); the two meet only through the seeded inputs of
``padoc_synth``.

What it computes, and where the paper defines it
------------------------------------------------
* Visibility (Sec. 3.2, "Training Paradigm", ancestor sets): every token of a
  node V attends to all tokens of V's ancestors and to the non-future tokens
  of V itself.  Generalised to a segment tree: a query token ``(s, p)`` sees
  key ``(t, j)`` iff ``t == s and j <= p`` or ``t`` is a proper ancestor of
  ``s`` and ``j < F(s, t)``, where ``F(s, t)`` is the fork offset of the child
  of ``t`` on the path to ``s`` (the number of leading tokens of ``t`` visible
  below that child; App. C, packed sample ``[M | Y_1..Y_N]`` with ``M_{<=f_k}``).
* Attention (App. E, the Attn equation): ``softmax(Q K^T / sqrt(d) + A_M) V``
  with ``A_M`` the additive mask.  Masked keys are left out of every sum
  (select-masking), which is the same value.  The log-sum-exp output is
  ``LSE = ln sum_visible exp(scale * q . k)`` (natural log, scale included).
* The paper's "reference implementation" materialises the dense Boolean
  ancestor mask and runs masked softmax attention on it (App. C, Dense SDPA);
  this oracle does exactly that, per page, in fp64.
* Masked parallel decoding (App. E, Algorithm "Masked parallel decoding"):
  :func:`simulate_masked_parallel_decoding` runs a synthetic event trace and
  writes down the fused mask rows it implies (a row is what its stream was
  given when it opened plus its own cached tokens), so the tests can pin the
  visibility rule and the fork-offset reading to the decoding semantics.

Readings of points the paper leaves open are listed in the repository's design
notes; the ones this file depends on: fork offsets are half-open counts
(``[0, f)``); the page prefix is causal in itself; a branch's branch-start
token is its own position 0; GQA maps query head ``h`` to KV head
``h // (Hq // Hkv)``; queries of a segment are its last ``q_len`` tokens.

Inputs are numpy arrays or torch tensors (converted exactly to float64; bf16
values are represented exactly).  Nothing here is tuned for speed beyond
processing query rows in batches (each row's arithmetic is unchanged).
"""
from __future__ import annotations

from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "page_nodes", "canonical_layout", "ancestors", "visible_counts", "page_of",
    "dense_mask", "masked_attention", "tree_attention", "tree_attention_paged",
    "gather_paged", "paged_slots", "chunk_slot", "simulate_masked_parallel_decoding",
    "visible_pair_count", "decoding_depths", "remaining_paths", "budgeted_decoding",
]

Node = Tuple[int, int, int, int]   # (parent, fork, length, q_len)


def _f64(x) -> np.ndarray:
    try:
        import torch
        if isinstance(x, torch.Tensor):
            return x.detach().to("cpu", torch.float64).numpy()
    except ImportError:  # pragma: no cover
        pass
    return np.asarray(x, dtype=np.float64)


def _as_nodes(nodes) -> List[Node]:
    out = []
    for n in nodes:
        if isinstance(n, tuple) and len(n) == 4:
            out.append(tuple(int(v) for v in n))
        else:
            out.append((int(n.parent), int(n.fork), int(n.length), int(n.q_len)))
    return out


# --------------------------------------------------------------------------
# Tree structure
# --------------------------------------------------------------------------

def page_nodes(pages) -> List[Node]:
    """The paper's packed sample per page, ``[prefix | stream | Y_1..Y_N]``
    (App. C), as segments: the prefix is a root; the layout stream is its
    child and sees the whole prefix (fork = P); branch ``Y_k`` is a child of
    the stream with fork ``f_k`` (it sees stream tokens ``[0, f_k)``; its
    branch-start token is its own position 0, Sec. 3.2 last paragraph).
    Pages are concatenated."""
    nodes: List[Node] = []
    for pg in pages:
        get = (lambda k: pg[k]) if isinstance(pg, dict) else (lambda k: getattr(pg, k))
        root = len(nodes)
        nodes.append((-1, 0, int(get("prefix_len")), int(get("prefix_q"))))
        stream = len(nodes)
        nodes.append((root, int(get("prefix_len")), int(get("stream_len")), int(get("stream_q"))))
        for b in get("branches"):
            bget = (lambda k: b[k]) if isinstance(b, dict) else (lambda k: getattr(b, k))
            nodes.append((stream, int(bget("fork")), int(bget("length")), int(bget("q_len"))))
    return nodes


def canonical_layout(nodes, block_size: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """Packed order = node order.  ``kv_off[s]``: first K/V row of segment s
    (packed) or first block-table entry (paged: each segment owns
    ``ceil(len / block_size)`` consecutive entries).  ``q_off[s]``: first
    Q/O/LSE row (segments' queries concatenated in node order)."""
    nodes = _as_nodes(nodes)
    kv_off = np.zeros(len(nodes), dtype=np.int64)
    q_off = np.zeros(len(nodes), dtype=np.int64)
    kv = q = 0
    for i, (_, _, n, ql) in enumerate(nodes):
        kv_off[i] = kv
        q_off[i] = q
        kv += n if block_size == 0 else -(-n // block_size)
        q += ql
    return kv_off, q_off


def ancestors(nodes, s: int) -> List[Tuple[int, int]]:
    """Proper ancestors of segment s, root first, each with ``F(s, t)``: the
    fork of the child of t that lies on the path to s."""
    nodes = _as_nodes(nodes)
    chain = []
    child = s
    t = nodes[s][0]
    while t >= 0:
        chain.append((t, nodes[child][1]))
        child = t
        t = nodes[t][0]
    return chain[::-1]


def visible_counts(nodes, s: int, p: int) -> Dict[int, int]:
    """Query token p of segment s sees keys ``[0, count)`` of each listed
    segment (ancestors via their fork offsets, itself causally)."""
    out = {t: f for t, f in ancestors(nodes, s)}
    out[s] = p + 1
    return out


def page_of(nodes) -> np.ndarray:
    nodes = _as_nodes(nodes)
    root = np.zeros(len(nodes), dtype=np.int64)
    for i, (par, _, _, _) in enumerate(nodes):
        root[i] = i if par < 0 else root[par]
    return root


def dense_mask(nodes, root: int) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Dense Boolean ancestor mask of one page (App. C, Dense SDPA).

    Returns ``(seg, pos, mask)``: the page's tokens in packed order tagged with
    their segment and position, and ``mask[a, b]`` = token a may see token b,
    straight from the rule: same segment and not in the future, or an ancestor
    segment's token before the fork offset on the path."""
    nodes = _as_nodes(nodes)
    roots = page_of(nodes)
    segs = [i for i in range(len(nodes)) if roots[i] == root]
    seg = np.concatenate([np.full(nodes[i][2], i, dtype=np.int64) for i in segs]) if segs else np.zeros(0, np.int64)
    pos = np.concatenate([np.arange(nodes[i][2], dtype=np.int64) for i in segs]) if segs else np.zeros(0, np.int64)
    n = seg.size
    mask = np.zeros((n, n), dtype=bool)
    for a in range(n):
        s, p = int(seg[a]), int(pos[a])
        anc = dict(ancestors(nodes, s))
        for b in range(n):
            t, j = int(seg[b]), int(pos[b])
            if t == s:
                mask[a, b] = j <= p
            elif t in anc:
                mask[a, b] = j < anc[t]
    return seg, pos, mask


def visible_pair_count(nodes) -> int:
    """Number of visible (query, key) pairs, queries = last q_len tokens."""
    nodes = _as_nodes(nodes)
    total = 0
    for s, (_, _, n, ql) in enumerate(nodes):
        anc = sum(f for _, f in ancestors(nodes, s))
        for p in range(n - ql, n):
            total += anc + p + 1
    return total


# --------------------------------------------------------------------------
# Attention by definition
# --------------------------------------------------------------------------

def masked_attention(q, k, v, mask, scale: float, return_probs: bool = False):
    """Masked softmax attention of one head, fp64, by definition.

    ``q [nq, d]``, ``k, v [nk, d]``, ``mask [nq, nk]`` (True = visible).
    Per row: scores ``s_j = scale * q . k_j`` over visible j, ``m = max s``,
    ``w_j = exp(s_j - m)``, ``l = sum w``, ``o = sum (w_j / l) v_j``,
    ``lse = m + ln l``.  Masked keys enter no sum."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    mask = np.asarray(mask, dtype=bool)
    if mask.shape[0] and not mask.any(axis=1).all():
        raise ValueError("a query row sees no key")
    s = scale * (q @ k.T)
    m = np.max(np.where(mask, s, -np.inf), axis=1, keepdims=True)
    w = np.where(mask, np.exp(np.where(mask, s - m, 0.0)), 0.0)
    l = w.sum(axis=1, keepdims=True)
    p = w / l
    o = p @ v
    lse = (m + np.log(l))[:, 0]
    if return_probs:
        return o, lse, p
    return o, lse


def tree_attention(nodes, q, k, v, scale: float, num_heads_q: int, num_heads_kv: int,
                   kv_off=None, q_off=None, rows: Optional[Iterable[int]] = None,
                   return_probs: bool = False, row_batch: int = 512):
    """Packed tree attention by definition.

    ``q [n_q, Hq, d]``; ``k, v [T, Hkv, d]`` with segment s's tokens at rows
    ``kv_off[s] ..``; segment s's queries (its last ``q_len`` tokens) at Q rows
    ``q_off[s] ..``.  Offsets default to :func:`canonical_layout`.

    Returns ``(O [n_q, Hq, d], LSE [n_q, Hq])`` in fp64 (rows not requested via
    ``rows`` are NaN).  With ``return_probs`` also ``P [n_q, Hq, T]``."""
    nodes = _as_nodes(nodes)
    if num_heads_q % num_heads_kv:
        raise ValueError("Hq must be a multiple of Hkv")
    G = num_heads_q // num_heads_kv
    k64, v64 = _f64(k), _f64(v)
    q64 = _f64(q)
    if kv_off is None or q_off is None:
        ko, qo = canonical_layout(nodes, 0)
        kv_off = ko if kv_off is None else kv_off
        q_off = qo if q_off is None else q_off
    n_q = q64.shape[0]
    dv = v64.shape[2]
    O = np.full((n_q, num_heads_q, dv), np.nan)
    LSE = np.full((n_q, num_heads_q), np.nan)
    P = np.zeros((n_q, num_heads_q, k64.shape[0])) if return_probs else None
    want = None if rows is None else set(int(r) for r in rows)
    roots = page_of(nodes)
    for root in sorted(set(int(r) for r in roots)):
        segs = [i for i in range(len(nodes)) if roots[i] == root]
        starts, total = {}, 0
        for i in segs:
            starts[i] = total
            total += nodes[i][2]
        kv_rows = np.concatenate([kv_off[i] + np.arange(nodes[i][2], dtype=np.int64) for i in segs]) \
            if total else np.zeros(0, np.int64)
        # query tokens of this page, in packed order: (segment, position, Q row)
        qs, qp, qr = [], [], []
        for s in segs:
            n, ql = nodes[s][2], nodes[s][3]
            for p in range(n - ql, n):
                r = int(q_off[s] + p - (n - ql))
                if want is None or r in want:
                    qs.append(s)
                    qp.append(p)
                    qr.append(r)
        if not qr:
            continue
        qr = np.array(qr)
        # mask rows of the query tokens, straight from the visibility rule
        mask = np.zeros((len(qr), total), dtype=bool)
        for a, (s, p) in enumerate(zip(qs, qp)):
            mask[a, starts[s]: starts[s] + p + 1] = True
            for t, f in ancestors(nodes, s):
                mask[a, starts[t]: starts[t] + f] = True
        for h in range(num_heads_q):
            g = h // G
            kh = k64[kv_rows, g, :]
            vh = v64[kv_rows, g, :]
            for b0 in range(0, qr.size, row_batch):
                sel = slice(b0, b0 + row_batch)
                res = masked_attention(q64[qr[sel], h, :], kh, vh, mask[sel], scale,
                                       return_probs=return_probs)
                O[qr[sel], h, :] = res[0]
                LSE[qr[sel], h] = res[1]
                if return_probs:
                    P[np.ix_(qr[sel], [h], kv_rows)] = res[2][:, None, :]
    if return_probs:
        return O, LSE, P
    return O, LSE


# --------------------------------------------------------------------------
# Paged KV cache
# --------------------------------------------------------------------------

def paged_slots(nodes, block_table, block_size: int, bt_off=None):
    """Physical location of every token: ``(block_id, slot)`` arrays in packed
    token order.  Token t of segment s lives in block
    ``block_table[bt_off[s] + t // block_size]`` at slot ``t % block_size``."""
    nodes = _as_nodes(nodes)
    bt = np.asarray(block_table, dtype=np.int64)
    if bt_off is None:
        bt_off, _ = canonical_layout(nodes, block_size)
    blk, slot = [], []
    for s, (_, _, n, _) in enumerate(nodes):
        t = np.arange(n, dtype=np.int64)
        blk.append(bt[bt_off[s] + t // block_size])
        slot.append(t % block_size)
    if not blk:
        return np.zeros(0, np.int64), np.zeros(0, np.int64)
    return np.concatenate(blk), np.concatenate(slot)


def chunk_slot(t):
    """Slot of token ``t`` (0..15) inside a chunk-major K block: bits 2 and 3
    of ``t`` exchanged (the cache layout the library documents)."""
    t = np.asarray(t)
    return (t & 3) | ((t >> 3) & 1) << 2 | ((t >> 2) & 1) << 3


def gather_paged(nodes, pool, block_table, block_size: int, bt_off=None, d_major: bool = False,
                 layout: str = None) -> np.ndarray:
    """Read a paged cache back into packed token order ``[T, Hkv, d]``
    (fp64).  ``layout``:

    * ``"rows"``: ``pool [num_blocks, Hkv, block_size, d]``;
    * ``"d_major"`` (or ``d_major=True``): ``pool [num_blocks, Hkv, d, block_size]``;
    * ``"chunked"``: ``pool [num_blocks, Hkv, d/8, 16, 8]``, token ``t``'s dims
      ``[8c, 8c+8)`` at ``[c, chunk_slot(t), :]``."""
    layout = layout or ("d_major" if d_major else "rows")
    blk, slot = paged_slots(nodes, block_table, block_size, bt_off)
    if layout == "chunked":
        slot = chunk_slot(slot)
    try:
        import torch
        if isinstance(pool, torch.Tensor):
            bi = torch.as_tensor(blk, device=pool.device)
            si = torch.as_tensor(slot, device=pool.device)
            if layout == "d_major":
                got = pool[bi, :, :, si]
            elif layout == "chunked":
                got = pool[bi, :, :, si, :].reshape(len(blk), pool.shape[1], -1)
            else:
                got = pool[bi, :, si, :]
            return got.to("cpu", torch.float64).numpy()
    except ImportError:  # pragma: no cover
        pass
    p = _f64(pool)
    if layout == "d_major":
        return p[blk, :, :, slot]
    if layout == "chunked":
        return p[blk, :, :, slot, :].reshape(len(blk), p.shape[1], -1)
    return p[blk, :, slot, :]


def tree_attention_paged(nodes, q, k_pool, v_pool, block_table, scale: float,
                         num_heads_q: int, num_heads_kv: int, block_size: int = 16,
                         bt_off=None, q_off=None, rows=None):
    """Decode form: K/V in a paged cache, the library's cache format: K blocks
    chunk-major ``[num_blocks, Hkv, d/8, 16, 8]`` (see :func:`chunk_slot`), V
    blocks d-major ``[num_blocks, Hkv, d, 16]``.  Gathers every segment back
    into packed order with :func:`gather_paged`, then applies
    :func:`tree_attention`."""
    nodes = _as_nodes(nodes)
    k = gather_paged(nodes, k_pool, block_table, block_size, bt_off, layout="chunked")
    v = gather_paged(nodes, v_pool, block_table, block_size, bt_off, d_major=True)
    kv_off, qo = canonical_layout(nodes, 0)
    return tree_attention(nodes, q, k, v, scale, num_heads_q, num_heads_kv,
                          kv_off=kv_off, q_off=qo if q_off is None else q_off, rows=rows)


# --------------------------------------------------------------------------
# Decoding depth (Sec. 3.1) and forward steps (App. D)
# --------------------------------------------------------------------------

def decoding_depths(nodes):
    """Per page root: ``(D_seq, D_crit)``.

    The roots are the page inputs (prefilled, not decoded); every other
    segment is decoded one token per step.  Sequential decoding emits the
    decoded segments one after another: ``D_seq`` = the sum of their lengths
    (Sec. 3.1, layout length plus every content length).  Decoding all
    streams concurrently, a segment can start once its parent has produced
    the ``fork`` tokens it conditions on, so it starts at step
    ``start(s) = start(parent) + fork`` (0 below a root) and finishes at
    ``start(s) + len(s)``; ``D_crit`` = the latest finish over the page
    (Sec. 3.1 critical path ``max_k [l(B_<=k) + l(Y_k)]``, also bounded below
    by the layout length; App. D ``F_PaDoc``).  Returns a dict root ->
    (D_seq, D_crit)."""
    nodes = _as_nodes(nodes)
    root = page_of(nodes)
    start = {}
    out = {}
    for s, (parent, fork, n, _) in enumerate(nodes):
        r = int(root[s])
        seq, crit = out.get(r, (0, 0))
        if parent < 0:
            out[r] = (seq, crit)
            continue
        start[s] = (start[parent] if nodes[parent][0] >= 0 else 0) + (fork if nodes[parent][0] >= 0 else 0)
        out[r] = (seq + n, max(crit, start[s] + n))
    return out


def _started(nodes, produced):
    """Which decoded segments have started: a child of a root with its page,
    a deeper one once its parent has started and produced ``fork`` tokens
    (Sec. 3.1 dependency: a content stream conditions on the layout tokens
    before its region)."""
    started = [False] * len(nodes)
    for s, (parent, fork, _, _) in enumerate(nodes):
        if parent < 0:
            continue
        if nodes[parent][0] < 0:
            started[s] = True
        else:
            started[s] = started[parent] and produced[parent] >= fork
    return started


def remaining_paths(nodes, progress=None):
    """Remaining critical path of every segment, by running the decoding:
    from the state where segment s has produced ``progress[s]`` tokens,
    every started segment produces one token per step (ideal parallel
    scheduling, Sec. 3.1).  For a decoded segment s: the steps until s and
    the segments below it that have not started yet are done, counted from
    the step s starts in if it has not started.  For a root: the steps until
    its whole page is done.  Returns an int64 array."""
    nodes = _as_nodes(nodes)
    n = len(nodes)
    prog = [0] * n if progress is None else [int(x) for x in progress]
    for s, nd in enumerate(nodes):
        if nd[0] < 0:
            prog[s] = 0
    start_state = _started(nodes, prog)
    root = page_of(nodes)
    children: Dict[int, List[int]] = {}
    for s, nd in enumerate(nodes):
        if nd[0] >= 0:
            children.setdefault(nd[0], []).append(s)

    def group(s):
        """Segments whose completion s waits for, as defined above."""
        if nodes[s][0] < 0:
            return [t for t in range(n) if root[t] == s and nodes[t][0] >= 0]
        out, todo = [s], [c for c in children.get(s, []) if not start_state[c]]
        while todo:
            c = todo.pop()
            out.append(c)
            todo.extend(children.get(c, []))
        return out

    out = np.zeros(n, dtype=np.int64)
    for s in range(n):
        members = group(s)
        produced = list(prog)
        steps = 0
        while any(produced[t] < nodes[t][2] for t in members):
            started = _started(nodes, produced)
            if nodes[s][0] < 0 or started[s]:
                steps += 1
            for t in range(n):
                if nodes[t][0] >= 0 and started[t] and produced[t] < nodes[t][2]:
                    produced[t] += 1
        out[s] = steps
    return out


def budgeted_decoding(nodes, max_rows: int, by_priority: bool):
    """Decode every page of the tree with at most ``max_rows`` rows per step.
    Each step the started, unfinished segments are the candidates, ranked by
    the order they started in (ties by segment index: the opening order);
    if more than ``max_rows``, the first ``max_rows`` of them in that order
    advance (``by_priority`` False), or those with the largest remaining
    critical path (:func:`remaining_paths` at the step's progress), equal
    paths in that order.  Returns the list of advanced segment sets, one per
    step."""
    nodes = _as_nodes(nodes)
    n = len(nodes)
    produced = [0] * n
    opened_at: Dict[int, int] = {}
    steps = []
    step = 0
    while True:
        started = _started(nodes, produced)
        for s in range(n):
            if started[s] and s not in opened_at:
                opened_at[s] = step
        cand = [s for s in range(n) if nodes[s][0] >= 0 and started[s] and produced[s] < nodes[s][2]]
        if not cand:
            return steps
        cand.sort(key=lambda s: (opened_at[s], s))
        if 0 < max_rows < len(cand):
            if by_priority:
                rem = remaining_paths(nodes, produced)
                cand = sorted(cand, key=lambda s: -int(rem[s]))   # stable: keeps the opening order
            cand = cand[:max_rows]
        for s in cand:
            produced[s] += 1
        steps.append(sorted(cand))
        step += 1


# --------------------------------------------------------------------------
# Masked parallel decoding (App. E), on the logical fused mask
# --------------------------------------------------------------------------

def _run_event_trace(decide, max_steps: int):
    """The event trace alone: at each step every live stream emits one token
    (live streams in opening order, the layout stream 0 first), then
    ``decide`` says what follows for each.  Returns ``(emitted, born)``:
    ``emitted[t]`` lists ``(stream, index)`` of the tokens cached at step t,
    ``born[c]`` is the step after which content stream c opened (the step at
    which the layout stream's output closed a region)."""
    live = [0]
    count = {0: 0}
    born: Dict[int, int] = {}
    emitted: List[List[Tuple[int, int]]] = []
    for t in range(max_steps):
        if not live:
            break
        emitted.append([(c, count[c]) for c in live])
        for c in live:
            count[c] += 1
        outcome = {c: decide(t, c, c == 0) for c in live}
        nxt = [c for c in live if outcome[c] != "eos"]
        if outcome.get(0) == "fork":
            c_new = max(count) + 1
            count[c_new] = 0
            born[c_new] = t
            nxt.append(c_new)
        live = nxt
    return emitted, born


def simulate_masked_parallel_decoding(prefix_len: int, decide, max_steps: int = 64):
    """Masked parallel decoding (App. E, algorithm "Masked parallel
    decoding") reduced to the fused mask it builds over the shared cache.

    ``decide(step, stream_id, is_layout)`` gives what happens after a stream
    has been decoded at ``step``: ``"continue"``, ``"eos"`` (the stream
    stops), or, for the layout stream only, ``"fork"`` (its output closes a
    region, which opens a content stream).  Stream 0 is the layout stream;
    content streams are numbered 1, 2, ... as they open.

    The trace is run first (:func:`_run_event_trace`); the fused mask is then
    written down as a function of it.  The method gives each stream one mask
    row over the cache columns.  A row holds what the stream was given when
    it opened -- the page prefix for the layout stream, the layout stream's
    row of that moment for a content stream -- and, from then on, exactly
    the columns of the tokens the stream itself puts into the cache (each
    step appends one column per live stream, set only in its own row).  The
    token a stream caches at step t is queried with its row as it stands
    after that step's columns are added.  A region close happens after the
    step's outputs are sampled, so the closing output is not yet cached when
    the content stream's row is taken (it enters at the next step, in the
    layout row only).

    Returns ``(tags, queries, forks)``: ``tags[l] = (stream, index)`` names
    the token at cache position l (stream -1 = page prefix); ``queries`` lists
    ``(stream, index, row)`` with the Boolean row used for that token, over
    the cache positions present at that step; ``forks[c]`` = layout-stream
    tokens in the cache when stream c opened."""
    emitted, born = _run_event_trace(decide, max_steps)
    tags: List[Tuple[int, int]] = [(-1, i) for i in range(prefix_len)]
    step_of: List[int] = [-1] * prefix_len       # step that cached each column
    width: List[int] = []                        # cache columns after each step
    for t, toks in enumerate(emitted):
        tags.extend(toks)
        step_of.extend([t] * len(toks))
        width.append(len(tags))
    tag_stream = np.array([c for c, _ in tags], dtype=np.int64)
    col_step = np.array(step_of, dtype=np.int64)

    def row_after(c: int, t: int) -> np.ndarray:
        """Stream c's row once step t's columns are in the cache (over every
        column of the trace; columns cached later are never set)."""
        own = (tag_stream == c) & (col_step <= t)
        if c == 0:
            given = tag_stream == -1
        else:
            given = row_after(0, born[c])
        return given | own

    queries = []
    for t, toks in enumerate(emitted):
        for c, i in toks:
            queries.append((c, i, row_after(c, t)[: width[t]]))
    forks = {c: sum(1 for t2 in range(tb + 1) for s, _ in emitted[t2] if s == 0)
             for c, tb in born.items()}
    return tags, queries, forks
