"""Alg.-1 replay shared by the session tests.

Pages run masked parallel decoding (App. E) on one ``DecodeSession``: each
page's prefix is prefilled as a root stream, the layout stream forks off it,
and at every step each live stream appends one token and queries it; a
seeded ``decide(step, stream, is_layout)`` picks the events (layout stream:
continue / fork a content stream / end; content stream: continue / end).
The oracle (``simulate_masked_parallel_decoding``) replays the same events
on the logical fused mask, page by page; the tests compare each query's
visible cache positions (host) or its attention output (GPU) with what the
oracle's mask row selects.
"""
from __future__ import annotations

from typing import Dict, List, Tuple

import numpy as np

from oracle import dense as od


def make_decide(seed: int, page: int, steps: int, p_fork: float = 0.35, p_end: float = 0.15):
    """Layout stream ends at step steps-1 at the latest, content streams at
    step steps+8."""
    def decide(step, c, is_layout):
        u = np.random.default_rng([seed, page, step, c + 1]).random()
        if is_layout:
            if step >= steps - 1 or u < 0.04:
                return "eos"
            return "fork" if u < p_fork else "continue"
        return "eos" if (u < p_end or step >= steps + 8) else "continue"
    return decide


class Alg1Run:
    """Drives a session through the events of ``decides`` (one per page) and
    records, per step, each row's (page, stream, index)."""

    def __init__(self, sess, prefix_lens: List[int], decides):
        self.s = sess
        self.P = list(prefix_lens)
        self.decides = decides
        self.sid_of: Dict[Tuple[int, int], int] = {}
        self.tag_of: Dict[int, Tuple[int, int]] = {}   # stream id -> (page, c); c = -1 for the prefix
        self.count: Dict[Tuple[int, int], int] = {}
        self.next_c = [1] * len(prefix_lens)
        self.step_no = 0

    def prefill_rows(self):
        """Open the page roots; returns (n_new, n_query) of the prefill step."""
        for pg in range(len(self.P)):
            sid = self.s.open(-1, 0)
            self.sid_of[(pg, -1)] = sid
            self.tag_of[sid] = (pg, -1)
        n = np.array(self.P, dtype=np.int32)
        return n, np.zeros_like(n)

    def after_prefill(self):
        """Open the layout streams and close the roots."""
        for pg in range(len(self.P)):
            lay = self.s.open(self.sid_of[(pg, -1)], self.P[pg])
            self.sid_of[(pg, 0)] = lay
            self.tag_of[lay] = (pg, 0)
            self.count[(pg, 0)] = 0
            self.s.close(self.sid_of[(pg, -1)])

    def rows(self, row_ids) -> List[Tuple[int, int, int]]:
        """(page, stream, index of its new token) of each row of a step."""
        out = []
        for sid in row_ids:
            pg, c = self.tag_of[int(sid)]
            out.append((pg, c, self.count[(pg, c)]))
        return out

    def events(self, row_ids):
        """Apply the step's events after its launch (or commit)."""
        for sid in row_ids:
            pg, c = self.tag_of[int(sid)]
            self.count[(pg, c)] += 1
        for sid in row_ids:
            pg, c = self.tag_of[int(sid)]
            ev = self.decides[pg](self.step_no, c, c == 0)
            if c == 0 and ev == "fork":
                cid = self.next_c[pg]
                self.next_c[pg] += 1
                child = self.s.open(int(sid), self.count[(pg, 0)])
                self.sid_of[(pg, cid)] = child
                self.tag_of[child] = (pg, cid)
                self.count[(pg, cid)] = 0
            elif ev == "eos":
                self.s.close(int(sid))
        self.step_no += 1


def oracle_rows(prefix_lens, decides, max_steps: int):
    """Per page: (tags, {(c, i): mask row}) from the oracle's replay."""
    out = []
    for pg, P in enumerate(prefix_lens):
        tags, queries, _ = od.simulate_masked_parallel_decoding(P, decides[pg], max_steps=max_steps)
        out.append((tags, {(c, i): row for c, i, row in queries}))
    return out


def session_visible_tags(view, run: Alg1Run, row: int):
    """Cache positions (page, stream, index) the session's step tree lets
    row `row` see, by the tree's visibility rule (the oracle's helper applied
    to the session's tree)."""
    seg = view["seg"]
    nodes = [(int(g["parent"]), int(g["fork"]), int(g["len"]), int(g["q_len"])) for g in seg]
    sid = int(view["row_id"][row])
    s = int(np.nonzero(view["seg_id"] == sid)[0][0])
    p = nodes[s][2] - 1
    vis = od.visible_counts(nodes, s, p)
    tags = set()
    for t, cnt in vis.items():
        pg, c = run.tag_of[int(view["seg_id"][t])]
        for j in range(cnt):
            tags.add((pg, c, j))
    return tags
