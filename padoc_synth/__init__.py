"""Seeded synthetic inputs for PaDoc tree attention.

This module only draws random structure and random values.  It holds none of
the attention arithmetic and none of the tree-to-layout conversion: both the
HIP path and the CPU oracle consume what it produces, each with its own code.

Structures
----------
* ``Page``: one document page as the paper's packed sample ``[M | Y_1 .. Y_N]``
  (Appendix C, "Attention Backends"): a shared prefix ``X`` (image + prompt
  tokens), one layout stream forked at the end of the prefix, and content
  branches ``Y_k`` forked off the stream at offsets ``f_k``.  Every segment
  carries ``q_len``: its queries are its LAST ``q_len`` tokens.
* ``Node``: a generic tree segment ``(parent, fork, len, q_len)`` in packed
  order (parent index < own index, ``parent == -1`` for a page root).  Used for
  random trees deeper than the paper's three levels.

Draw order (all ``numpy.random.default_rng`` / PCG64, documented so any run is
reproducible from its seed) is given in each config function's docstring.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence

import numpy as np

__all__ = [
    "Branch", "Page", "Node", "Workload", "CONFIGS", "make_workload",
    "random_tree", "count_tokens", "count_queries", "count_blocks",
    "pages_as_dicts", "draw_normal", "draw_block_ids", "BLOCK",
]

BLOCK = 16  # paged KV block size (tokens) used by every paged workload


@dataclasses.dataclass(frozen=True)
class Branch:
    fork: int      # number of leading stream tokens the branch sees
    length: int    # tokens in the branch (position 0 = branch-start token)
    q_len: int     # queries = last q_len tokens of the branch


@dataclasses.dataclass(frozen=True)
class Page:
    prefix_len: int
    prefix_q: int
    stream_len: int
    stream_q: int
    branches: tuple  # tuple[Branch, ...], in packed order


@dataclasses.dataclass(frozen=True)
class Node:
    parent: int
    fork: int
    length: int
    q_len: int


@dataclasses.dataclass
class Workload:
    name: str
    kind: str                 # "forward" (packed) or "decode" (paged)
    pages: List[Page]
    num_heads_q: int
    num_heads_kv: int
    head_dim: int
    dtype: str                # "f32" or "bf16"
    block_size: int           # 0 = packed contiguous K/V, 16 = paged
    seed: int
    prescale: bool = False    # also multiply drawn Q/K/V by 1/sqrt(d)
    pool_bytes: int = 0       # paged: bytes per K (and per V) pool; 0 = decided by caller
    description: str = ""

    @property
    def softmax_scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)


# --------------------------------------------------------------------------
# Configurations (structure only)
# --------------------------------------------------------------------------

def _tiny_fp32_forward(seed: int) -> Workload:
    """1 page: prefix 256, stream 64, 4 branches of 32 tokens forking at stream
    offsets 8/24/40/56; Hq=4, Hkv=1, d=64, fp32; every token is a query.
    No random structure draws."""
    br = tuple(Branch(f, 32, 32) for f in (8, 24, 40, 56))
    page = Page(256, 256, 64, 64, br)
    return Workload("tiny_fp32_forward", "forward", [page], 4, 1, 64, "f32", 0, seed,
                    description="1 page P=256 S=64 4x32-token branches, fp32, packed forward")


def _single_page_decode(seed: int) -> Workload:
    """1 page: prefix 2048 (no queries), stream 256 with its newest token as
    the query, 16 live branches.  Draws: lengths L_k ~ U{16..256} (16 draws),
    then forks f_k ~ U{1..255} (16 draws, sorted ascending).  Forks stop one
    short of the stream length: the stream's newest token is appended in this
    step and is visible to the stream alone.  Every branch queries its newest
    token.  Hq=16, Hkv=2, d=128, bf16, paged (block 16)."""
    rng = np.random.default_rng(seed)
    S = 256
    L = rng.integers(16, 257, size=16)
    f = np.sort(rng.integers(1, S, size=16))
    br = tuple(Branch(int(a), int(b), 1) for a, b in zip(f, L))
    page = Page(2048, 0, S, 1, br)
    return Workload("single_page_decode", "decode", [page], 16, 2, 128, "bf16", BLOCK, seed,
                    pool_bytes=16 << 30,
                    description="1 page P=2048 S=256 16 branches L~U[16,256], 17 queries, paged bf16")


def _packed_forward_8pages(seed: int) -> Workload:
    """8 pages packed varlen, every token a query.  Per page, in this order:
    P ~ U{1024..4096}, S ~ U{128..512}, N ~ U{8..48}, forks f ~ U{1..S} (N
    draws, sorted), lengths L = clip(rint(lognormal(ln 80, 0.5)), 4, 1024)
    (N draws).  Hq=16, Hkv=2, d=128, bf16."""
    rng = np.random.default_rng(seed)
    pages = []
    for _ in range(8):
        P = int(rng.integers(1024, 4097))
        S = int(rng.integers(128, 513))
        N = int(rng.integers(8, 49))
        f = np.sort(rng.integers(1, S + 1, size=N))
        L = np.clip(np.rint(rng.lognormal(math.log(80.0), 0.5, size=N)), 4, 1024).astype(np.int64)
        br = tuple(Branch(int(a), int(b), int(b)) for a, b in zip(f, L))
        pages.append(Page(P, P, S, S, br))
    return Workload("packed_forward_8pages", "forward", pages, 16, 2, 128, "bf16", 0, seed,
                    description="8 pages P~U[1024,4096] S~U[128,512] N~U[8,48] L~logN(80,0.5), packed bf16")


def _concurrent_decode_64pages(seed: int) -> Workload:
    """64 pages, each: prefix 3072 (no queries), stream 256 (newest token is a
    query), 24 branches.  Per page, in this order: L ~ U{1..1024} (24 draws),
    f ~ U{1..255} (24 draws, sorted).  1536 branch + 64 stream queries.
    Hq=16, Hkv=2, d=128, bf16, paged; the pool is sized by the caller
    (the benchmark takes most of HBM)."""
    rng = np.random.default_rng(seed)
    S = 256
    pages = []
    for _ in range(64):
        L = rng.integers(1, 1025, size=24)
        f = np.sort(rng.integers(1, S, size=24))
        br = tuple(Branch(int(a), int(b), 1) for a, b in zip(f, L))
        pages.append(Page(3072, 0, S, 1, br))
    return Workload("concurrent_decode_64pages", "decode", pages, 16, 2, 128, "bf16", BLOCK, seed,
                    pool_bytes=0,
                    description="64 pages x (P=3072, S=256, 24 branches L~U[1,1024]), 1600 queries, paged bf16")


def _dense_page_mixed_step(seed: int) -> Workload:
    """1 page: prefix 8192 (no queries), stream 1024 (newest token a query),
    128 branches.  Draws: f ~ U{1..1023} (128 draws, sorted ascending), then
    L ~ U{64..2048} (96 draws).  The 96 earliest-forked branches are decoding
    (q_len 1); the 32 latest-forked ones were just created and extend 8 tokens
    in this launch (len 8, all 8 are queries).  353 query tokens in one
    launch.  Hq=28, Hkv=4, d=128, bf16, paged."""
    rng = np.random.default_rng(seed)
    S = 1024
    f = np.sort(rng.integers(1, S, size=128))
    L = rng.integers(64, 2049, size=96)
    br = [Branch(int(f[i]), int(L[i]), 1) for i in range(96)]
    br += [Branch(int(f[i]), 8, 8) for i in range(96, 128)]
    page = Page(8192, 0, S, 1, tuple(br))
    return Workload("dense_page_mixed_step", "decode", [page], 28, 4, 128, "bf16", BLOCK, seed,
                    pool_bytes=16 << 30,
                    description="1 page P=8192 S=1024 128 branches (96 decoding + 32 new 8-token forks), 353 queries, Hq=28 Hkv=4")


CONFIGS = {
    "tiny_fp32_forward": _tiny_fp32_forward,
    "single_page_decode": _single_page_decode,
    "packed_forward_8pages": _packed_forward_8pages,
    "concurrent_decode_64pages": _concurrent_decode_64pages,
    "dense_page_mixed_step": _dense_page_mixed_step,
}


def make_workload(name: str, seed: int = 0) -> Workload:
    return CONFIGS[name](seed)


# --------------------------------------------------------------------------
# Random generic trees (tests)
# --------------------------------------------------------------------------

def random_tree(seed: int, n_pages: int = 2, max_depth: int = 5, max_children: int = 3,
                max_len: int = 6, q_mode: str = "all", max_nodes: int = 40) -> List[Node]:
    """Random segment tree in packed order (depth-first per page).

    Draw order per node: ``len ~ U{1..max_len}``; for non-roots ``fork ~
    U{0..len(parent)}``; ``q_len`` is ``len`` (q_mode "all"), ``U{0..len}``
    ("some") or ``min(len, U{0..2})`` ("tail"); then the child count
    ``~ U{0..max_children}`` (0 at ``max_depth``).
    """
    rng = np.random.default_rng(seed)
    nodes: List[Node] = []

    def q_of(n: int) -> int:
        if q_mode == "all":
            return n
        if q_mode == "some":
            return int(rng.integers(0, n + 1))
        return int(min(n, rng.integers(0, 3)))

    def grow(parent: int, depth: int) -> None:
        if len(nodes) >= max_nodes:
            return
        n = int(rng.integers(1, max_len + 1))
        fork = 0 if parent < 0 else int(rng.integers(0, nodes[parent].length + 1))
        me = len(nodes)
        nodes.append(Node(parent, fork, n, q_of(n)))
        kids = 0 if depth >= max_depth else int(rng.integers(0, max_children + 1))
        for _ in range(kids):
            grow(me, depth + 1)

    for _ in range(n_pages):
        grow(-1, 1)
    return nodes


# --------------------------------------------------------------------------
# Counting helpers (sizes of the arrays to draw)
# --------------------------------------------------------------------------

def _page_lengths(p: Page):
    yield p.prefix_len, p.prefix_q
    yield p.stream_len, p.stream_q
    for b in p.branches:
        yield b.length, b.q_len


def count_tokens(pages: Sequence[Page]) -> int:
    return int(sum(n for p in pages for n, _ in _page_lengths(p)))


def count_queries(pages: Sequence[Page]) -> int:
    return int(sum(q for p in pages for _, q in _page_lengths(p)))


def count_blocks(pages: Sequence[Page], block: int = BLOCK) -> int:
    return int(sum(-(-n // block) for p in pages for n, _ in _page_lengths(p)))


def pages_as_dicts(pages: Sequence[Page]) -> list:
    return [dataclasses.asdict(p) for p in pages]


# --------------------------------------------------------------------------
# Values
# --------------------------------------------------------------------------

def draw_normal(shape, seed: int, stream: int, dtype: str = "bf16", device: str = "cpu",
                prescale: Optional[float] = None):
    """N(0,1) samples as a torch tensor of ``shape``.

    fp32 samples are drawn first (CPU: numpy PCG64 seeded with
    ``[seed, stream]``; CUDA: torch's device generator seeded with
    ``seed * 1000003 + stream``), optionally multiplied by ``prescale``, then
    rounded to bf16 with round-to-nearest-even when ``dtype == "bf16"``.
    Q, K and V use streams 1, 2 and 3.
    """
    import torch
    if device == "cpu":
        rng = np.random.default_rng([seed, stream])
        x = torch.from_numpy(rng.standard_normal(size=tuple(shape), dtype=np.float32))
    else:
        g = torch.Generator(device=device)
        g.manual_seed(seed * 1000003 + stream)
        x = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    if prescale is not None:
        x = x * prescale
    if dtype == "bf16":
        return x.to(torch.bfloat16)
    return x


def draw_block_ids(n_needed: int, n_pool: int, seed: int) -> np.ndarray:
    """``n_needed`` distinct physical block ids drawn uniformly without
    replacement from ``[0, n_pool)`` (numpy PCG64 seeded ``[seed, 4]``), in
    draw order: the i-th logical block gets the i-th id."""
    if n_needed > n_pool:
        raise ValueError(f"pool of {n_pool} blocks cannot hold {n_needed}")
    rng = np.random.default_rng([seed, 4])
    if n_pool <= 4 * n_needed or n_pool <= (1 << 20):
        return rng.permutation(n_pool)[:n_needed].astype(np.int32)
    # Large pool: rejection sampling keeps memory O(n_needed).
    out = np.empty(0, dtype=np.int64)
    while out.size < n_needed:
        cand = rng.integers(0, n_pool, size=2 * (n_needed - out.size) + 16)
        out = np.concatenate([out, cand])
        _, first = np.unique(out, return_index=True)
        out = out[np.sort(first)]
    return out[:n_needed].astype(np.int32)
