"""Seeded synthetic workloads shaped like the paper's FacTool / RAG pipelines.

This module only draws trees, arrival orders and payloads. It holds none of the
routing or aggregation arithmetic: it never packs keys, hashes, sorts by ancestry,
checks completion or pools payloads. Both the CPU oracle and the HIP path receive
the same arrays from here.

Representation (nested ancestry, Section 4.2 of the paper): a fragment (leaf) at
depth ``d`` carries one int32 tag per level, level 1 being the root request and
level ``d`` the leaf.

* ``path[l-1][i]``: tag of fragment ``i`` at level ``l``. Level 1 is the request id;
  levels >= 2 are the 0-based index of the element within its parent's stream
  (the index that a pmap entry pushes).
* ``fan[l-1][i]`` for ``l = 1..d-1``: declared child count of the fragment's
  level-``l`` ancestor (the end-of-output information of Section 3.1, carried by
  every descendant).
* ``payload_i32[i]``: a token id or a document id.
* ``payload_f32[i, :]``: an embedding row.

Arrays are level-major and in arrival order. Trees are drawn with numpy's PCG64
from ``seed``; arrival permutations and fp32 payloads are drawn with torch
generators seeded from ``seed`` on the device the caller asks for, which keeps the
64M-fragment workload fast to build.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, List, Optional, Sequence

import numpy as np
import torch

SEED_BASE = 2403043110


@dataclass
class Workload:
    """One synthetic batch (or one whole stream, cut into steps)."""

    name: str
    bits: tuple                 # key bit width per level, level 1 first
    route_level: int            # Lr (0 = one destination)
    num_dest: int               # D
    agg_level: int              # La
    op: str                     # "concat" or "mean"
    dim: int                    # payload row width (1 for concat)
    mask_level: int             # Lm (0 = no mask)
    path: torch.Tensor          # int32 [d][n]
    fan: torch.Tensor           # int32 [d-1][n]
    payload_i32: Optional[torch.Tensor] = None   # int32 [n]
    payload_f32: Optional[torch.Tensor] = None   # float32 [n][dim]
    step: int = 0               # fragments per stream step (0 = one batch)
    info: dict = field(default_factory=dict)

    @property
    def depth(self) -> int:
        return len(self.bits)

    @property
    def n(self) -> int:
        return int(self.path.shape[1])


# ----------------------------------------------------------------------------
# tree construction (canonical depth-first order)
# ----------------------------------------------------------------------------

def expand_tree(level_fans: Sequence[np.ndarray], root_ids: np.ndarray):
    """Leaves of a tree given each level's child counts, in depth-first order.

    ``level_fans[l-1]`` holds the child count of every level-``l`` node in
    depth-first order (``l = 1..d-1``); ``len(level_fans[l]) == level_fans[l-1].sum()``.
    Returns ``path`` int32 [d][n_leaves] and ``fan`` int32 [d-1][n_leaves].
    """
    d = len(level_fans) + 1
    counts = [len(root_ids)] + [int(f.sum()) for f in level_fans]
    for l in range(1, d - 1):
        assert len(level_fans[l]) == counts[l], "inconsistent level sizes"
    # parent index and child index of every node at levels 2..d
    parent = [None]
    child = [None]
    for l in range(d - 1):
        f = level_fans[l].astype(np.int64)
        par = np.repeat(np.arange(len(f), dtype=np.int64), f)
        start = np.cumsum(f) - f
        child.append((np.arange(counts[l + 1], dtype=np.int64) - start[par]).astype(np.int32))
        parent.append(par)
    n = counts[-1]
    path = np.empty((d, n), dtype=np.int32)
    fan = np.empty((d - 1, n), dtype=np.int32)
    anc = np.arange(n, dtype=np.int64)          # ancestor index at the current level
    for l in range(d - 1, -1, -1):              # 0-based level index
        if l == 0:
            path[0] = root_ids[anc]
        else:
            path[l] = child[l][anc]
        if l < d - 1:
            fan[l] = level_fans[l][anc]
        if l > 0:
            anc = parent[l][anc]
    return path, fan


def draw_topdown(rng: np.random.Generator, root_ids: np.ndarray,
                 samplers: Sequence[Callable[[np.random.Generator, int], np.ndarray]]):
    """Top-down tree: ``samplers[l-1](rng, k)`` draws child counts of the k level-l nodes."""
    fans = []
    k = len(root_ids)
    for s in samplers:
        f = np.asarray(s(rng, k), dtype=np.int32)
        assert f.min() >= 1
        fans.append(f)
        k = int(f.sum())
    return fans


def uniform_int(lo: int, hi: int):
    """Integer-inclusive uniform U{lo..hi}."""
    return lambda rng, k: rng.integers(lo, hi + 1, size=k)


def const_int(c: int):
    return lambda rng, k: np.full(k, c, dtype=np.int64)


def zt_poisson(lam: float, cap: int):
    """Zero-truncated Poisson, also truncated above ``cap``, both by resampling."""
    def f(rng, k):
        out = rng.poisson(lam, size=k)
        bad = (out < 1) | (out > cap)
        while bad.any():
            out[bad] = rng.poisson(lam, size=int(bad.sum()))
            bad = (out < 1) | (out > cap)
        return out
    return f


def geometric(p: float, cap: int):
    """Geometric on {1, 2, ...} with mean 1/p, truncated above ``cap`` by resampling."""
    def f(rng, k):
        out = rng.geometric(p, size=k)
        bad = out > cap
        while bad.any():
            out[bad] = rng.geometric(p, size=int(bad.sum()))
            bad = out > cap
        return out
    return f


def zipf_trunc(rng: np.random.Generator, s: float, cap: int, k: int) -> np.ndarray:
    """Zipf(s) truncated to 1..cap by rejection."""
    out = np.empty(0, dtype=np.int64)
    while len(out) < k:
        z = rng.zipf(s, size=max(2 * (k - len(out)), 1024))
        out = np.concatenate([out, z[z <= cap]])
    return out[:k]


def draw_until(rng: np.random.Generator, s: float, cap: int, total: int) -> np.ndarray:
    """Zipf child counts drawn until they sum to ``total`` exactly (last one cut)."""
    parts = []
    acc = 0
    while acc < total:
        z = zipf_trunc(rng, s, cap, max(1024, int(1.2 * (total - acc) / 150) + 16))
        parts.append(z)
        acc += int(z.sum())
    f = np.concatenate(parts)
    c = np.cumsum(f)
    last = int(np.searchsorted(c, total))      # first index with c >= total
    f = f[: last + 1].copy()
    f[-1] -= int(c[last] - total)
    assert f.min() >= 1 and int(f.sum()) == total
    return f


def distinct_ids(rng: np.random.Generator, k: int) -> np.ndarray:
    """k distinct random non-negative int32 request ids."""
    ids = np.unique(rng.integers(0, 2**31, size=2 * k + 16, dtype=np.int64))
    ids = rng.permutation(ids)[:k]
    assert len(ids) == k
    return ids.astype(np.int32)


# ----------------------------------------------------------------------------
# helpers
# ----------------------------------------------------------------------------

def _torch_gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) & ((1 << 63) - 1))
    return g


def _to_dev(a: np.ndarray, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def shuffle_arrival(path, fan, extra, seed: int, device):
    """Seeded uniform shuffle of the leaves (arrival order)."""
    n = path.shape[1]
    g = _torch_gen(device, seed)
    order = torch.randperm(n, generator=g, device=device)
    p = _to_dev(path, device)[:, order].contiguous()
    f = _to_dev(fan, device)[:, order].contiguous()
    e = None if extra is None else _to_dev(extra, device)[order].contiguous()
    return p, f, e, order


def randn_rows(n: int, dim: int, seed: int, device) -> torch.Tensor:
    g = _torch_gen(device, seed)
    return torch.randn(n, dim, generator=g, device=device, dtype=torch.float32)


def tokens(rng: np.random.Generator, n: int) -> np.ndarray:
    return rng.integers(0, 50000, size=n).astype(np.int32)


# ----------------------------------------------------------------------------
# the benchmarked workloads
# ----------------------------------------------------------------------------

def tiny_tree(device="cpu", seed: int = SEED_BASE + 1) -> Workload:
    """Tiny depth-4 tree: query / doc / sentence / token, concat at sentence level."""
    rng = np.random.default_rng(seed)
    roots = distinct_ids(rng, 64)
    fans = draw_topdown(rng, roots, [uniform_int(1, 4), uniform_int(1, 8), uniform_int(1, 16)])
    path, fan = expand_tree(fans, roots)
    tok = tokens(rng, path.shape[1])
    p, f, t, _ = shuffle_arrival(path, fan, tok, seed + 101, device)
    return Workload("tiny_concat", (31, 2, 3, 4), 1, 8, 3, "concat", 1, 0, p, f,
                    payload_i32=t)


def factool_fans(rng, roots):
    """query / claim / search query / doc / sentence child counts."""
    return draw_topdown(rng, roots, [uniform_int(1, 8), uniform_int(1, 3), const_int(5),
                                     zt_poisson(20.0, 255)])


def doc_ids_per_sentence(rng, fans) -> np.ndarray:
    """A corpus id (uniform in [0, 2^31)) per document, repeated over its sentences."""
    ndocs = len(fans[3])
    ids = rng.integers(0, 2**31, size=ndocs).astype(np.int32)
    return np.repeat(ids, fans[3].astype(np.int64))


def factool_batch(device="cpu", seed: int = SEED_BASE + 2, queries: int = 1024) -> Workload:
    """FacTool-shaped depth-5 tree; mean-pool 768-d sentence vectors per document.

    The follow-on stage (concat of document ids per claim) consumes the records the
    first stage emits; see ``FACTOOL_CLAIM_STAGE``.
    """
    rng = np.random.default_rng(seed)
    roots = distinct_ids(rng, queries)
    fans = factool_fans(rng, roots)
    path, fan = expand_tree(fans, roots)
    docid = doc_ids_per_sentence(rng, fans)
    p, f, t, _ = shuffle_arrival(path, fan, docid, seed + 101, device)
    x = randn_rows(path.shape[1], 768, seed + 202, device)
    return Workload("factool_mean_concat", (31, 3, 2, 3, 8), 2, 32, 4, "mean", 768, 0,
                    p, f, payload_i32=t, payload_f32=x)


# second stage of the FacTool batch and stream: records of level-4 groups (depth-4 keys)
FACTOOL_CLAIM_STAGE = dict(bits=(31, 3, 2, 3), route_level=2, num_dest=32, agg_level=2,
                       op="concat", dim=1, mask_level=0)


def token_stream(device="cpu", seed: int = SEED_BASE + 3, generators: int = 256,
            sentences: int = 64, step: int = 4096) -> Workload:
    """Token stream: request / sentence / token, round-robin over generators."""
    rng = np.random.default_rng(seed)
    roots = distinct_ids(rng, generators)
    fans = draw_topdown(rng, roots, [const_int(sentences), geometric(1.0 / 24.0, 4095)])
    path, fan = expand_tree(fans, roots)
    tok = tokens(rng, path.shape[1])
    # per generator, tokens are emitted in depth-first order; one token per
    # generator per tick, generators in index order within a tick
    per_gen = np.add.reduceat(fans[1].astype(np.int64), np.arange(0, len(fans[1]), sentences))
    gen = np.repeat(np.arange(generators, dtype=np.int64), per_gen)
    tick = np.arange(path.shape[1], dtype=np.int64) - np.repeat(np.cumsum(per_gen) - per_gen, per_gen)
    order = np.lexsort((gen, tick))
    w = Workload("token_stream", (31, 6, 12), 2, 64, 2, "concat", 1, 0,
                 _to_dev(path[:, order], device), _to_dev(fan[:, order], device),
                 payload_i32=_to_dev(tok[order], device), step=step)
    w.info["generators"] = generators
    return w


DELIM_TOKEN = 50000   # a token id outside the range tokens() draws: a sentence end


def text_tokens(seed: int, n: int, p_delim: float, delim: int = DELIM_TOKEN) -> np.ndarray:
    """Token ids of n stream positions, each the delimiter with probability p_delim."""
    rng = np.random.default_rng(seed)
    t = tokens(rng, n)
    t[rng.random(n) < p_delim] = delim
    return t


@dataclass
class TextStreams:
    """Token streams at a pmap entry: one stream per level-(d-1) node (the parent),
    a token's leaf tag being its position in the stream."""

    bits: tuple                 # input layout (..., parent, position)
    seg_bits: int               # bits of the segment level the split pushes
    tok_bits: int               # bits of the token index within a segment
    delim: int
    path: torch.Tensor          # int32 [d][n], arrival order
    fan: torch.Tensor           # int32 [d-1][n]; row d-2 is the stream length
    tokens: torch.Tensor        # int32 [n]
    tree_path: torch.Tensor     # int32 [d+1][n]: tags the position was written from (-1 for delimiters)
    tree_fan: torch.Tensor      # int32 [d][n]: counts of those nodes (0 for delimiters)

    @property
    def n(self) -> int:
        return int(self.path.shape[1])


def token_stream_text(device="cpu", seed: int = SEED_BASE + 3, generators: int = 256,
                 sentences: int = 64) -> TextStreams:
    """The token streams the token stream's sentences come from: every generator writes its
    sentences as one stream, each sentence followed by a delimiter token, and a pmap
    entry cuts the streams back into sentences. Same draws as token_stream (same seed,
    same generators: the same requests, sentence lengths and token ids).
    Layout (request 31 bits, position 18 bits) -> (request, sentence 6, token 12);
    arrival round-robin over generators, in order within each. The streams are laid
    out with torch on ``device`` (the draws stay numpy)."""
    rng = np.random.default_rng(seed)
    roots = distinct_ids(rng, generators)
    fans = draw_topdown(rng, roots, [const_int(sentences), geometric(1.0 / 24.0, 4095)])
    L_np = fans[1].astype(np.int64)                    # sentence lengths, request-major
    tok = _to_dev(tokens(rng, int(L_np.sum())), device)
    L = _to_dev(L_np, device)
    rt = _to_dev(roots, device)
    width = L + 1                                      # each sentence and its delimiter
    rlen = width.view(generators, sentences).sum(1)
    n = int(rlen.sum())
    # request-major concatenation of the streams
    g = torch.arange(n, device=device)
    req = torch.repeat_interleave(torch.arange(generators, device=device), rlen)
    pos = g - torch.repeat_interleave(torch.cumsum(rlen, 0) - rlen, rlen)
    assert int(pos.max()) < (1 << 18)
    sent = torch.repeat_interleave(torch.arange(len(L_np), device=device), width)   # global sentence index
    idx = g - torch.repeat_interleave(torch.cumsum(width, 0) - width, width)        # index within the sentence
    del g
    is_delim = idx == L[sent]
    tk = torch.full((n,), DELIM_TOKEN, dtype=torch.int32, device=device)
    tk[~is_delim] = tok
    order = torch.argsort(pos, stable=True)            # tick-major, generators in index order
    req, pos, sent, idx, is_delim, tk = req[order], pos[order], sent[order], idx[order], is_delim[order], tk[order]
    p2 = torch.stack([rt[req], pos.to(torch.int32)])
    f1 = rlen[req].to(torch.int32)[None, :]
    tp = torch.stack([rt[req], (sent % sentences).to(torch.int32), idx.to(torch.int32)])
    tp[:, is_delim] = -1
    tf = torch.stack([torch.full((n,), sentences, dtype=torch.int32, device=device), L[sent].to(torch.int32)])
    tf[:, is_delim] = 0
    return TextStreams((31, 18), 6, 12, DELIM_TOKEN, p2.contiguous(), f1.contiguous(), tk, tp, tf)


def random_text(seed: int, depth: int, roots: int, max_fan: Sequence[int], bits: Sequence[int], p_delim: float,
                drop: float = 0.0, seg_bits: int = 8, tok_bits: int = 10, delim: int = DELIM_TOKEN):
    """Random token streams: a depth-``depth`` tree whose leaf tags are stream
    positions (U{1..max_fan[-1]} tokens per stream), shuffled, optionally with a
    fraction of tokens dropped (incomplete streams). Returns (path, fan, tokens)
    as numpy arrays in arrival order."""
    path, fan = random_tree(seed, depth, roots, max_fan, bits)
    tok = text_tokens(seed + 1, path.shape[1], p_delim, delim)
    if drop:
        path, fan, keep = drop_leaves(path, fan, drop, seed + 2)
        tok = tok[keep]
    (path, fan, tok), _ = permute([path, fan, tok], seed + 3)
    return path, fan, tok


def factool_stream(device="cpu", seed: int = SEED_BASE + 4, steps: int = 10000, step: int = 4096,
            target_frac: float = 0.30, ring_steps: int = 256) -> Workload:
    """FacTool-shaped trees as a continuous windowed stream of ``steps`` x ``step``.

    Queries are appended back to back; the leaves of a query are spread uniformly
    over a window of ``W`` fragments starting at the query's cumulative offset.
    ``W`` is chosen by bisection so that about ``target_frac`` of the document
    groups have their first and last sentence at least 10 steps apart. Payload rows
    repeat with period ``ring_steps`` steps (``payload_f32`` holds the ring only).
    """
    total = steps * step
    rng = np.random.default_rng(seed)
    # enough queries to cover the stream plus one window of spill-over
    est = int(total / 900 * 1.15) + 64
    roots = distinct_ids(rng, est)
    fans = factool_fans(rng, roots)
    path, fan = expand_tree(fans, roots)
    docid = doc_ids_per_sentence(rng, fans)
    n = path.shape[1]
    assert n > total, "not enough queries drawn"
    qsize = _leaves_per_root(fans)
    qoff = np.cumsum(qsize) - qsize
    qidx = np.repeat(np.arange(est), qsize)
    u = rng.random(n)
    doc_start = np.cumsum(fans[3].astype(np.int64)) - fans[3]

    def frac(W):
        s = ((qoff[qidx] + u * W) // step).astype(np.int64)
        lo = np.minimum.reduceat(s, doc_start)
        hi = np.maximum.reduceat(s, doc_start)
        ok = hi < steps
        return float(((hi - lo)[ok] >= 10).mean())

    lo_w, hi_w = 8.0 * step, 16.0 * step
    for _ in range(14):
        mid = 0.5 * (lo_w + hi_w)
        if frac(mid) < target_frac:
            lo_w = mid
        else:
            hi_w = mid
    W = 0.5 * (lo_w + hi_w)
    pos = qoff[qidx] + u * W
    g = torch.from_numpy(pos).to(device)
    order = torch.argsort(g, stable=True)[:total]
    p = _to_dev(path, device)[:, order].contiguous()
    f = _to_dev(fan, device)[:, order].contiguous()
    t = _to_dev(docid, device)[order].contiguous()
    x = randn_rows(ring_steps * step, 768, seed + 202, device)
    w = Workload("factool_stream", (31, 3, 2, 3, 8), 2, 32, 4, "mean", 768, 0, p, f,
                 payload_i32=t, payload_f32=x, step=step)
    w.info.update(window=W, ring_steps=ring_steps, steps=steps, calibrated_frac=frac(W))
    return w


def _leaves_per_root(fans):
    """Leaf count under each root (helper for the windowed stream)."""
    c = fans[-1].astype(np.int64)            # leaves under each level-(d-1) node
    for f in reversed(fans[:-1]):            # f: child counts one level up
        f = f.astype(np.int64)
        c = np.add.reduceat(c, np.cumsum(f) - f)
    return c


def zipf_tree_fans(seed: int = SEED_BASE + 5, leaves: int = 1 << 26, s: float = 1.2,
                 cap: int = 4096, depth: int = 6):
    """Skewed depth-6 tree built bottom-up from truncated Zipf child counts."""
    rng = np.random.default_rng(seed)
    fans: List[np.ndarray] = []
    total = leaves
    for _ in range(depth - 1):
        f = draw_until(rng, s, cap, total)
        fans.append(f.astype(np.int32))
        total = len(f)
    fans.reverse()
    roots = np.arange(total, dtype=np.int32)     # dense 0..R-1
    return fans, roots


def zipf_tree(device="cpu", seed: int = SEED_BASE + 5, leaves: int = 1 << 26,
            with_payload: bool = True) -> Workload:
    """Skewed Zipf depth-6 tree, 128-d mean at level 4, completion mask at level 2."""
    fans, roots = zipf_tree_fans(seed, leaves)
    path, fan = expand_tree(fans, roots)
    p, f, _, _ = shuffle_arrival(path, fan, None, seed + 101, device)
    del path, fan
    x = randn_rows(leaves, 128, seed + 202, device) if with_payload else None
    w = Workload("zipf_mean_mask", (3, 12, 12, 12, 12, 12), 4, 256, 4, "mean", 128, 2,
                 p, f, payload_f32=x)
    w.info["level_nodes"] = [len(roots)] + [int(x.sum()) for x in fans]
    return w


# ----------------------------------------------------------------------------
# small random trees for parity and edge-case tests
# ----------------------------------------------------------------------------

def random_tree(seed: int, depth: int, roots: int, max_fan: Sequence[int], bits: Sequence[int],
                dense_roots: bool = False):
    """Top-down tree with U{1..max_fan[l]} children; returns (path, fan) in DFS order."""
    rng = np.random.default_rng(seed)
    if dense_roots:
        ids = np.arange(roots, dtype=np.int32)
    else:
        space = min(2 ** bits[0], 1 << 31)
        ids = np.unique(rng.integers(0, space, size=4 * roots + 8))
        ids = rng.permutation(ids)[:roots]
        assert len(ids) == roots, "id space too small for distinct roots"
        ids = ids.astype(np.int32)
    fans = draw_topdown(rng, ids, [uniform_int(1, m) for m in max_fan])
    return expand_tree(fans, ids)


def drop_leaves(path, fan, frac: float, seed: int):
    """Remove a seeded fraction of leaves (makes some groups incomplete)."""
    rng = np.random.default_rng(seed)
    keep = rng.random(path.shape[1]) >= frac
    return path[:, keep], fan[:, keep], keep


def permute(arrs, seed: int):
    """Apply one seeded permutation to the last axis of several numpy arrays."""
    n = arrs[0].shape[-1]
    order = np.random.default_rng(seed).permutation(n)
    return [None if a is None else a[..., order] for a in arrs], order
