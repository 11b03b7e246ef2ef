"""Seeded synthetic graph generators and canonical in-CSR construction.

These produce the *inputs* of a GNN layer (the graph structure of the
layer's problem statement: an adjacency matrix handed over as a
destination-major CSR).  Nothing here computes any stage of the message
passing layer; both the CPU oracle and the GPU path consume what this module
returns.

Generators:
  * ``er_directed``      Erdos-Renyi G(n, M) over distinct ordered pairs u != v.
  * ``ba_undirected``    Barabasi-Albert preferential attachment (m edges per
                         new vertex, distinct targets, degree-list sampling).
  * ``rmat``             R-MAT recursive quadrant sampling; every sample kept
                         (multi-edges and generated self-loops included).
  * ``torus_rgg``        random geometric graph on the unit torus.
  * ``to_in_csr``        canonical destination-major CSR, rows ordered by
                         (dst), entries within a row by (src, generation order).
"""
from __future__ import annotations

import concurrent.futures as _cf
import os

import numpy as np

MASTER_SEED = 200900804


def seed_seq(*key: int) -> np.random.SeedSequence:
    """The seed of one input stream: master seed plus a spawn key."""
    return np.random.SeedSequence(MASTER_SEED, spawn_key=tuple(int(k) for k in key))


def rng_for(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed_seq(*key)))


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


# --------------------------------------------------------------------------
# Erdos-Renyi G(n, M), directed, distinct ordered pairs, no self-loops
# --------------------------------------------------------------------------
def er_directed(n: int, m: int, rng: np.random.Generator):
    """M distinct ordered pairs (u, v), u != v, uniformly among n(n-1)."""
    total = n * (n - 1)
    if m > total:
        raise ValueError("too many edges for G(n, M)")
    idx = rng.choice(total, size=m, replace=False)
    u = idx // (n - 1)
    r = idx % (n - 1)
    v = r + (r >= u)  # skip the diagonal
    return u.astype(np.int64), v.astype(np.int64)


# --------------------------------------------------------------------------
# Barabasi-Albert
# --------------------------------------------------------------------------
def ba_undirected(n: int, m: int, rng: np.random.Generator, m0: int | None = None):
    """Preferential attachment: vertex t >= m0 links to m distinct earlier
    vertices chosen with probability proportional to degree.

    The first new vertex links to all m0 seed vertices (they have degree 0).
    Returns each undirected edge once as (new vertex, target).
    """
    m0 = m if m0 is None else m0
    if m0 < m:
        raise ValueError("m0 must be >= m")
    src = np.empty((n - m0) * m, dtype=np.int64)
    dst = np.empty((n - m0) * m, dtype=np.int64)
    # degree list: every endpoint of every edge appears once
    deglist = np.empty(2 * (n - m0) * m, dtype=np.int64)
    nd = 0
    k = 0
    for t in range(m0, n):
        if t == m0:
            targets = np.arange(m0 - m, m0, dtype=np.int64)
        else:
            chosen: list[int] = []
            seen = set()
            while len(chosen) < m:
                draw = deglist[rng.integers(0, nd, size=2 * m)]
                for x in draw.tolist():
                    if x not in seen:
                        seen.add(x)
                        chosen.append(x)
                        if len(chosen) == m:
                            break
            targets = np.asarray(chosen, dtype=np.int64)
        src[k:k + m] = t
        dst[k:k + m] = targets
        k += m
        deglist[nd:nd + m] = targets
        deglist[nd + m:nd + 2 * m] = t
        nd += 2 * m
    return src, dst


# --------------------------------------------------------------------------
# R-MAT
# --------------------------------------------------------------------------
def _rmat_chunk(scale, count, a, b, c, ss):
    rng = np.random.Generator(np.random.PCG64(ss))
    src = np.zeros(count, dtype=np.int32)
    dst = np.zeros(count, dtype=np.int32)
    ab = np.float32(a + b)
    abc = np.float32(a + b + c)
    fa = np.float32(a)
    q = np.empty(count, dtype=np.float32)
    for _ in range(scale):
        rng.random(out=q, dtype=np.float32)
        sbit = q >= ab                      # quadrants c, d: source bit 1
        dbit = (q >= fa) & (q < ab)         # quadrant b: destination bit 1
        dbit |= q >= abc                    # quadrant d: destination bit 1
        src <<= 1
        dst <<= 1
        src |= sbit
        dst |= dbit
    return src, dst


def rmat(scale: int, n_edges: int, a: float, b: float, c: float, key: tuple,
         chunk: int = 1 << 22):
    """R-MAT: each edge descends ``scale`` levels; at each level it picks
    quadrant a=(0,0), b=(0,1), c=(1,0), d=(1,1) for the (source bit,
    destination bit).  No noise.  Chunks use independent child seeds so the
    result does not depend on the thread count."""
    nchunks = (n_edges + chunk - 1) // chunk
    src = np.empty(n_edges, dtype=np.int32)
    dst = np.empty(n_edges, dtype=np.int32)

    def work(i):
        lo = i * chunk
        hi = min(n_edges, lo + chunk)
        s, d = _rmat_chunk(scale, hi - lo, a, b, c, seed_seq(*key, i))
        src[lo:hi] = s
        dst[lo:hi] = d

    with _cf.ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(work, range(nchunks)))
    return src, dst


# --------------------------------------------------------------------------
# Random geometric graph on the unit torus
# --------------------------------------------------------------------------
def torus_rgg(n: int, radius: float, rng: np.random.Generator):
    """n uniform points on the unit torus; an undirected edge joins every
    pair at (periodic) distance < radius.  Returns each pair once (i < j)."""
    from scipy.spatial import cKDTree

    pts = rng.random((n, 2))
    tree = cKDTree(pts, boxsize=1.0)
    pairs = tree.query_pairs(radius, output_type="ndarray")
    pairs = pairs[np.lexsort((pairs[:, 1], pairs[:, 0]))]
    return pairs[:, 0].astype(np.int64), pairs[:, 1].astype(np.int64)


# --------------------------------------------------------------------------
# Edge-list transforms
# --------------------------------------------------------------------------
def symmetrise(src, dst):
    """Store every undirected edge in both directions."""
    return np.concatenate([src, dst]), np.concatenate([dst, src])


def add_self_loops(src, dst, n):
    loops = np.arange(n, dtype=src.dtype)
    return np.concatenate([src, loops]), np.concatenate([dst, loops])


def relabel(src, dst, perm, chunk: int = 1 << 22):
    """Rename vertex x to perm[x] (threaded over edge chunks)."""
    perm = np.asarray(perm)
    out_s = np.empty(src.shape, dtype=src.dtype)
    out_d = np.empty(dst.shape, dtype=dst.dtype)

    def work(lo):
        hi = min(src.shape[0], lo + chunk)
        out_s[lo:hi] = perm[src[lo:hi]]
        out_d[lo:hi] = perm[dst[lo:hi]]

    with _cf.ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(work, range(0, src.shape[0], chunk)))
    return out_s, out_d


# --------------------------------------------------------------------------
# Canonical in-CSR
# --------------------------------------------------------------------------
def to_in_csr(num_dst: int, src, dst, num_src: int | None = None,
              want_eid: bool = False):
    """Destination-major CSR of an edge list.

    Row v lists the sources of v's in-edges, ordered by (source id, position
    in the edge list).  Returns ``row_ptr`` (int32, num_dst+1), ``col_idx``
    (int32, E) and, if asked, ``eid`` (int64, E): the edge-list position of
    each CSR entry.  Large inputs without ``want_eid`` take a threaded
    bucket sort that yields the same arrays (entries with equal (dst, src)
    are indistinguishable there).
    """
    num_src = num_dst if num_src is None else num_src
    src = np.asarray(src)
    dst = np.asarray(dst)
    E = src.shape[0]
    if E >= 2 ** 31:
        raise ValueError("edge count must fit int32")
    sbits = max(1, int(num_src - 1).bit_length())
    if not want_eid and E >= (1 << 22):
        return _csr_large(num_dst, sbits, src, dst)
    key = (dst.astype(np.int64) << sbits) | src.astype(np.int64)
    order = np.argsort(key, kind="stable")
    skey = key[order]
    col_idx = (skey & ((1 << sbits) - 1)).astype(np.int32)
    counts = np.bincount(skey >> sbits, minlength=num_dst).astype(np.int64)
    row_ptr = np.zeros(num_dst + 1, dtype=np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    out = (row_ptr.astype(np.int32), col_idx)
    if want_eid:
        out = out + (order.astype(np.int64),)
    return out


def _csr_large(num_dst, sbits, src, dst, nbuckets=64, chunk=1 << 22):
    E = src.shape[0]
    dbits = max(1, int(num_dst - 1).bit_length())
    shift = sbits + max(0, dbits - 6)  # bucket = top 6 bits of dst
    starts = list(range(0, E, chunk))
    parts = [None] * len(starts)
    counts = np.zeros((len(starts), nbuckets), dtype=np.int64)
    rowcnt = [None] * len(starts)

    def pass1(i):
        lo = starts[i]
        hi = min(E, lo + chunk)
        k = (dst[lo:hi].astype(np.int64) << sbits) | src[lo:hi].astype(np.int64)
        b = (k >> shift).astype(np.uint8)
        o = np.argsort(b, kind="stable")
        parts[i] = k[o]
        counts[i] = np.bincount(b, minlength=nbuckets)
        rowcnt[i] = np.bincount(dst[lo:hi], minlength=num_dst)

    with _cf.ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(pass1, range(len(starts))))
    bsize = counts.sum(axis=0)
    bstart = np.zeros(nbuckets + 1, dtype=np.int64)
    np.cumsum(bsize, out=bstart[1:])
    # position of chunk i's run of bucket k: bucket start + earlier chunks
    off = bstart[:-1][None, :] + np.cumsum(counts, axis=0) - counts
    out = np.empty(E, dtype=np.int64)

    def pass2(i):
        cs = np.zeros(nbuckets + 1, dtype=np.int64)
        np.cumsum(counts[i], out=cs[1:])
        for k in range(nbuckets):
            n = counts[i, k]
            if n:
                out[off[i, k]:off[i, k] + n] = parts[i][cs[k]:cs[k] + n]
        parts[i] = None

    with _cf.ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(pass2, range(len(starts))))
    col_idx = np.empty(E, dtype=np.int32)
    mask = (1 << sbits) - 1

    def pass3(k):
        lo, hi = bstart[k], bstart[k + 1]
        if hi > lo:
            seg = np.sort(out[lo:hi])
            col_idx[lo:hi] = seg & mask

    with _cf.ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(pass3, range(nbuckets)))
    del out
    rc = np.zeros(num_dst, dtype=np.int64)
    for r in rowcnt:
        rc += r
    row_ptr = np.zeros(num_dst + 1, dtype=np.int64)
    np.cumsum(rc, out=row_ptr[1:])
    return row_ptr.astype(np.int32), col_idx
