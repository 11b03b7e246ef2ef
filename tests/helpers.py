"""Shared test helpers: error metric and tiny hand-made graphs."""
import numpy as np

FP32_TOL = 1e-4
BF16_TOL = 2e-2


def rel_err(y, r):
    """max_i |y_i - r_i| / max(|r_i|, rms(r)): the relative error with its
    denominator floored by the rms of the reference tensor, so that values
    near zero (cancellation, ReLU zeros) do not produce spurious failures."""
    y = np.asarray(y, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    assert y.shape == r.shape, (y.shape, r.shape)
    if r.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(r * r)))
    den = np.maximum(np.abs(r), rms if rms > 0 else 1.0)
    return float(np.max(np.abs(y - r) / den))


def rel_err_terms(y, r, mag):
    """max_i |y_i - r_i| / max(|r_i|, mag_i), where mag_i is the magnitude of
    the terms summed into r_i (the same computation on absolute values).  A
    floating-point sum of n terms errs by about n * eps * mag_i at most, so
    this bounds every element by its own conditioning rather than by the
    rms of the whole tensor (rel_err's floor)."""
    y = np.asarray(y, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    mag = np.asarray(mag, dtype=np.float64)
    assert y.shape == r.shape == mag.shape, (y.shape, r.shape, mag.shape)
    if r.size == 0:
        return 0.0
    den = np.maximum(np.abs(r), mag)
    den = np.where(den > 0, den, 1.0)
    return float(np.max(np.abs(y - r) / den))


def edges_to_csr(n, src, dst):
    """Destination-major CSR via plain Python (rows by dst, then src, then
    edge order) -- independent of synth.graphs.to_in_csr."""
    order = sorted(range(len(src)), key=lambda e: (dst[e], src[e], e))
    col = [src[e] for e in order]
    rp = [0] * (n + 1)
    for e in order:
        rp[dst[e] + 1] += 1
    for v in range(n):
        rp[v + 1] += rp[v]
    return np.array(rp, dtype=np.int32), np.array(col, dtype=np.int32), order


def dense_adjacency(n, src, dst):
    """A[v, u] = number of copies of edge u -> v."""
    A = np.zeros((n, n))
    for u, v in zip(src, dst):
        A[v, u] += 1
    return A


def tiny_graphs():
    """Small edge lists covering multi-edges, self-loops, empty rows, a star
    hub and a chain.  Returns list of (name, n, src, dst)."""
    out = []
    # multigraph with self-loops and an empty row (vertex 5 has no in-edges)
    src = [1, 1, 2, 3, 0, 0, 4, 4, 4, 2, 3, 3, 1]
    dst = [0, 0, 0, 0, 1, 2, 2, 3, 4, 4, 3, 1, 4]
    out.append(("multi", 6, src, dst))
    # star: every leaf points to the hub 0, hub points to every leaf
    n = 40
    s = list(range(1, n)) + [0] * (n - 1)
    d = [0] * (n - 1) + list(range(1, n))
    out.append(("star", n, s, d))
    # directed chain 0 -> 1 -> ... -> n-1 with self-loops
    n = 17
    s = list(range(n - 1)) + list(range(n))
    d = list(range(1, n)) + list(range(n))
    out.append(("chain", n, s, d))
    # random multigraph with repeated pairs
    rng = np.random.default_rng(7)
    n = 50
    s = rng.integers(0, n, 300).tolist()
    d = (rng.integers(0, n, 300) // 2).tolist()  # upper half of ids: empty rows
    out.append(("random", n, s, d))
    return out


def plan_edge_limit(num_dst, seg_len, row_cost):
    """Largest num_edges a plan accepts (the header's rule): num_edges < 2^31
    and the total segment cost num_edges + row_cost * (num_dst +
    ceil(num_edges / seg_len)) below 2^31 - 1."""
    def ok(e):
        return e < 2**31 and e + row_cost * (num_dst + -(-e // seg_len)) <= 2**31 - 2

    lo, hi = 0, 2**31 - 1
    while lo < hi:
        mid = (lo + hi + 1) // 2
        if ok(mid):
            lo = mid
        else:
            hi = mid - 1
    return lo

