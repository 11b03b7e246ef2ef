"""Seeded dense inputs: vertex/edge features, weights, biases, and their
bfloat16 storage variants.

Inputs only: nothing here evaluates a stage of the layer.
"""
from __future__ import annotations

import concurrent.futures as _cf

import numpy as np

from .graphs import _threads, seed_seq


def padded(rows: int, cols: int, ld: int, dtype) -> np.ndarray:
    """A rows x ld buffer whose first ``cols`` columns are the matrix.

    Padding columns are filled with NaN (floats) so that any consumer which
    reads them by mistake produces visibly wrong results."""
    buf = np.empty((rows, ld), dtype=dtype)
    if ld > cols:
        if np.dtype(dtype) == np.uint16:
            buf[:, cols:] = 0x7FC0  # bfloat16 quiet NaN
        else:
            buf[:, cols:] = np.nan
    return buf


def normal_matrix(rows: int, cols: int, key: tuple, ld: int | None = None,
                  chunk_rows: int = 4096) -> np.ndarray:
    """rows x cols float32 N(0, 1), row chunks drawn from child seeds."""
    ld = cols if ld is None else ld
    out = padded(rows, cols, ld, np.float32)
    nchunks = (rows + chunk_rows - 1) // chunk_rows

    def work(i):
        lo = i * chunk_rows
        hi = min(rows, lo + chunk_rows)
        rng = np.random.Generator(np.random.PCG64(seed_seq(*key, i)))
        out[lo:hi, :cols] = rng.standard_normal((hi - lo, cols), dtype=np.float32)

    with _cf.ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(work, range(nchunks)))
    return out


def sparse_binary_matrix(rows: int, cols: int, p: float, rng: np.random.Generator):
    """float32 matrix with entries 1 where U(0,1) < p, else 0."""
    return (rng.random((rows, cols)) < p).astype(np.float32)


def glorot(fan_in: int, fan_out: int, rng: np.random.Generator, shape=None):
    """Glorot-uniform U(-s, s), s = sqrt(6 / (fan_in + fan_out)), float32."""
    s = np.sqrt(6.0 / (fan_in + fan_out))
    shape = (fan_in, fan_out) if shape is None else shape
    return rng.uniform(-s, s, size=shape).astype(np.float32)


def bias(fan_in: int, n: int, rng: np.random.Generator):
    """U(-1/sqrt(fan_in), 1/sqrt(fan_in)), float32."""
    s = 1.0 / np.sqrt(fan_in)
    return rng.uniform(-s, s, size=n).astype(np.float32)


# --------------------------------------------------------------------------
# bfloat16 storage
# --------------------------------------------------------------------------
def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round to nearest, ties to even); returns the
    16-bit patterns as uint16.  Inputs must be finite."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact float32 value of bfloat16 bit patterns."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_padded_from_f32(x: np.ndarray, cols: int, ld: int) -> np.ndarray:
    """bfloat16 copy (uint16 bits) of the first ``cols`` columns of x, in a
    buffer with leading dimension ``ld`` (padding set to NaN)."""
    out = padded(x.shape[0], cols, ld, np.uint16)
    step = 4096

    def work(lo):
        hi = min(x.shape[0], lo + step)
        out[lo:hi, :cols] = bf16_bits(x[lo:hi, :cols])

    with _cf.ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(work, range(0, x.shape[0], step)))
    return out
