"""Helpers for the GPU parity tests (device placement, padded buffers)."""
import numpy as np
import torch

from helpers import rel_err  # noqa: F401


def device():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda:0")


def lib():
    import paper_2009_00804_amd.saga as S

    S.lib()  # raises if libsaga.so is missing: no fallback path
    return S


def dev_int(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(device())


def dev_padded(a, dtype=torch.float32, ld=None, fill=float("nan")):
    """Device copy of a 2-D array inside a buffer with ld >= cols whose
    padding holds ``fill`` (NaN by default, so that stray reads show)."""
    a = np.asarray(a)
    rows, cols = a.shape
    es = 2 if dtype == torch.bfloat16 else 4
    step = 16 // es
    ld = ld or (cols + step - 1) // step * step
    buf = torch.full((rows, ld), fill, dtype=torch.float32)
    buf[:, :cols] = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return buf.to(dtype).to(device())[:, :cols]


def dev_bf16_from_bits(bits, cols=None):
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)
    t = t.to(device())
    return t if cols is None else t[:, :cols]


def to_np(t):
    return t.float().cpu().numpy().astype(np.float64)


def graph(row_ptr, col_idx, num_src=None, **opts):
    S = lib()
    return S.Graph(dev_int(row_ptr), dev_int(col_idx), num_src=num_src, **opts)
