"""Helpers shared by the GPU tests: host <-> device moves with the dtypes the
binding expects (uint32 travels as int32, uint64 as int64)."""
import numpy as np
import torch

_VIEW = {np.dtype(np.uint32): np.int32, np.dtype(np.uint64): np.int64}


def dev(a):
    a = np.ascontiguousarray(a)
    v = _VIEW.get(a.dtype)
    if v is not None:
        a = a.view(v)
    return torch.from_numpy(a).to("cuda")


def host(t, dtype=None):
    a = t.cpu().numpy()
    if dtype is not None:
        a = a.view(dtype)
    return a


def pack(prompts):
    """bytes prompts -> (text uint8, offsets uint64) on the host."""
    lens = [len(p) for p in prompts]
    offsets = np.zeros(len(prompts) + 1, dtype=np.uint64)
    offsets[1:] = np.cumsum(lens, dtype=np.uint64)
    text = np.frombuffer(b"".join(prompts), dtype=np.uint8).copy()
    return text, offsets


def rel_close(a, b, rtol):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    both_nan = np.isnan(a) & np.isnan(b)
    scale = np.maximum(np.abs(b), 1e-300)
    ok = (np.abs(a - b) <= rtol * scale) | (a == b) | both_nan
    return bool(ok.all()), (np.abs(a - b) / scale)[~both_nan].max() if a.size else 0.0
