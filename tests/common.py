"""Shared helpers of the GPU tests (marshalling and the tolerance metric; no method arithmetic)."""
import numpy as np

TOL = 2e-3  # max relative error on binary32-accumulated outputs
U_ACT = {0: 2.0 ** -11, 1: 2.0 ** -8}  # unit roundoff of fp16 / bf16 outputs


def rel_err(y, ref, floor=1e-2):
    """max_{b,j} |y - ref| / max(|ref[b,j]|, floor * max_i |ref[b,i]|).

    The floor keeps near-zero outputs from dominating: it is 1% of the largest
    magnitude in the same batch row."""
    y = np.asarray(y, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if ref.ndim == 1:
        ref = ref[None]
        y = y[None]
    scale = np.maximum(np.abs(ref), floor * np.max(np.abs(ref), axis=1, keepdims=True))
    scale = np.where(scale == 0, 1.0, scale)
    return float(np.max(np.abs(y - ref) / scale))


def torch_dev_from_np(a):
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).cuda()
    return torch.from_numpy(a.copy()).cuda()


def np_from_dev(t, np_dtype):
    a = t.cpu().numpy()
    return a.view(np_dtype) if a.dtype != np_dtype else a


class Pinned:
    """Pinned host buffer from the library, with a numpy view."""

    def __init__(self, hg, ctx, shape, np_dtype):
        self.hg, self.ctx = hg, ctx
        self.nbytes = int(np.prod(shape)) * np.dtype(np_dtype).itemsize
        self.ptr = hg.hetegen_host_alloc(ctx, self.nbytes)
        self.a = hg.host_view(self.ptr, shape, np_dtype)

    def free(self):
        if self.ptr:
            self.hg.hetegen_host_free(self.ctx, self.ptr)
            self.ptr = 0


class Pageable:
    """Plain (pageable) host buffer from an anonymous mapping, with a numpy view."""

    def __init__(self, shape, np_dtype):
        import mmap
        n = int(np.prod(shape))
        self.nbytes = n * np.dtype(np_dtype).itemsize
        self.mm = mmap.mmap(-1, max(self.nbytes, 4096))
        self.a = np.frombuffer(self.mm, dtype=np_dtype, count=n).reshape(shape)
        self.ptr = self.a.ctypes.data

    def free(self):
        pass  # the mapping goes with the object
