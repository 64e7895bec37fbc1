"""Python binding of the heterogeneous-parallel Linear C ABI (include/hetegen.h).

Argument marshalling only: every step of the path runs in libhetegen.so (gfx950
kernels and the host runtime).  Pointers are plain integers (device addresses,
for instance ``tensor.data_ptr()``, or pinned host addresses); streams are
``hipStream_t`` values as integers (``torch.cuda.current_stream().cuda_stream``).
Importing fails loudly when the library has not been built.
"""
import ctypes
import os

import numpy as np

# torch first: it carries its own HIP runtime, whose SONAME (libamdhip64.so.7) then
# satisfies the library's dependency, so the process holds ONE HIP runtime and
# torch's device pointers and stream handles are valid in the library's calls.
# Loading the library first would bring in /opt/rocm's runtime beside torch's.
import torch  # noqa: F401

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libhetegen.so")

F16, BF16, F32 = 0, 1, 2
OK, ERR_INVALID_ARG, ERR_NOT_PINNED, ERR_UNSUPPORTED, ERR_OOM, ERR_HIP, ERR_INTERNAL = range(7)
PLAN_APPROX = 1
EXEC_AUTO, EXEC_PERSISTENT, EXEC_GRAPH, EXEC_EAGER = 0, 1, 2, 3
BENCH_CROSSING, BENCH_WALL = 0, 1
STATUS_NAMES = {0: "OK", 1: "INVALID_ARG", 2: "NOT_PINNED", 3: "UNSUPPORTED", 4: "OOM", 5: "HIP", 6: "INTERNAL"}

if not os.path.exists(LIB_PATH):
    raise ImportError("libhetegen.so is not built: run `python paper_2403_01164_amd/build.py` "
                      "(or __graft_entry__.build())")


class Config(ctypes.Structure):
    _fields_ = [("device", ctypes.c_int), ("cpu_threads", ctypes.c_int), ("chunk_bytes", ctypes.c_size_t),
                ("ring_depth", ctypes.c_int), ("pin_threads", ctypes.c_int), ("pin_ring", ctypes.c_int),
                ("numa_node", ctypes.c_int)]


class Shape(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int), ("K", ctypes.c_int), ("dtype", ctypes.c_int), ("resident", ctypes.c_int)]


class Bw(ctypes.Structure):
    _fields_ = [("cpu_Bps", ctypes.c_double), ("h2d_Bps", ctypes.c_double), ("hbm_gemv_Bps", ctypes.c_double),
                ("pin_Bps", ctypes.c_double)]


class Profile(ctypes.Structure):
    _fields_ = [("wall_ms", ctypes.c_double), ("cpu_ms", ctypes.c_double), ("h2d_ms", ctypes.c_double),
                ("gpu_ms", ctypes.c_double), ("h2d_bytes", ctypes.c_double), ("gpu_bytes", ctypes.c_double),
                ("cpu_bytes", ctypes.c_double), ("gemv_launches", ctypes.c_int64), ("pin_ms", ctypes.c_double),
                ("pin_bytes", ctypes.c_double), ("xwait_ms", ctypes.c_double), ("tailwait_ms", ctypes.c_double),
                ("cpu_shares", ctypes.c_int64), ("hetlin_ms", ctypes.c_double), ("res_gpu_ms", ctypes.c_double),
                ("res_gpu_bytes", ctypes.c_double)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


_lib = ctypes.CDLL(LIB_PATH)
_vp, _i, _d, _sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_double, ctypes.c_size_t
_SIGS = {
    "hetegen_create": ([ctypes.POINTER(Config), ctypes.POINTER(_vp)], _i),
    "hetegen_destroy": ([_vp], _i),
    "hetegen_last_error": ([_vp], ctypes.c_char_p),
    "hetegen_cpu_share_isa": ([], ctypes.c_char_p),
    "hetegen_host_alloc": ([_vp, _sz, ctypes.POINTER(_vp)], _i),
    "hetegen_host_free": ([_vp, _vp], _i),
    "hetegen_linear": ([_vp, _vp, _i, _i, _vp, _vp, _i, _i, _vp, _vp, _d, _vp, _i, _vp], _i),
    "hetegen_tiled_bytes": ([_i, _i], _sz),
    "hetegen_tile_weights": ([_vp, _vp, _i, _i, _vp, _vp], _i),
    "hetegen_linear_tiled": ([_vp, _vp, _i, _i, _vp, _i, _i, _vp, _vp, _i, _vp], _i),
    "hetegen_linear_tiled_noalloc": ([_vp, _vp, _i, _i, _vp, _i, _i, _vp, _vp, _i, _vp], _i),
    "hetegen_layer_plan": ([ctypes.POINTER(Shape), _i, ctypes.POINTER(Bw), _i, _i, ctypes.POINTER(_d)], _i),
    "hetegen_probe": ([_vp, _vp, _i, _i, _i, _i, _i, _i, ctypes.POINTER(Bw)], _i),
    "hetegen_alpha_fit": ([ctypes.POINTER(_d), ctypes.POINTER(_d), ctypes.POINTER(_d), _i, _i, _d, _d,
                           ctypes.POINTER(_d), ctypes.POINTER(_i)], _i),
    "hetegen_alpha_benchmark": ([_vp, _vp, _i, _i, _vp, _i, _i, _vp, _vp, _vp, _d, _d, _d, _i, _i, _vp,
                                 ctypes.POINTER(_d), ctypes.POINTER(_i)], _i),
    "hetegen_model_create": ([_vp, _i, _i, _i, _i, ctypes.POINTER(_vp), ctypes.POINTER(_vp), ctypes.POINTER(_d),
                              ctypes.POINTER(_i), _i, ctypes.POINTER(_vp)], _i),
    "hetegen_model_set_alpha": ([_vp, ctypes.POINTER(_d)], _i),
    "hetegen_model_set_exec": ([_vp, _i, ctypes.c_uint32], _i),
    "hetegen_model_alpha_benchmark": ([_vp, _vp, _vp, _vp, _i, _d, _d, _i, _i, _i, _vp, ctypes.POINTER(_d),
                                       ctypes.POINTER(_i)], _i),
    "hetegen_alpha_minimize": ([ctypes.POINTER(_d), ctypes.POINTER(_d), _i, _i, _d, _d, ctypes.POINTER(_d)], _i),
    "hetegen_model_get_alpha": ([_vp, ctypes.POINTER(_d)], _i),
    "hetegen_model_linear_ms": ([_vp, ctypes.POINTER(_d)], _i),
    "hetegen_model_read_ms": ([_vp, _vp, _i, _vp, ctypes.POINTER(_d)], _i),
    "hetegen_cpu_linear": ([_vp, _i, _i, _vp, _i, _vp, _i, _i, _vp, _i, _i], _i),
    "hetegen_probe_hbm": ([_vp, _sz, _i, ctypes.POINTER(_d)], _i),
    "hetegen_probe_link": ([_vp, _sz, _i, ctypes.POINTER(_d)], _i),
    "hetegen_probe_launch": ([_vp, _i, _vp, ctypes.POINTER(_d)], _i),
    "hetegen_model_kv_create": ([_vp, _vp, _i, _i], _i),
    "hetegen_model_kv_write": ([_vp, _vp, _i, _i, _i, _i, _vp, _vp, _vp], _i),
    "hetegen_model_kv_read": ([_vp, _vp, _i, _i, _i, _i, _vp, _vp, _vp], _i),
    "hetegen_decode_step_kv": ([_vp, _vp, _vp, _vp, _i, _i, _vp], _i),
    "hetegen_module_schedule": ([ctypes.POINTER(_d), ctypes.POINTER(_d), ctypes.POINTER(_i), _i, _d,
                                 ctypes.POINTER(_i), ctypes.POINTER(_d)], _i),
    "hetegen_model_last_exec": ([_vp], _i),
    "hetegen_model_layouts": ([_vp], _i),
    "hetegen_decode_step": ([_vp, _vp, _vp, _vp, _i, _vp], _i),
    "hetegen_model_trace_bytes": ([_vp, _i], _sz),
    "hetegen_model_set_trace": ([_vp, _vp, _sz], _i),
    "hetegen_model_destroy": ([_vp, _vp], _i),
    "hetegen_set_profiling": ([_vp, _i], _i),
    "hetegen_get_profile": ([_vp, ctypes.POINTER(Profile), _i], _i),
}
for _name, (_args, _res) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = _res

EXPORTED = tuple(_SIGS)


class HetegenError(RuntimeError):
    def __init__(self, status, message):
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, status), message))
        self.status = status


def _check(rc, ctx=None):
    if rc != OK:
        msg = _lib.hetegen_last_error(ctx)
        raise HetegenError(rc, msg.decode() if msg else "")


def hetegen_create(device=0, cpu_threads=0, chunk_bytes=0, ring_depth=0, pin_threads=0, pin_ring=0,
                   numa_node=None):
    """numa_node: None leaves pinned host memory to the calling thread's policy; n binds it to node n."""
    cfg = Config(device, cpu_threads, chunk_bytes, ring_depth, pin_threads, pin_ring,
                 0 if numa_node is None else int(numa_node) + 1)
    out = _vp()
    _check(_lib.hetegen_create(ctypes.byref(cfg), ctypes.byref(out)))
    return out.value


def hetegen_destroy(ctx):
    _check(_lib.hetegen_destroy(ctx))


def hetegen_last_error(ctx):
    m = _lib.hetegen_last_error(ctx)
    return m.decode() if m else ""


def hetegen_cpu_share_isa():
    """Instruction set of the CPU share on this host ("avx512+bf16", "avx512", "avx2", "scalar")."""
    return _lib.hetegen_cpu_share_isa().decode()


def hetegen_host_alloc(ctx, nbytes):
    p = _vp()
    _check(_lib.hetegen_host_alloc(ctx, nbytes, ctypes.byref(p)), ctx)
    return p.value


def hetegen_host_free(ctx, ptr):
    _check(_lib.hetegen_host_free(ctx, ptr), ctx)


def hetegen_linear(ctx, x_dev, B, K, W_host, W_dev_resident, N, w_dtype, bias_host, bias_dev, alpha, y_dev,
                   y_dtype, stream=0):
    _check(_lib.hetegen_linear(ctx, x_dev, B, K, W_host, W_dev_resident or None, N, w_dtype, bias_host or None,
                               bias_dev or None, float(alpha), y_dev, y_dtype, stream or None), ctx)


def hetegen_linear_status(ctx, *args):
    """Same arguments as hetegen_linear; returns the raw status instead of raising."""
    (x_dev, B, K, W_host, W_dev_resident, N, w_dtype, bias_host, bias_dev, alpha, y_dev, y_dtype, stream) = args
    return _lib.hetegen_linear(ctx, x_dev, B, K, W_host, W_dev_resident or None, N, w_dtype, bias_host or None,
                               bias_dev or None, float(alpha), y_dev, y_dtype, stream or None)


def hetegen_tiled_bytes(rows, K):
    return _lib.hetegen_tiled_bytes(rows, K)


def hetegen_tile_weights(ctx, W_dev, rows, K, W_tiled_dev, stream=0):
    _check(_lib.hetegen_tile_weights(ctx, W_dev, rows, K, W_tiled_dev, stream or None), ctx)


def hetegen_linear_tiled(ctx, x_dev, B, K, W_tiled_dev, N, w_dtype, bias_dev, y_dev, y_dtype, stream=0):
    _check(_lib.hetegen_linear_tiled(ctx, x_dev, B, K, W_tiled_dev, N, w_dtype, bias_dev or None, y_dev, y_dtype,
                                     stream or None), ctx)


def hetegen_linear_tiled_noalloc(ctx, x_dev, B, K, W_tiled_dev, N, w_dtype, bias_dev, y_dev, y_dtype, stream=0):
    _check(_lib.hetegen_linear_tiled_noalloc(ctx, x_dev, B, K, W_tiled_dev, N, w_dtype, bias_dev or None, y_dev,
                                             y_dtype, stream or None), ctx)


def hetegen_linear_tiled_noalloc_status(ctx, *args):
    """Same arguments as hetegen_linear_tiled_noalloc; returns the raw status instead of raising."""
    (x_dev, B, K, W_tiled_dev, N, w_dtype, bias_dev, y_dev, y_dtype, stream) = args
    return _lib.hetegen_linear_tiled_noalloc(ctx, x_dev, B, K, W_tiled_dev, N, w_dtype, bias_dev or None, y_dev,
                                             y_dtype, stream or None)


def hetegen_linear_tiled_status(ctx, *args):
    """Same arguments as hetegen_linear_tiled; returns the raw status instead of raising."""
    (x_dev, B, K, W_tiled_dev, N, w_dtype, bias_dev, y_dev, y_dtype, stream) = args
    return _lib.hetegen_linear_tiled(ctx, x_dev, B, K, W_tiled_dev, N, w_dtype, bias_dev or None, y_dev, y_dtype,
                                     stream or None)


def hetegen_layer_plan(shapes, bws, flags=0):
    """shapes: list of (N, K, dtype, resident); bws: list of (cpu, h2d, hbm, pin) bytes/s, one or len(shapes)."""
    n = len(shapes)
    sh = (Shape * max(n, 1))(*[Shape(*s) for s in shapes])
    bw = (Bw * len(bws))(*[Bw(*b) for b in bws])
    out = (_d * max(n, 1))()
    rc = _lib.hetegen_layer_plan(sh, n, bw, len(bws), flags, out)
    if rc != OK:
        raise HetegenError(rc, "hetegen_layer_plan")
    return [out[i] for i in range(n)]


PROBE_CONCURRENT = 1


def hetegen_probe(ctx, W_host, N, K, dtype, B=1, reps=3, flags=0):
    bw = Bw()
    _check(_lib.hetegen_probe(ctx, W_host, N, K, dtype, B, reps, flags, ctypes.byref(bw)), ctx)
    return {"cpu_Bps": bw.cpu_Bps, "h2d_Bps": bw.h2d_Bps, "hbm_gemv_Bps": bw.hbm_gemv_Bps, "pin_Bps": bw.pin_Bps}


def hetegen_alpha_fit(alphas, t_cpu, t_com, degree, lo, hi):
    """Refined CPU fraction from samples; returns (alpha, crossed)."""
    n = len(alphas)
    arr = lambda v: (_d * n)(*[float(x) for x in v])
    out, crossed = _d(), _i()
    rc = _lib.hetegen_alpha_fit(arr(alphas), arr(t_cpu), arr(t_com), n, degree, float(lo), float(hi),
                                ctypes.byref(out), ctypes.byref(crossed))
    if rc != OK:
        raise HetegenError(rc, "hetegen_alpha_fit")
    return out.value, bool(crossed.value)


def hetegen_alpha_benchmark(ctx, x_dev, B, K, W_host, N, dtype, bias_host, bias_dev, y_dev, alpha0, gamma=0.05,
                            lam=0.01, degree=2, reps=2, stream=0):
    """Measured refinement of one linear's CPU fraction; returns (alpha, crossed)."""
    out, crossed = _d(), _i()
    _check(_lib.hetegen_alpha_benchmark(ctx, x_dev, B, K, W_host, N, dtype, bias_host or None, bias_dev or None, y_dev,
                                        float(alpha0), float(gamma), float(lam), degree, reps, stream or None,
                                        ctypes.byref(out), ctypes.byref(crossed)), ctx)
    return out.value, bool(crossed.value)


def hetegen_model_create(ctx, L, H, F, dtype, W_host, bias_host, alpha, resident, max_batch=1):
    n = 4 * L
    W = (_vp * n)(*W_host)
    b = (_vp * n)(*bias_host) if bias_host is not None else None
    a = (_d * n)(*[float(v) for v in alpha])
    r = (_i * n)(*[int(v) for v in resident])
    out = _vp()
    _check(_lib.hetegen_model_create(ctx, L, H, F, dtype, W, b, a, r, max_batch, ctypes.byref(out)), ctx)
    return out.value


def hetegen_model_set_alpha(model, alpha):
    a = (_d * len(alpha))(*[float(v) for v in alpha])
    rc = _lib.hetegen_model_set_alpha(model, a)
    if rc != OK:
        raise HetegenError(rc, "hetegen_model_set_alpha")


def hetegen_model_alpha_benchmark(ctx, model, x_dev, out_dev, B, gamma=0.05, lam=0.01, degree=2, reps=1,
                                  objective=BENCH_WALL, stream=0):
    """Step-level refinement; returns (delta, crossed).  The model keeps the refined fractions."""
    d, crossed = _d(), _i()
    _check(_lib.hetegen_model_alpha_benchmark(ctx, model, x_dev, out_dev, B, float(gamma), float(lam), degree, reps,
                                              objective, stream or None, ctypes.byref(d), ctypes.byref(crossed)), ctx)
    return d.value, bool(crossed.value)


def hetegen_module_schedule(t_cpu, mem, layer, budget):
    """Resident flag per module (Sec. 4.5, Eq. 13) and the bytes they take."""
    n = len(t_cpu)
    res = (_i * max(n, 1))()
    used = _d()
    rc = _lib.hetegen_module_schedule((_d * max(n, 1))(*[float(v) for v in t_cpu]),
                                      (_d * max(n, 1))(*[float(v) for v in mem]),
                                      (_i * max(n, 1))(*[int(v) for v in layer]), n, float(budget), res,
                                      ctypes.byref(used))
    if rc != OK:
        raise HetegenError(rc, "hetegen_module_schedule")
    return [res[i] for i in range(n)], used.value


def hetegen_alpha_minimize(alphas, t, degree, lo, hi):
    n = len(alphas)
    arr = lambda v: (_d * n)(*[float(x) for x in v])
    out = _d()
    rc = _lib.hetegen_alpha_minimize(arr(alphas), arr(t), n, degree, float(lo), float(hi), ctypes.byref(out))
    if rc != OK:
        raise HetegenError(rc, "hetegen_alpha_minimize")
    return out.value


def hetegen_model_get_alpha(model, n):
    out = (_d * n)()
    rc = _lib.hetegen_model_get_alpha(model, out)
    if rc != OK:
        raise HetegenError(rc, "hetegen_model_get_alpha")
    return [out[i] for i in range(n)]


def hetegen_model_linear_ms(model, n):
    out = (_d * n)()
    rc = _lib.hetegen_model_linear_ms(model, out)
    if rc != OK:
        raise HetegenError(rc, "hetegen_model_linear_ms")
    return [out[i] for i in range(n)]


def hetegen_model_read_ms(ctx, model, reps=5, stream=0):
    """Median ms of one pass of plain streaming reads over the model's resident GPU
    rows, one launch per resident linear in step order (a lower bound of the step)."""
    out = _d()
    _check(_lib.hetegen_model_read_ms(ctx, model, reps, stream, ctypes.byref(out)), ctx)
    return out.value


def hetegen_model_set_exec(model, mode, barrier_spin_limit=0):
    rc = _lib.hetegen_model_set_exec(model, mode, barrier_spin_limit)
    if rc != OK:
        raise HetegenError(rc, "hetegen_model_set_exec")


def hetegen_model_last_exec(model):
    return _lib.hetegen_model_last_exec(model)


LAYOUT_ROWMAJOR, LAYOUT_TILED, LAYOUT_KMAJOR, LAYOUT_SEGMAJOR = 1, 2, 4, 8


def hetegen_model_layouts(model):
    """Bitmask of the layouts the model keeps its resident rows in (LAYOUT_ROWMAJOR, LAYOUT_TILED)."""
    return _lib.hetegen_model_layouts(model)


def hetegen_decode_step(ctx, model, x_dev, out_dev, B, stream=0):
    _check(_lib.hetegen_decode_step(ctx, model, x_dev, out_dev, B, stream or None), ctx)


def hetegen_model_trace_bytes(model, B):
    return _lib.hetegen_model_trace_bytes(model, B)


def hetegen_model_set_trace(model, trace_dev, nbytes):
    rc = _lib.hetegen_model_set_trace(model, trace_dev or None, nbytes)
    if rc != OK:
        raise HetegenError(rc, "hetegen_model_set_trace")


def hetegen_model_destroy(ctx, model):
    _check(_lib.hetegen_model_destroy(ctx, model), ctx)


def hetegen_set_profiling(ctx, on):
    _check(_lib.hetegen_set_profiling(ctx, int(bool(on))), ctx)


def hetegen_get_profile(ctx, reset=False):
    p = Profile()
    _check(_lib.hetegen_get_profile(ctx, ctypes.byref(p), int(bool(reset))), ctx)
    return p.as_dict()


def host_view(ptr, shape, np_dtype):
    """numpy view of pinned host memory at address ptr (no copy)."""
    count = int(np.prod(shape))
    buf = (ctypes.c_char * (count * np.dtype(np_dtype).itemsize)).from_address(ptr)
    return np.frombuffer(buf, dtype=np_dtype, count=count).reshape(shape)


def hetegen_model_kv_create(ctx, model, max_seq, head_dim):
    _check(_lib.hetegen_model_kv_create(ctx, model, max_seq, head_dim), ctx)


def hetegen_model_kv_write(ctx, model, layer, B, pos0, n, k_dev, v_dev, stream=0):
    _check(_lib.hetegen_model_kv_write(ctx, model, layer, B, pos0, n, k_dev, v_dev, stream or None), ctx)


def hetegen_model_kv_read(ctx, model, layer, B, pos0, n, k_dev, v_dev, stream=0):
    _check(_lib.hetegen_model_kv_read(ctx, model, layer, B, pos0, n, k_dev, v_dev, stream or None), ctx)


def hetegen_decode_step_kv(ctx, model, x_dev, out_dev, B, pos, stream=0):
    _check(_lib.hetegen_decode_step_kv(ctx, model, x_dev, out_dev, B, pos, stream or None), ctx)


def hetegen_cpu_linear(x_f32, W_ptr, bias_ptr, dtype, r0, r1, threads=0):
    """CPU share of rows [r0, r1): x_f32 numpy float32 [B, K]; returns float32 [B, r1 - r0]."""
    import numpy as np
    x = np.ascontiguousarray(x_f32, dtype=np.float32)
    B, K = x.shape
    y = np.zeros((B, max(r1 - r0, 0)), np.float32)
    rc = _lib.hetegen_cpu_linear(x.ctypes.data, B, K, W_ptr, dtype, bias_ptr or None, r0, r1, y.ctypes.data,
                                 max(r1 - r0, 1), threads)
    if rc != OK:
        raise HetegenError(rc, "hetegen_cpu_linear")
    return y


def hetegen_probe_hbm(ctx, nbytes, reps=5):
    """Achievable HBM read bandwidth in bytes/s."""
    out = _d()
    _check(_lib.hetegen_probe_hbm(ctx, nbytes, reps, ctypes.byref(out)), ctx)
    return out.value


def hetegen_probe_link(ctx, nbytes, reps=10):
    """Idle pinned host-to-device copy rate in bytes/s (median of reps copies)."""
    out = _d()
    _check(_lib.hetegen_probe_link(ctx, nbytes, reps, ctypes.byref(out)), ctx)
    return out.value


def hetegen_probe_launch(ctx, reps=1000, stream=0):
    """Empty-kernel launch + stream synchronisation round trip in microseconds (median)."""
    out = _d()
    _check(_lib.hetegen_probe_launch(ctx, reps, stream or None, ctypes.byref(out)), ctx)
    return out.value
