"""Python binding of the C ABI in include/mtx.h (argument marshalling only).

Every function named mtx_* calls the function of the same name in libmtx.so; all arithmetic of
the training step runs in the library's HIP kernels.  PyTorch is used only to allocate device
memory and to name the stream.  If libmtx.so is missing the import of the library raises; there
is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmtx.so")

MTX_OK, MTX_EINVAL, MTX_ENOMEM, MTX_EHIP, MTX_EUNSUPPORTED, MTX_ENONFINITE = 0, -1, -2, -3, -4, -5
MTX_F32, MTX_BF16 = 0, 1
MTX_FC, MTX_CONV, MTX_MAXPOOL, MTX_BN, MTX_ADD, MTX_ADDP = 0, 1, 2, 3, 4, 5
MTX_OPT_MOMENTUM, MTX_OPT_ADAM, MTX_OPT_ADAGRAD = 0, 1, 2

EXPORTS = ("mtx_model_sizes", "mtx_init_model", "mtx_init_model_static", "mtx_train_step", "mtx_average_grads",
           "mtx_sgd_update", "mtx_adam_update", "mtx_adagrad_update", "mtx_get_params",
           "mtx_set_params", "mtx_get_layer_output", "mtx_set_optimizer",
           "mtx_get_pool_argmax", "mtx_set_graph_replay", "mtx_set_overlap",
           "mtx_set_layerwise_update", "mtx_set_fused_update", "mtx_set_nonfinite_check",
           "mtx_set_timing",
           "mtx_get_timing", "mtx_get_launches", "mtx_free_model", "mtx_last_error")


class MtxError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"mtx error {code}: {msg}")
        self.code = code


class mtx_layer(C.Structure):
    _fields_ = [(n, C.c_int) for n in ("kind", "out", "k", "stride", "pad", "groups", "relu")]


class mtx_model_desc(C.Structure):
    _fields_ = [("in_c", C.c_int), ("in_h", C.c_int), ("in_w", C.c_int),
                ("n_layers", C.c_int), ("layers", C.POINTER(mtx_layer)), ("compute", C.c_int)]


class mtx_sizes(C.Structure):
    _fields_ = [("n_params", C.c_size_t), ("grad_stride", C.c_size_t),
                ("workspace_bytes", C.c_size_t)]


class mtx_kernel_time(C.Structure):
    _fields_ = [("name", C.c_char * 32), ("layer", C.c_int), ("launches", C.c_int),
                ("total_ms", C.c_double)]


class mtx_launch_info(C.Structure):
    _fields_ = [("site", C.c_char * 32), ("layer", C.c_int), ("tile_rows", C.c_int),
                ("tile_cols", C.c_int), ("k_tile", C.c_int), ("splits", C.c_int),
                ("flags", C.c_int)]


MTX_GEMM_INTERLEAVED, MTX_GEMM_DIRECT_LDS, MTX_GEMM_FUSED_UPDATE = 1, 2, 4


class mtx_buffers(C.Structure):
    _fields_ = [("w", C.c_void_p), ("v", C.c_void_p), ("grads", C.c_void_p),
                ("grad_avg", C.c_void_p), ("workspace", C.c_void_p),
                ("workspace_bytes", C.c_size_t)]


_lib = None


def lib() -> C.CDLL:
    """Load libmtx.so (built by paper_1704_04560_amd/build.py).  Raises if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run paper_1704_04560_amd/build.py")
        L = C.CDLL(LIB_PATH)
        vp, sz, i32, f32 = C.c_void_p, C.c_size_t, C.c_int, C.c_float
        sig = {
            "mtx_model_sizes": (i32, [C.POINTER(mtx_model_desc), i32, i32, C.POINTER(mtx_sizes)]),
            "mtx_init_model": (i32, [C.POINTER(mtx_model_desc), i32, i32, C.c_uint64,
                                     C.POINTER(mtx_buffers), vp, C.POINTER(vp)]),
            "mtx_init_model_static": (i32, [C.POINTER(mtx_model_desc), i32, i32, C.c_uint64,
                                            C.POINTER(mtx_buffers), vp, C.POINTER(vp)]),
            "mtx_train_step": (i32, [vp, vp, vp, f32, f32, vp, vp]),
            "mtx_average_grads": (i32, [vp, i32, sz, sz, vp, vp]),
            "mtx_sgd_update": (i32, [vp, vp, vp, i32, sz, sz, f32, f32, vp, vp]),
            "mtx_adam_update": (i32, [vp, vp, vp, vp, i32, sz, sz, f32, f32, f32, f32,
                                      C.c_longlong, vp, vp]),
            "mtx_adagrad_update": (i32, [vp, vp, vp, i32, sz, sz, f32, f32, vp, vp]),
            "mtx_get_params": (i32, [vp, vp, vp]),
            "mtx_set_params": (i32, [vp, vp, vp]),
            "mtx_get_layer_output": (i32, [vp, i32, vp, sz]),
            "mtx_get_pool_argmax": (i32, [vp, i32, vp, sz]),
            "mtx_set_graph_replay": (i32, [vp, i32]),
            "mtx_set_optimizer": (i32, [vp, i32, f32, f32, f32, vp]),
            "mtx_set_layerwise_update": (i32, [vp, i32]),
            "mtx_set_fused_update": (i32, [vp, i32]),
            "mtx_set_nonfinite_check": (i32, [vp, i32]),
            "mtx_set_overlap": (i32, [vp, i32]),
            "mtx_set_timing": (i32, [vp, i32]),
            "mtx_get_timing": (i32, [vp, C.POINTER(mtx_kernel_time), i32, C.POINTER(i32), i32]),
            "mtx_get_launches": (i32, [vp, C.POINTER(mtx_launch_info), i32, C.POINTER(i32)]),
            "mtx_free_model": (None, [vp]),
            "mtx_last_error": (C.c_char_p, []),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(rc: int):
    if rc != MTX_OK:
        msg = lib().mtx_last_error()
        raise MtxError(rc, msg.decode() if msg else "")


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream or None
    if isinstance(stream, int):
        return stream or None
    return stream.cuda_stream or None


def make_desc(in_shape: Sequence[int], layers: Sequence[Sequence[int]], compute: int):
    arr = (mtx_layer * len(layers))()
    for i, t in enumerate(layers):
        for name, val in zip(("kind", "out", "k", "stride", "pad", "groups", "relu"), t):
            setattr(arr[i], name, int(val))
    d = mtx_model_desc(int(in_shape[0]), int(in_shape[1]), int(in_shape[2]), len(layers),
                       C.cast(arr, C.POINTER(mtx_layer)), int(compute))
    d._keep = arr
    return d


# ---- the C ABI, one Python function per entry point -------------------------------------------

def mtx_model_sizes(desc, R: int, shard_batch: int) -> Tuple[int, int, int]:
    out = mtx_sizes()
    _check(lib().mtx_model_sizes(C.byref(desc), R, shard_batch, C.byref(out)))
    return out.n_params, out.grad_stride, out.workspace_bytes


def mtx_init_model(desc, R, shard_batch, seed, w, v, grads, grad_avg, workspace, stream=None):
    bufs = mtx_buffers(_ptr(w), _ptr(v), _ptr(grads), _ptr(grad_avg), _ptr(workspace),
                       workspace.numel() * workspace.element_size())
    handle = C.c_void_p()
    _check(lib().mtx_init_model(C.byref(desc), R, shard_batch, C.c_uint64(seed), C.byref(bufs),
                                _stream(stream), C.byref(handle)))
    return handle


def mtx_init_model_static(desc, R, shard_batch, seed, w, v, grads, grad_avg, stream=None):
    bufs = mtx_buffers(_ptr(w), _ptr(v), _ptr(grads), _ptr(grad_avg), None, 0)
    handle = C.c_void_p()
    _check(lib().mtx_init_model_static(C.byref(desc), R, shard_batch, C.c_uint64(seed),
                                       C.byref(bufs), _stream(stream), C.byref(handle)))
    return handle


def mtx_train_step(handle, x, labels, lr, momentum, loss_out=None, stream=None):
    _check(lib().mtx_train_step(handle, _ptr(x), _ptr(labels), lr, momentum, _ptr(loss_out),
                                _stream(stream)))


def mtx_average_grads(grads, R, n, ld, avg, stream=None):
    _check(lib().mtx_average_grads(_ptr(grads), R, n, ld, _ptr(avg), _stream(stream)))


def mtx_sgd_update(w, v, grads, R, n, ld, lr, momentum, avg_out=None, stream=None):
    _check(lib().mtx_sgd_update(_ptr(w), _ptr(v), _ptr(grads), R, n, ld, lr, momentum,
                                _ptr(avg_out), _stream(stream)))


def mtx_adam_update(w, m, v, grads, R, n, ld, lr, beta1, beta2, eps, step, avg_out=None,
                    stream=None):
    _check(lib().mtx_adam_update(_ptr(w), _ptr(m), _ptr(v), _ptr(grads), R, n, ld, lr, beta1,
                                 beta2, eps, step, _ptr(avg_out), _stream(stream)))


def mtx_adagrad_update(w, acc, grads, R, n, ld, lr, eps, avg_out=None, stream=None):
    _check(lib().mtx_adagrad_update(_ptr(w), _ptr(acc), _ptr(grads), R, n, ld, lr, eps,
                                    _ptr(avg_out), _stream(stream)))


def mtx_set_optimizer(handle, kind, beta1=0.9, beta2=0.999, eps=1e-8, s2=None):
    _check(lib().mtx_set_optimizer(handle, kind, beta1, beta2, eps, _ptr(s2)))


def mtx_get_params(handle, w_host: np.ndarray, v_host: Optional[np.ndarray] = None):
    _check(lib().mtx_get_params(handle, _ptr(w_host), _ptr(v_host)))


def mtx_set_params(handle, w_host: np.ndarray, v_host: Optional[np.ndarray] = None):
    w_host = np.ascontiguousarray(w_host, dtype=np.float32)
    v_host = None if v_host is None else np.ascontiguousarray(v_host, dtype=np.float32)
    _check(lib().mtx_set_params(handle, _ptr(w_host), _ptr(v_host)))


def mtx_get_layer_output(handle, layer: int, dst: np.ndarray):
    _check(lib().mtx_get_layer_output(handle, layer, _ptr(dst), dst.size))


def mtx_get_pool_argmax(handle, layer: int, dst: np.ndarray):
    _check(lib().mtx_get_pool_argmax(handle, layer, _ptr(dst), dst.size))


def mtx_set_graph_replay(handle, enable: bool):
    _check(lib().mtx_set_graph_replay(handle, 1 if enable else 0))


def mtx_set_overlap(handle, enable: bool):
    _check(lib().mtx_set_overlap(handle, 1 if enable else 0))


def mtx_set_layerwise_update(handle, enable: bool):
    _check(lib().mtx_set_layerwise_update(handle, 1 if enable else 0))


def mtx_set_fused_update(handle, enable: bool):
    _check(lib().mtx_set_fused_update(handle, 1 if enable else 0))


def mtx_set_nonfinite_check(handle, enable: bool):
    _check(lib().mtx_set_nonfinite_check(handle, 1 if enable else 0))


def mtx_set_timing(handle, enable: bool):
    _check(lib().mtx_set_timing(handle, 1 if enable else 0))


def mtx_get_timing(handle, reset: bool = False):
    """[(name, layer, launches, total_ms)] per launch site of the training step."""
    cap = 256
    buf = (mtx_kernel_time * cap)()
    cnt = C.c_int()
    _check(lib().mtx_get_timing(handle, buf, cap, C.byref(cnt), 1 if reset else 0))
    return [(buf[i].name.decode(), buf[i].layer, buf[i].launches, buf[i].total_ms)
            for i in range(min(cnt.value, cap))]


def mtx_get_launches(handle):
    """[dict(site, layer, tile_rows, tile_cols, k_tile, splits, flags)] per matrix launch of the
    last enqueued training step."""
    cap = 1024
    buf = (mtx_launch_info * cap)()
    cnt = C.c_int()
    _check(lib().mtx_get_launches(handle, buf, cap, C.byref(cnt)))
    return [dict(site=buf[i].site.decode(), layer=buf[i].layer, tile_rows=buf[i].tile_rows,
                 tile_cols=buf[i].tile_cols, k_tile=buf[i].k_tile, splits=buf[i].splits,
                 flags=buf[i].flags) for i in range(min(cnt.value, cap))]


def mtx_free_model(handle):
    lib().mtx_free_model(handle)


# ---- convenience wrapper owning the device buffers --------------------------------------------

class Model:
    """A network bound to caller-owned device buffers (allocated here with torch)."""

    def __init__(self, in_shape, layers, compute, R, shard_batch, seed=0, stream=None,
                 static_workspace=False):
        import torch
        self.in_shape = tuple(in_shape)
        self.layers = [tuple(int(v) for v in t) for t in layers]
        self.compute = compute
        self.R, self.Nb = R, shard_batch
        self.B = R * shard_batch
        self.desc = make_desc(in_shape, layers, compute)
        self.P, self.ld, self.ws_bytes = mtx_model_sizes(self.desc, R, shard_batch)
        dev = torch.device("cuda")
        self.w = torch.empty(self.P, dtype=torch.float32, device=dev)
        self.v = torch.empty(self.P, dtype=torch.float32, device=dev)
        self.grads = torch.empty(R * self.ld, dtype=torch.float32, device=dev)
        self.grad_avg = torch.empty(self.P, dtype=torch.float32, device=dev)
        if static_workspace:  # the library's static array (mtx_init_model_static)
            self.workspace = None
            self.handle = mtx_init_model_static(self.desc, R, shard_batch, seed, self.w, self.v,
                                                self.grads, self.grad_avg, stream)
        else:
            self.workspace = torch.empty(max(self.ws_bytes, 256), dtype=torch.uint8, device=dev)
            self.handle = mtx_init_model(self.desc, R, shard_batch, seed, self.w, self.v,
                                         self.grads, self.grad_avg, self.workspace, stream)
        self._shapes = self._out_shapes()

    def _out_shapes(self):
        c, h, w = self.in_shape
        out = []
        for (kind, o, k, s, p, g, relu) in self.layers:
            if kind == MTX_CONV:
                c, h, w = o, (h + 2 * p - k) // s + 1, (w + 2 * p - k) // s + 1
            elif kind == MTX_FC:
                c, h, w = o, 1, 1
            elif kind in (MTX_BN, MTX_ADD, MTX_ADDP):
                pass
            else:
                h, w = (h - k) // s + 1, (w - k) // s + 1
            out.append((c, h, w))
        return out

    def train_step(self, x, labels, lr, momentum, loss_out=None, stream=None):
        mtx_train_step(self.handle, x, labels, lr, momentum, loss_out, stream)

    def set_optimizer(self, kind, beta1=0.9, beta2=0.999, eps=1e-8):
        """Select the update rule of train_step; Adam gets a zeroed second-moment buffer."""
        import torch
        self.s2 = None
        if kind == MTX_OPT_ADAM:
            self.s2 = torch.zeros(self.P, dtype=torch.float32, device=self.w.device)
        mtx_set_optimizer(self.handle, kind, beta1, beta2, eps, self.s2)

    def get_params(self):
        w = np.empty(self.P, np.float32)
        v = np.empty(self.P, np.float32)
        mtx_get_params(self.handle, w, v)
        return w, v

    def set_params(self, w, v=None):
        mtx_set_params(self.handle, w, v)

    def grads_host(self):
        """Per-shard gradients [R, P] (device-to-host copy through torch)."""
        import torch
        torch.cuda.synchronize()
        return self.grads.view(self.R, self.ld)[:, :self.P].cpu().numpy()

    def layer_output(self, layer: int) -> np.ndarray:
        dst = np.empty(int(np.prod(self._shapes[layer])) * self.B, np.float32)
        mtx_get_layer_output(self.handle, layer, dst)
        return dst

    def pool_argmax(self, layer: int) -> np.ndarray:
        dst = np.empty(int(np.prod(self._shapes[layer])) * self.B, np.uint8)
        mtx_get_pool_argmax(self.handle, layer, dst)
        return dst

    def close(self):
        if self.handle:
            mtx_free_model(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
