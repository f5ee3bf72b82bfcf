"""Python binding of ``libqlin.so`` (argument marshalling only).

The functions mirror the C ABI in ``include/qlin.h`` one to one; ``QLinear``
wraps a handle for torch callers.  torch supplies device memory and the
current stream; every step of the computation runs in the HIP kernels.  The
module raises if the library has not been built - there is no fallback.
"""

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# QLIN_LIB selects another build of the same library (the sanitizer build of
# the CPU tests); by default the in-tree libqlin.so
LIB_PATH = os.environ.get("QLIN_LIB") or os.path.join(_HERE, "libqlin.so")

QLIN_OK = 0
QLIN_ERR_INVALID = -1
QLIN_ERR_UNSUPPORTED = -2
QLIN_ERR_ALIGN = -3
QLIN_ERR_OOM = -4
QLIN_ERR_HIP = -5

PATH_AUTO, PATH_GEMV, PATH_SKINNY, PATH_TILED, PATH_REGS = 0, 1, 2, 3, 4

# every symbol include/qlin.h declares
EXPORTS = ("qlin_create", "qlin_create_symmetric", "qlin_forward", "qlin_forward_path",
           "qlin_plan", "qlin_destroy", "qlin_last_error", "qlin_unpack_codes",
           "qlin_dequantize", "qlin_shape", "qlin_last_status", "qlin_stream_read", "qlin_quantize",
           "qlin_swa_plan", "qlin_swa_attention", "qlin_forward_group", "qlin_group_plan",
           "qlin_workspace_bytes", "qlin_forward_group_noalloc")

_lib = None


class QlinError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"qlin error {code}: {msg}")
        self.code = code


def lib():
    """Load ``libqlin.so`` (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"HIP library {LIB_PATH} is missing: run __graft_entry__.build() first")
    L = ctypes.CDLL(LIB_PATH)
    P, I64, I32, VP = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p
    L.qlin_create.restype = P
    L.qlin_create.argtypes = [I64, I64, I64, VP, VP, VP]
    L.qlin_create_symmetric.restype = P
    L.qlin_create_symmetric.argtypes = [I64, I64, I64, VP, VP]
    L.qlin_quantize.restype = I32
    L.qlin_quantize.argtypes = [I64, I64, I64, VP, VP, VP, VP, VP]
    L.qlin_forward.restype = I32
    L.qlin_forward.argtypes = [P, I64, VP, VP, VP]
    L.qlin_forward_path.restype = I32
    L.qlin_forward_path.argtypes = [P, I32, I64, I64, VP, VP, VP]
    L.qlin_plan.restype = I32
    L.qlin_plan.argtypes = [P, I32, I64, I64, ctypes.c_char_p, I64]
    L.qlin_destroy.restype = None
    L.qlin_destroy.argtypes = [P]
    L.qlin_last_error.restype = ctypes.c_char_p
    L.qlin_last_error.argtypes = []
    L.qlin_last_status.restype = I32
    L.qlin_last_status.argtypes = []
    L.qlin_unpack_codes.restype = I32
    L.qlin_unpack_codes.argtypes = [P, VP, VP]
    L.qlin_dequantize.restype = I32
    L.qlin_dequantize.argtypes = [P, I32, VP, VP]
    L.qlin_stream_read.restype = I32
    L.qlin_stream_read.argtypes = [VP, I64, I32, VP, VP]
    L.qlin_swa_plan.restype = I32
    L.qlin_swa_plan.argtypes = [I64, I64, I64, I64, I64, I64, I64, ctypes.POINTER(I64), ctypes.POINTER(I64),
                                ctypes.c_char_p, I64]
    L.qlin_swa_attention.restype = I32
    L.qlin_swa_attention.argtypes = [I64, I64, I64, I64, I64, I64, I64, I64, VP, VP, VP, VP, VP, I64, VP]
    L.qlin_forward_group.restype = I32
    L.qlin_forward_group.argtypes = [I64, VP, I32, I64, I64, VP, VP, VP, I64, VP]
    L.qlin_forward_group_noalloc.restype = I32
    L.qlin_forward_group_noalloc.argtypes = [I64, VP, I32, I64, I64, VP, VP, VP]
    L.qlin_group_plan.restype = I32
    L.qlin_group_plan.argtypes = [I64, VP, I32, I64, I64, I64, ctypes.POINTER(I64), ctypes.c_char_p, I64]
    L.qlin_workspace_bytes.restype = I32
    L.qlin_workspace_bytes.argtypes = [P, ctypes.POINTER(I64)]
    L.qlin_shape.restype = I32
    L.qlin_shape.argtypes = [P, ctypes.POINTER(I64), ctypes.POINTER(I64)]
    _lib = L
    return L


def last_error():
    return lib().qlin_last_error().decode()


def qlin_last_error():
    return last_error()


def qlin_last_status():
    return lib().qlin_last_status()


def _check(rc):
    if rc != QLIN_OK:
        raise QlinError(rc, last_error())
    return rc


def _host_ptr(a, dtype):
    """(keep-alive object, address) of a host array, or of a device tensor
    (any object with data_ptr(), passed through as is)."""
    if a is None:
        return None, None
    if hasattr(a, "data_ptr"):
        return a, a.data_ptr()
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data


# ---------------------------------------------------------------- C ABI mirror

def qlin_create(K, N, group, packed_w, scales, zeros):
    """Host numpy arrays in; returns the handle (int) or raises QlinError."""
    p, pp = _host_ptr(packed_w, np.uint32)
    s, sp = _host_ptr(scales, np.uint16)
    z, zp = _host_ptr(zeros, np.uint16)
    h = lib().qlin_create(K, N, group, pp, sp, zp)
    if not h:
        raise QlinError(lib().qlin_last_status(), last_error())
    return h


def qlin_create_symmetric(K, N, group, packed_w, scales):
    p, pp = _host_ptr(packed_w, np.uint32)
    s, sp = _host_ptr(scales, np.uint16)
    h = lib().qlin_create_symmetric(K, N, group, pp, sp)
    if not h:
        raise QlinError(lib().qlin_last_status(), last_error())
    return h


def qlin_quantize(K, N, group, w_ptr, scales_ptr, zeros_ptr, packed_ptr, stream):
    return lib().qlin_quantize(K, N, group, w_ptr, scales_ptr, zeros_ptr, packed_ptr, stream)


def quantize(w, scales, zeros=None, group=128):
    """Device bf16 weights [N, K] -> device packed codes (torch.int32 view of
    uint32 words) [N, K/8] on the frozen grid (scales, zeros device bf16
    [N, K/128]; zeros=None is the symmetric format)."""
    import torch
    N, K = w.shape
    w = w.contiguous()
    packed = torch.empty((N, K // 8), dtype=torch.int32, device=w.device)
    zp = zeros.contiguous().data_ptr() if zeros is not None else None
    _check(qlin_quantize(K, N, group, w.data_ptr(), scales.contiguous().data_ptr(), zp, packed.data_ptr(),
                         torch.cuda.current_stream().cuda_stream))
    return packed


def qlin_forward(h, M, x_ptr, y_ptr, stream):
    return lib().qlin_forward(h, M, x_ptr, y_ptr, stream)


def qlin_forward_path(h, path, split_k, M, x_ptr, y_ptr, stream):
    return lib().qlin_forward_path(h, path, split_k, M, x_ptr, y_ptr, stream)


def qlin_plan(h, path, split_k, M):
    buf = ctypes.create_string_buffer(256)
    _check(lib().qlin_plan(h, path, split_k, M, buf, len(buf)))
    return buf.value.decode()


def _handles(hs):
    arr = (ctypes.c_void_p * len(hs))(*hs)
    return arr


def qlin_forward_group(hs, path, split_k, M, x_ptr, y_ptrs, ws_ptr, ws_bytes, stream):
    """hs: sequence of handles; y_ptrs: sequence of device addresses."""
    ys = (ctypes.c_void_p * len(y_ptrs))(*y_ptrs)
    return lib().qlin_forward_group(len(hs), _handles(hs), path, split_k, M, x_ptr, ys, ws_ptr, ws_bytes, stream)


def qlin_forward_group_noalloc(hs, path, split_k, M, x_ptr, y_ptrs, stream):
    ys = (ctypes.c_void_p * len(y_ptrs))(*y_ptrs)
    return lib().qlin_forward_group_noalloc(len(hs), _handles(hs), path, split_k, M, x_ptr, ys, stream)


def qlin_group_plan(hs, path, split_k, M, ws_bytes=-1):
    """(workspace bytes the plan uses, plan text) for a workspace of ws_bytes (-1: no limit)."""
    need = ctypes.c_int64()
    buf = ctypes.create_string_buffer(256)
    _check(lib().qlin_group_plan(len(hs), _handles(hs), path, split_k, M, ws_bytes, ctypes.byref(need), buf,
                                 len(buf)))
    return need.value, buf.value.decode()


def qlin_workspace_bytes(h):
    b = ctypes.c_int64()
    _check(lib().qlin_workspace_bytes(h, ctypes.byref(b)))
    return b.value


def qlin_destroy(h):
    lib().qlin_destroy(h)


def qlin_unpack_codes(h, q_ptr, stream):
    return lib().qlin_unpack_codes(h, q_ptr, stream)


def qlin_dequantize(h, routine, w_ptr, stream):
    return lib().qlin_dequantize(h, routine, w_ptr, stream)


def qlin_stream_read(buf_ptr, nbytes, grid, sink_ptr, stream):
    return lib().qlin_stream_read(buf_ptr, nbytes, grid, sink_ptr, stream)


def qlin_shape(h):
    K, N = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().qlin_shape(h, ctypes.byref(K), ctypes.byref(N)))
    return K.value, N.value


def qlin_swa_plan(Hq, Hkv, head_dim, nq, T, window, splits=0):
    """(splits, workspace_bytes, text) of the drafter attention's plan."""
    S, ws = ctypes.c_int64(), ctypes.c_int64()
    buf = ctypes.create_string_buffer(256)
    _check(lib().qlin_swa_plan(Hq, Hkv, head_dim, nq, T, window, splits, ctypes.byref(S), ctypes.byref(ws),
                               buf, len(buf)))
    return S.value, ws.value, buf.value.decode()


def qlin_swa_attention(Hq, Hkv, head_dim, nq, T, kv_stride, window, splits, q_ptr, k_ptr, v_ptr, out_ptr,
                       ws_ptr, ws_bytes, stream):
    return lib().qlin_swa_attention(Hq, Hkv, head_dim, nq, T, kv_stride, window, splits, q_ptr, k_ptr, v_ptr,
                                    out_ptr, ws_ptr, ws_bytes, stream)


# ---------------------------------------------------------------- torch wrappers

def swa_attention(q, k, v, window, T=None, splits=0, out=None, workspace=None):
    """Drafter block attention with a symmetric window (include/qlin_attn.h).

    q: CUDA bf16 [Hq, nq, 128]; k, v: CUDA bf16 [Hkv, capacity, 128] with the
    first T tokens valid (T defaults to the capacity); window 0 = full
    attention.  ``workspace`` (a CUDA tensor of at least the planned bytes) is
    allocated when needed and not given.  Returns ``out`` [Hq, nq, 128].
    """
    import torch
    for name, t in (("q", q), ("k", k), ("v", v)):
        if t.dtype != torch.bfloat16 or not t.is_cuda or t.dim() != 3 or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous CUDA bf16 tensor of rank 3")
    Hq, nq, D = q.shape
    Hkv, cap, _ = k.shape
    if v.shape != k.shape:
        raise ValueError("k and v must have the same shape")
    if k.device != q.device or v.device != q.device:
        raise ValueError("q, k and v must be on one device")
    T = cap if T is None else T
    S, ws_bytes, _ = qlin_swa_plan(Hq, Hkv, D, nq, T, window, splits)
    if out is None:
        out = torch.empty((Hq, nq, D), dtype=torch.bfloat16, device=q.device)
    _check_out(out, (Hq, nq, D), q.device)
    if ws_bytes and workspace is None:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=q.device)
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_len = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(qlin_swa_attention(Hq, Hkv, D, nq, T, cap, window, splits, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                              out.data_ptr(), ws_ptr, ws_len, torch.cuda.current_stream().cuda_stream))
    return out


def _check_out(out, shape, device):
    import torch
    if (not isinstance(out, torch.Tensor) or out.dtype != torch.bfloat16 or out.device != device
            or tuple(out.shape) != tuple(shape) or not out.is_contiguous()):
        raise ValueError(f"out must be a contiguous bf16 tensor of shape {tuple(shape)} on {device}")


def new_workspace(nbytes, device=None):
    """A zero-filled device workspace for forward_group (zero before first use)."""
    import torch
    return torch.zeros(max(int(nbytes), 16), dtype=torch.uint8, device=device or "cuda")


def forward_group(lins, x, outs=None, path=PATH_AUTO, split_k=0, workspace=None):
    """One launch over QLinear layers that share x (qlin_forward_group).
    ``workspace``: a zero-filled CUDA uint8 tensor (new_workspace), or None
    for plans without a K split.  Returns the list of outputs."""
    import torch
    K = lins[0].K
    for l in lins:
        if l.K != K:
            raise ValueError("the layers of a group must share K")
    x = lins[0]._check_x(x)
    M = x.shape[0]
    if outs is None:
        outs = [torch.empty((M, l.N), dtype=torch.bfloat16, device=x.device) for l in lins]
    for l, o in zip(lins, outs):
        _check_out(o, (M, l.N), x.device)
    wp, wb = (workspace.data_ptr(), workspace.numel() * workspace.element_size()) if workspace is not None else (None, 0)
    _check(qlin_forward_group([l.h for l in lins], path, split_k, M, x.data_ptr(), [o.data_ptr() for o in outs],
                              wp, wb, torch.cuda.current_stream().cuda_stream))
    return outs


def group_plan(lins, M, path=PATH_AUTO, split_k=0, ws_bytes=-1):
    """(workspace bytes, plan text) of forward_group over lins for M rows."""
    return qlin_group_plan([l.h for l in lins], path, split_k, M, ws_bytes)


class QLinear:
    """One W4A16 linear layer on the current GPU.

    ``packed``/``scales``/``zeros`` are host arrays or device tensors in the
    canonical layout (see include/qlin.h); ``zeros=None`` selects the
    symmetric format.
    """

    def __init__(self, packed, scales, zeros=None, group=128):
        if not hasattr(packed, "data_ptr"):
            packed = np.asarray(packed)
        self.N, K8 = packed.shape
        self.K = K8 * 8
        import torch
        self.device = torch.device("cuda", torch.cuda.current_device())
        if zeros is None:
            self.h = qlin_create_symmetric(self.K, self.N, group, packed, scales)
        else:
            self.h = qlin_create(self.K, self.N, group, packed, scales, zeros)

    def _stream(self):
        import torch
        return torch.cuda.current_stream().cuda_stream

    def _check_x(self, x):
        import torch
        if x.dtype != torch.bfloat16 or x.device != self.device or x.dim() != 2 or x.shape[1] != self.K:
            raise ValueError(f"x must be a bf16 tensor of shape [M, {self.K}] on {self.device}")
        return x.contiguous()

    def forward(self, x, out=None, path=PATH_AUTO, split_k=0, workspace=None):
        """y = x . w^T.  With ``workspace`` (new_workspace) the call goes
        through qlin_forward_group and may use the plans that need it."""
        import torch
        if workspace is not None:
            return forward_group([self], x, None if out is None else [out], path, split_k, workspace)[0]
        x = self._check_x(x)
        M = x.shape[0]
        y = out if out is not None else torch.empty((M, self.N), dtype=torch.bfloat16, device=x.device)
        _check_out(y, (M, self.N), x.device)
        _check(qlin_forward_path(self.h, path, split_k, M, x.data_ptr(), y.data_ptr(), self._stream()))
        return y

    __call__ = forward

    def workspace_bytes(self):
        """Bytes of the handle's own workspace."""
        return qlin_workspace_bytes(self.h)

    def plan(self, M, path=PATH_AUTO, split_k=0):
        return qlin_plan(self.h, path, split_k, M)

    def unpack_codes(self):
        import torch
        q = torch.empty((self.N, self.K), dtype=torch.uint8, device="cuda")
        _check(qlin_unpack_codes(self.h, q.data_ptr(), self._stream()))
        return q

    def dequantize(self, routine=0):
        import torch
        w = torch.empty((self.N, self.K), dtype=torch.bfloat16, device="cuda")
        _check(qlin_dequantize(self.h, routine, w.data_ptr(), self._stream()))
        return w

    def close(self):
        if getattr(self, "h", None):
            qlin_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
