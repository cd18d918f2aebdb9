"""ctypes binding of libminitensor_hip (argument marshalling only).

Every function here builds ``mt_tensor`` descriptors from torch tensors
(device memory owned by torch) and calls the C entry point of the same name
on the current HIP stream; all arithmetic runs in the library's HIP kernels.
Importing this module raises ImportError when the library has not been built
(``python paper_2602_00125_amd/build.py``): there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# MT_LIB_OVERRIDE: a differently built copy of the library (the host-only
# sanitizer build the CPU tests load); default: the in-tree build
LIB_PATH = os.environ.get("MT_LIB_OVERRIDE") or os.path.join(_HERE, "libminitensor_hip.so")
if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run `python paper_2602_00125_amd/build.py`")
lib = ctypes.CDLL(LIB_PATH)

MAX_DIMS = 8
F32, BF16 = 0, 1
ACCUMULATE, REDUCE_INTO, CONV_REUSE_UNFOLD = 1, 2, 4
STATUS = {0: "MT_OK", 1: "MT_ERR_NULL", 2: "MT_ERR_NDIM", 3: "MT_ERR_SHAPE", 4: "MT_ERR_DTYPE",
          5: "MT_ERR_LAYOUT", 6: "MT_ERR_ALIAS", 7: "MT_ERR_WORKSPACE", 8: "MT_ERR_HIP",
          9: "MT_ERR_INVALID"}

EXPORTS = ["mt_linear_fwd", "mt_linear_bwd", "mt_linear_bwd_workspace", "mt_matmul",
           "mt_matmul_workspace",
           "mt_reduce_broadcast_grad", "mt_reduce_broadcast_grad_workspace", "mt_broadcast_shape",
           "mt_matmul_shape", "mt_debug_set", "mt_status_str", "mt_last_error",
           "mt_linear_act_fwd", "mt_act_bwd", "mt_act_bwd_workspace", "mt_mse_loss",
           "mt_mse_loss_workspace", "mt_sgd_step", "mt_adam_step", "mt_rmsprop_step",
           "mt_conv2d_fwd", "mt_conv2d_fwd_workspace", "mt_conv2d_bwd", "mt_conv2d_bwd_workspace",
           "mt_workspace_bytes", "mt_linear_bwd_noalloc"]
NOALLOC_SCRATCH_BYTES = 32 << 20  # MT_NOALLOC_SCRATCH_BYTES
NUM_GEMM_CFG = 16  # tile configurations mt_debug_set("cfg", i) accepts
ACT = {"none": 0, "relu": 1, "sigmoid": 2, "tanh": 3, "gelu": 4}


class MtTensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * MAX_DIMS), ("stride", ctypes.c_int64 * MAX_DIMS)]


_P = ctypes.POINTER(MtTensor)
_vp, _sz, _u32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_uint32
_I64P = ctypes.POINTER(ctypes.c_int64)
lib.mt_linear_fwd.argtypes = [_P, _P, _P, _P, _vp]
lib.mt_linear_bwd.argtypes = [_P, _P, _P, _P, _P, _P, _u32, _vp, _sz, _vp]
lib.mt_linear_bwd_workspace.argtypes = [_P, _P, _P, _P, _P, _P, ctypes.POINTER(_sz)]
lib.mt_linear_bwd_noalloc.argtypes = [_P, _P, _P, _P, _P, _P, _u32, _vp]
lib.mt_matmul.argtypes = [_P, _P, _P, _u32, _vp, _sz, _vp]
lib.mt_matmul_workspace.argtypes = [_P, _P, _P, _u32, ctypes.POINTER(_sz)]
lib.mt_reduce_broadcast_grad.argtypes = [_P, _P, _u32, _vp, _sz, _vp]
lib.mt_reduce_broadcast_grad_workspace.argtypes = [_P, _P, ctypes.POINTER(_sz)]
lib.mt_broadcast_shape.argtypes = [ctypes.c_int32, _I64P, ctypes.c_int32, _I64P,
                                   ctypes.POINTER(ctypes.c_int32), _I64P]
lib.mt_matmul_shape.argtypes = lib.mt_broadcast_shape.argtypes
lib.mt_linear_act_fwd.argtypes = [_P, _P, _P, ctypes.c_int32, _P, _P, _vp]
lib.mt_act_bwd.argtypes = [ctypes.c_int32, _P, _P, _P, _P, _u32, _vp, _sz, _vp]
lib.mt_act_bwd_workspace.argtypes = [ctypes.c_int32, _P, _P, _P, _P, ctypes.POINTER(_sz)]
lib.mt_mse_loss.argtypes = [_P, _P, _P, _P, _vp, _sz, _vp]
lib.mt_mse_loss_workspace.argtypes = [_P, _P, ctypes.POINTER(_sz)]
_f = ctypes.c_float
lib.mt_sgd_step.argtypes = [ctypes.c_int32, _P, _P, _P, _f, _f, _f, _vp]
lib.mt_adam_step.argtypes = [ctypes.c_int32, _P, _P, _P, _P, _f, _f, _f, _f, ctypes.c_int64, _vp]
lib.mt_rmsprop_step.argtypes = [ctypes.c_int32, _P, _P, _P, _f, _f, _f, _vp]
_i32 = ctypes.c_int32
lib.mt_conv2d_fwd.argtypes = [_P, _P, _P, _P, _i32, _i32, _i32, _i32, _vp, _sz, _vp]
lib.mt_conv2d_fwd_workspace.argtypes = [_P, _P, _P, _P, _i32, _i32, _i32, _i32, ctypes.POINTER(_sz)]
lib.mt_conv2d_bwd.argtypes = [_P, _P, _P, _P, _P, _P, _i32, _i32, _i32, _i32, _u32, _vp, _sz, _vp]
lib.mt_conv2d_bwd_workspace.argtypes = [_P, _P, _P, _P, _P, _P, _i32, _i32, _i32, _i32,
                                        ctypes.POINTER(_sz)]
lib.mt_workspace_bytes.argtypes = [ctypes.c_int32, ctypes.POINTER(_P), ctypes.c_int32]
lib.mt_debug_set.argtypes = [ctypes.c_char_p, ctypes.c_int64]
lib.mt_status_str.argtypes = [ctypes.c_int]
lib.mt_status_str.restype = ctypes.c_char_p
lib.mt_last_error.argtypes = []
lib.mt_last_error.restype = ctypes.c_char_p
for _name in EXPORTS:
    if _name not in ("mt_status_str", "mt_last_error", "mt_workspace_bytes"):
        getattr(lib, _name).restype = ctypes.c_int
lib.mt_workspace_bytes.restype = _sz
OP = {"matmul": 0, "matmul_reduce_into": 1, "linear_fwd": 2, "linear_bwd": 3,
      "reduce_broadcast_grad": 4, "mse_loss": 5}


class MtError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        self.name = STATUS.get(status, str(status))
        msg = lib.mt_last_error().decode()
        super().__init__(f"{where}: {self.name}: {msg}")


def _check(status: int, where: str) -> None:
    if status != 0:
        raise MtError(status, where)


def raw_desc(ptr: int, dtype: int, shape, stride) -> MtTensor:
    """A descriptor from raw values (tests of the host-side validation)."""
    d = MtTensor()
    d.data = ptr
    d.dtype = dtype
    d.ndim = len(shape)
    for i, (s, st) in enumerate(zip(shape, stride)):
        d.shape[i] = int(s)
        d.stride[i] = int(st)
    return d


def desc(t: torch.Tensor | None):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("libminitensor_hip works on device tensors (got a CPU tensor)")
    if t.dtype == torch.float32:
        dt = F32
    elif t.dtype == torch.bfloat16:
        dt = BF16
    else:
        raise TypeError(f"unsupported dtype {t.dtype}")
    if t.dim() > MAX_DIMS:
        raise ValueError(f"rank {t.dim()} > {MAX_DIMS}")
    return raw_desc(t.data_ptr(), dt, t.shape, t.stride())


def _ref(d):
    return None if d is None else ctypes.byref(d)


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _ws(workspace):
    if workspace is None:
        return None, 0
    assert workspace.is_cuda
    return workspace.data_ptr(), workspace.numel() * workspace.element_size()


def linear_fwd(x, w, b, y, stream=None) -> None:
    """y = x w^T + b on the device (b may be None)."""
    dx_, dw_, db_, dy_ = desc(x), desc(w), desc(b), desc(y)
    _check(lib.mt_linear_fwd(_ref(dx_), _ref(dw_), _ref(db_), _ref(dy_), _stream(stream)),
           "mt_linear_fwd")


def linear_bwd_workspace(x, w, dy, dx=None, dw=None, db=None) -> int:
    n = _sz(0)
    ds = [desc(t) for t in (x, w, dy, dx, dw, db)]
    _check(lib.mt_linear_bwd_workspace(*[_ref(d) for d in ds], ctypes.byref(n)),
           "mt_linear_bwd_workspace")
    return int(n.value)


def linear_bwd(x, w, dy, dx=None, dw=None, db=None, accumulate=False, workspace=None,
               stream=None) -> None:
    """dx = dy w, dw = dy^T x, db = column sums of dy (None skips an output)."""
    ds = [desc(t) for t in (x, w, dy, dx, dw, db)]
    ptr, nbytes = _ws(workspace)
    _check(lib.mt_linear_bwd(*[_ref(d) for d in ds], ACCUMULATE if accumulate else 0, ptr, nbytes,
                             _stream(stream)), "mt_linear_bwd")


def linear_bwd_noalloc(x, w, dy, dx=None, dw=None, db=None, accumulate=False,
                       stream=None) -> None:
    """linear_bwd with the library's own scratch array as its workspace."""
    ds = [desc(t) for t in (x, w, dy, dx, dw, db)]
    _check(lib.mt_linear_bwd_noalloc(*[_ref(d) for d in ds], ACCUMULATE if accumulate else 0,
                                     _stream(stream)), "mt_linear_bwd_noalloc")


def matmul_workspace(a, b, c, accumulate=False, reduce_into=False) -> int:
    flags = (ACCUMULATE if accumulate else 0) | (REDUCE_INTO if reduce_into else 0)
    n = _sz(0)
    _check(lib.mt_matmul_workspace(_ref(desc(a)), _ref(desc(b)), _ref(desc(c)), flags,
                                   ctypes.byref(n)), "mt_matmul_workspace")
    return int(n.value)


def matmul(a, b, c, accumulate=False, reduce_into=False, workspace=None, stream=None) -> None:
    """c = a @ b with broadcasting (c summed over broadcast axes with reduce_into)."""
    flags = (ACCUMULATE if accumulate else 0) | (REDUCE_INTO if reduce_into else 0)
    da, db_, dc = desc(a), desc(b), desc(c)
    ptr, nbytes = _ws(workspace)
    _check(lib.mt_matmul(_ref(da), _ref(db_), _ref(dc), flags, ptr, nbytes, _stream(stream)),
           "mt_matmul")


def workspace_bytes(op: str, *tensors) -> int:
    """mt_workspace_bytes: the workspace of operation `op` (a key of OP) for
    these tensors (None where the call allows it)."""
    ds = [desc(t) for t in tensors]
    arr = (_P * max(1, len(ds)))(*[ctypes.pointer(d) if d is not None else _P() for d in ds])
    n = lib.mt_workspace_bytes(OP[op], arr, len(ds))
    if n == ctypes.c_size_t(-1).value:
        raise MtError(9, "mt_workspace_bytes")
    return int(n)


def reduce_broadcast_grad_workspace(grad_out, grad_in) -> int:
    n = _sz(0)
    _check(lib.mt_reduce_broadcast_grad_workspace(_ref(desc(grad_out)), _ref(desc(grad_in)),
                                                  ctypes.byref(n)),
           "mt_reduce_broadcast_grad_workspace")
    return int(n.value)


def reduce_broadcast_grad(grad_out, grad_in, accumulate=False, workspace=None, stream=None) -> None:
    """grad_in = grad_out summed over the axes grad_in was broadcast along."""
    ptr, nbytes = _ws(workspace)
    _check(lib.mt_reduce_broadcast_grad(_ref(desc(grad_out)), _ref(desc(grad_in)),
                                        ACCUMULATE if accumulate else 0, ptr, nbytes,
                                        _stream(stream)), "mt_reduce_broadcast_grad")


def _act_code(act) -> int:
    return ACT[act] if isinstance(act, str) else int(act)


def linear_act_fwd(x, w, b, act, y, z=None, stream=None) -> None:
    """y = act(x w^T + b); z (optional) receives the pre-activation."""
    ds = [desc(t) for t in (x, w, b)]
    _check(lib.mt_linear_act_fwd(*[_ref(d) for d in ds], _act_code(act), _ref(desc(z)),
                                 _ref(desc(y)), _stream(stream)), "mt_linear_act_fwd")


def act_bwd_workspace(act, z, dy, dz, db=None) -> int:
    n = _sz(0)
    ds = [desc(t) for t in (z, dy, dz, db)]
    _check(lib.mt_act_bwd_workspace(_act_code(act), *[_ref(d) for d in ds], ctypes.byref(n)),
           "mt_act_bwd_workspace")
    return int(n.value)


def act_bwd(act, z, dy, dz, db=None, accumulate=False, workspace=None, stream=None) -> None:
    """dz = dy * act'(z); db = column sums of dz (None skips it)."""
    ds = [desc(t) for t in (z, dy, dz, db)]
    ptr, nbytes = _ws(workspace)
    _check(lib.mt_act_bwd(_act_code(act), *[_ref(d) for d in ds], ACCUMULATE if accumulate else 0,
                          ptr, nbytes, _stream(stream)), "mt_act_bwd")


def mse_loss_workspace(pred, target) -> int:
    n = _sz(0)
    _check(lib.mt_mse_loss_workspace(_ref(desc(pred)), _ref(desc(target)), ctypes.byref(n)),
           "mt_mse_loss_workspace")
    return int(n.value)


def mse_loss(pred, target, loss=None, dpred=None, workspace=None, stream=None) -> None:
    """loss = mean((pred - target)^2) (1-element tensor), dpred = 2 (pred - target) / N."""
    ds = [desc(t) for t in (pred, target, loss, dpred)]
    ptr, nbytes = _ws(workspace)
    _check(lib.mt_mse_loss(*[_ref(d) for d in ds], ptr, nbytes, _stream(stream)), "mt_mse_loss")


def _desc_array(ts):
    arr = (MtTensor * max(1, len(ts)))()
    for i, t in enumerate(ts):
        arr[i] = desc(t)
    return arr


def sgd_step(params, grads, velocity, lr, momentum=0.0, weight_decay=0.0, stream=None) -> None:
    """In place: v = momentum v + g + weight_decay p; p -= lr v (lists of tensors)."""
    n = len(params)
    assert len(grads) == n and len(velocity) == n
    _check(lib.mt_sgd_step(n, _desc_array(params), _desc_array(grads), _desc_array(velocity),
                           lr, momentum, weight_decay, _stream(stream)), "mt_sgd_step")


def adam_step(params, grads, exp_avg, exp_avg_sq, lr, beta1, beta2, eps, step,
              stream=None) -> None:
    """In place Adam update at step `step` (>= 1) with bias-corrected moments."""
    n = len(params)
    assert len(grads) == n and len(exp_avg) == n and len(exp_avg_sq) == n
    _check(lib.mt_adam_step(n, _desc_array(params), _desc_array(grads), _desc_array(exp_avg),
                            _desc_array(exp_avg_sq), lr, beta1, beta2, eps, int(step),
                            _stream(stream)), "mt_adam_step")


def rmsprop_step(params, grads, sq_avg, lr, alpha, eps, stream=None) -> None:
    """In place: v = alpha v + (1 - alpha) g^2; p -= lr g / sqrt(v + eps)."""
    n = len(params)
    assert len(grads) == n and len(sq_avg) == n
    _check(lib.mt_rmsprop_step(n, _desc_array(params), _desc_array(grads), _desc_array(sq_avg),
                               lr, alpha, eps, _stream(stream)), "mt_rmsprop_step")


def _pair(v):
    return (int(v), int(v)) if isinstance(v, int) else (int(v[0]), int(v[1]))


def conv2d_fwd_workspace(x, w, b, y, stride=1, padding=0) -> int:
    n = _sz(0)
    st, pd = _pair(stride), _pair(padding)
    ds = [desc(t) for t in (x, w, b, y)]
    _check(lib.mt_conv2d_fwd_workspace(*[_ref(d) for d in ds], *st, *pd, ctypes.byref(n)),
           "mt_conv2d_fwd_workspace")
    return int(n.value)


def conv2d_fwd(x, w, b, y, stride=1, padding=0, workspace=None, stream=None) -> None:
    """y = conv2d(x, w) + b (Eq. (6)); y channels-last [N, CO, Ho, Wo]."""
    st, pd = _pair(stride), _pair(padding)
    ds = [desc(t) for t in (x, w, b, y)]
    ptr, nbytes = _ws(workspace)
    _check(lib.mt_conv2d_fwd(*[_ref(d) for d in ds], *st, *pd, ptr, nbytes, _stream(stream)),
           "mt_conv2d_fwd")


def conv2d_bwd_workspace(x, w, dy, dx=None, dw=None, db=None, stride=1, padding=0) -> int:
    n = _sz(0)
    st, pd = _pair(stride), _pair(padding)
    ds = [desc(t) for t in (x, w, dy, dx, dw, db)]
    _check(lib.mt_conv2d_bwd_workspace(*[_ref(d) for d in ds], *st, *pd, ctypes.byref(n)),
           "mt_conv2d_bwd_workspace")
    return int(n.value)


def conv2d_bwd(x, w, dy, dx=None, dw=None, db=None, stride=1, padding=0, accumulate=False,
               workspace=None, reuse_unfold=False, stream=None) -> None:
    """Pullbacks of conv2d: dx, dw, db (None skips one). reuse_unfold: the
    workspace still holds the forward's unfolded input."""
    st, pd = _pair(stride), _pair(padding)
    ds = [desc(t) for t in (x, w, dy, dx, dw, db)]
    ptr, nbytes = _ws(workspace)
    flags = (ACCUMULATE if accumulate else 0) | (CONV_REUSE_UNFOLD if reuse_unfold else 0)
    _check(lib.mt_conv2d_bwd(*[_ref(d) for d in ds], *st, *pd, flags, ptr, nbytes,
                             _stream(stream)), "mt_conv2d_bwd")


def _shape_call(fn, a, b, where):
    aa = (ctypes.c_int64 * max(1, len(a)))(*a)
    bb = (ctypes.c_int64 * max(1, len(b)))(*b)
    out = (ctypes.c_int64 * MAX_DIMS)()
    n = ctypes.c_int32(0)
    _check(fn(len(a), aa, len(b), bb, ctypes.byref(n), out), where)
    return tuple(out[i] for i in range(n.value))


def broadcast_shape(a, b) -> tuple:
    return _shape_call(lib.mt_broadcast_shape, tuple(a), tuple(b), "mt_broadcast_shape")


def matmul_shape(a, b) -> tuple:
    return _shape_call(lib.mt_matmul_shape, tuple(a), tuple(b), "mt_matmul_shape")


def debug_set(key: str, value: int) -> None:
    rc = lib.mt_debug_set(key.encode(), int(value))
    if rc == -1:
        raise KeyError(key)
    if rc != 0:
        raise ValueError(f"{key}={value} out of range")


def status_str(code: int) -> str:
    return lib.mt_status_str(code).decode()
