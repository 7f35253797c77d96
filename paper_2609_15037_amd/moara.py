"""Python binding of the MoARa HIP library (include/moara.h).

Argument marshalling only: every computation runs in libmoara.so's HIP kernels.
The function names mirror the C ABI. Tensors are torch tensors on the GPU (only
their data pointers, shapes and dtypes are used); before any pointer reaches
the library the binding checks that each buffer has exactly the shape, dtype,
device and contiguity the state expects, so a mismatched buffer raises here
instead of being read out of bounds on the GPU.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmoara.so")

MOARA_OK, MOARA_E_ARG, MOARA_E_SHAPE, MOARA_E_RANK = 0, -1, -2, -3
MOARA_E_UNSUPPORTED, MOARA_E_HIP, MOARA_E_OOM, MOARA_E_STATE = -4, -5, -6, -7
(MOARA_Q, MOARA_K, MOARA_V, MOARA_O, MOARA_GATE, MOARA_UP, MOARA_DOWN,
 MOARA_EXP_GATE, MOARA_EXP_UP, MOARA_EXP_DOWN) = range(10)
MOARA_NUM_MODULES = 10
MOARA_SIDE_AUTO, MOARA_SIDE_LEFT, MOARA_SIDE_RIGHT = 0, 1, 2
MOARA_F32, MOARA_BF16 = 0, 1
MOARA_T_P, MOARA_T_EXP_AVG, MOARA_T_EXP_AVG_SQ, MOARA_T_MAG_AVG, MOARA_T_MAG_AVG_SQ, MOARA_T_STEP = range(6)
MOARA_KERN_DECOMPOSE, MOARA_KERN_PROJECT, MOARA_KERN_BACKPROJ, MOARA_KERN_REFRESH, MOARA_KERN_ALIGN = range(5)
MOARA_NUM_KERNELS = 5

EXPORTED = (
    "moara_default_config", "moara_allocate_ranks", "moara_resolve_matrix", "moara_state_bytes",
    "moara_create_state", "moara_refresh_projector", "moara_step", "moara_step_noalloc", "moara_alignment",
    "moara_get_tensor",
    "moara_set_tensor", "moara_refresh_info",
    "moara_set_timing", "moara_kernel_stats", "moara_reset_kernel_stats", "moara_matrix_info",
    "moara_destroy_state", "moara_last_error", "moara_version",
)


class MoaraError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"moara status {status}: {message}")
        self.status = status


class moara_config(ctypes.Structure):
    _fields_ = [
        ("rank_table", ctypes.c_int32 * MOARA_NUM_MODULES),
        ("block_size", ctypes.c_int32),
        ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
        ("adam_eps", ctypes.c_float), ("decomp_eps", ctypes.c_float),
        ("scale", ctypes.c_float), ("weight_decay", ctypes.c_float),
        ("refresh_interval", ctypes.c_int32), ("bias_correction", ctypes.c_int32),
        ("decompose", ctypes.c_int32), ("weight_dtype", ctypes.c_int32),
        ("grad_dtype", ctypes.c_int32), ("operand_dtype", ctypes.c_int32),
        ("refresh_oversample", ctypes.c_int32), ("refresh_iters", ctypes.c_int32),
        ("refresh_seed", ctypes.c_uint64),
        ("zero_grad_mode", ctypes.c_int32), ("moment_dtype", ctypes.c_int32),
    ]


class moara_matrix_desc(ctypes.Structure):
    _fields_ = [
        ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
        ("module", ctypes.c_int32), ("rank_override", ctypes.c_int32),
        ("side", ctypes.c_int32), ("reserved", ctypes.c_int32),
    ]


_lib = None


def lib():
    """Load libmoara.so (built in-tree by paper_2609_15037_amd.build). Raises if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_15037_amd.build` "
                           "(there is no fallback implementation)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, u32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32
    P = ctypes.POINTER
    sig = {
        "moara_default_config": (ctypes.c_int, [P(moara_config)]),
        "moara_allocate_ranks": (ctypes.c_int, [i32, u32, u32, u32, i32, P(i32)]),
        "moara_resolve_matrix": (ctypes.c_int, [P(moara_config), P(moara_matrix_desc), P(i32), P(i32)]),
        "moara_state_bytes": (ctypes.c_int, [P(moara_config), P(moara_matrix_desc), i32, P(i64), P(i64)]),
        "moara_create_state": (ctypes.c_int, [P(moara_config), P(moara_matrix_desc), i32, vp, P(vp)]),
        "moara_refresh_projector": (ctypes.c_int, [vp, P(vp), P(ctypes.c_uint8), vp]),
        "moara_step": (ctypes.c_int, [vp, P(vp), P(vp), P(ctypes.c_uint8), ctypes.c_float, vp]),
        "moara_step_noalloc": (ctypes.c_int, [vp, P(vp), P(vp), P(ctypes.c_uint8), ctypes.c_float, vp]),
        "moara_alignment": (ctypes.c_int, [vp, P(vp), P(ctypes.c_uint8), P(ctypes.c_double), vp]),
        "moara_get_tensor": (ctypes.c_int, [vp, i32, i32, vp, ctypes.c_size_t, vp]),
        "moara_set_tensor": (ctypes.c_int, [vp, i32, i32, vp, ctypes.c_size_t, vp]),
        "moara_refresh_info": (ctypes.c_int, [vp, i32, P(i32), P(i32), P(i32), P(ctypes.c_float), vp]),
        "moara_set_timing": (ctypes.c_int, [vp, i32]),
        "moara_kernel_stats": (ctypes.c_int, [vp, i32, P(i64), P(ctypes.c_double), vp]),
        "moara_reset_kernel_stats": (ctypes.c_int, [vp, vp]),
        "moara_matrix_info": (ctypes.c_int, [vp, i32, P(i64), P(i64), P(i32), P(i32), P(i32)]),
        "moara_destroy_state": (None, [vp]),
        "moara_last_error": (ctypes.c_char_p, []),
        "moara_version": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def _check(rc: int):
    if rc != MOARA_OK:
        raise MoaraError(rc, lib().moara_last_error().decode(errors="replace"))


def moara_version() -> str:
    return lib().moara_version().decode()


def moara_last_error() -> str:
    return lib().moara_last_error().decode(errors="replace")


def moara_default_config(**overrides) -> moara_config:
    c = moara_config()
    _check(lib().moara_default_config(ctypes.byref(c)))
    for k, v in overrides.items():
        if k == "rank_table":
            for i in range(MOARA_NUM_MODULES):
                c.rank_table[i] = int(v[i]) if i < len(v) else 0
        else:
            setattr(c, k, v)
    return c


def moara_allocate_ranks(r_base: int, types: Sequence[int], donors: Sequence[int], receivers: Sequence[int],
                         delta_r: int) -> List[int]:
    mask = lambda xs: sum(1 << int(x) for x in set(xs))
    out = (ctypes.c_int32 * MOARA_NUM_MODULES)()
    _check(lib().moara_allocate_ranks(int(r_base), mask(types), mask(donors), mask(receivers), int(delta_r), out))
    return list(out)


def flatten_shape(shape) -> tuple:
    """The matrix a weight tensor is treated as (Appendix B.1, flattened tensors): the
    first axis stays, all remaining axes are flattened into the column axis, so a
    contiguous s0 x s1 x ... tensor is the row-major s0 x (s1 * ...) matrix."""
    shape = tuple(int(x) for x in shape)
    if len(shape) < 2:
        raise ValueError(f"a weight needs at least two axes, got shape {shape}")
    n = 1
    for x in shape[1:]:
        n *= x
    return shape[0], n


def make_descs(shapes_modules) -> ctypes.Array:
    """[(rows, cols, module[, rank_override[, side]]), ...] -> moara_matrix_desc array.
    An entry may also start with a full tensor shape, ((s0, s1, ...), module[, ...]),
    which is flattened by flatten_shape."""
    arr = (moara_matrix_desc * len(shapes_modules))()
    for i, t in enumerate(shapes_modules):
        if isinstance(t[0], (tuple, list)):
            t = (*flatten_shape(t[0]), *t[1:])
        arr[i].rows, arr[i].cols, arr[i].module = int(t[0]), int(t[1]), int(t[2])
        arr[i].rank_override = int(t[3]) if len(t) > 3 else 0
        arr[i].side = int(t[4]) if len(t) > 4 else MOARA_SIDE_AUTO
        arr[i].reserved = 0
    return arr


def moara_resolve_matrix(cfg: moara_config, desc: moara_matrix_desc):
    r, s = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().moara_resolve_matrix(ctypes.byref(cfg), ctypes.byref(desc), ctypes.byref(r), ctypes.byref(s)))
    return r.value, s.value


def moara_state_bytes(cfg: moara_config, descs) -> tuple:
    a, b = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().moara_state_bytes(ctypes.byref(cfg), descs, len(descs), ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


def _stream_ptr(stream) -> Optional[int]:
    if stream is None:
        return None
    if isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)


class State:
    """Owns one moara_state*. Holds the shapes and dtypes the buffers are checked against."""

    def __init__(self, handle: int, cfg: moara_config, descs):
        self.handle = handle
        self.cfg = cfg
        self.n = len(descs)
        self.shapes = [(int(d.rows), int(d.cols)) for d in descs]
        self.info = [moara_matrix_info(self, i) for i in range(self.n)]
        import torch
        self.device = torch.cuda.current_device()   # the library creates the state on the current device

    def __del__(self):
        if getattr(self, "handle", None):
            try:
                lib().moara_destroy_state(self.handle)
            except Exception:
                pass
            self.handle = None


def moara_create_state(cfg: moara_config, descs, stream=None) -> State:
    h = ctypes.c_void_p()
    _check(lib().moara_create_state(ctypes.byref(cfg), descs, len(descs), _stream_ptr(stream), ctypes.byref(h)))
    return State(h.value, cfg, descs)


def moara_destroy_state(st: State):
    if st.handle:
        lib().moara_destroy_state(st.handle)
        st.handle = None


def _ptr_array(st: State, tensors, what: str, dtype_name: str, active):
    import torch
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16}[dtype_name]
    if len(tensors) != st.n:
        raise ValueError(f"{what}: expected {st.n} tensors, got {len(tensors)}")
    arr = (ctypes.c_void_p * st.n)()
    for i, t in enumerate(tensors):
        if active is not None and not active[i]:
            arr[i] = t.data_ptr() if t is not None else None
            if t is None:
                continue
        if t is None:
            raise ValueError(f"{what}[{i}] is None for an active matrix")
        if (not t.is_cuda or t.dtype != tdt or not t.is_contiguous() or t.dim() < 2
                or flatten_shape(t.shape) != st.shapes[i]):
            raise ValueError(f"{what}[{i}]: need a contiguous {dtype_name} CUDA tensor of shape {st.shapes[i]} "
                             f"(or with that flattened shape), got {tuple(t.shape)} {t.dtype} cuda={t.is_cuda} "
                             f"contiguous={t.is_contiguous()}")
        if t.device.index != st.device:   # the kernels would read another GPU's memory
            raise ValueError(f"{what}[{i}] is on {t.device}, the state lives on cuda:{st.device}")
        arr[i] = t.data_ptr()
    return arr


def _active_array(st: State, active):
    if active is None:
        return None
    a = np.ascontiguousarray(np.asarray(active, dtype=np.uint8))
    if a.shape != (st.n,):
        raise ValueError("active must have one entry per matrix")
    return (ctypes.c_uint8 * st.n)(*a.tolist())


def moara_refresh_projector(st: State, grads, active=None, stream=None):
    g = _ptr_array(st, grads, "grads", "f32", active)
    _check(lib().moara_refresh_projector(st.handle, g, _active_array(st, active), _stream_ptr(stream)))


def moara_alignment(st: State, grads, active=None, stream=None) -> np.ndarray:
    """moara_alignment of the C ABI: S(W, t) = cos(G, G_recon) per matrix as a float64
    array of n entries (NaN for inactive matrices)."""
    g = _ptr_array(st, grads, "grads", "f32", active)
    out = np.full(st.n, np.nan, dtype=np.float64)
    _check(lib().moara_alignment(st.handle, g, _active_array(st, active),
                                 out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), _stream_ptr(stream)))
    return out


class StepArgs:
    """Pointer arrays of a fixed set of weight and gradient tensors, checked once, for callers
    that step the same buffers many times (the per-call checks cost microseconds per matrix)."""

    def __init__(self, st: State, weights, grads):
        wd = "bf16" if st.cfg.weight_dtype == MOARA_BF16 else "f32"
        self.w = _ptr_array(st, weights, "weights", wd, None)
        self.g = _ptr_array(st, grads, "grads", "f32", None)
        self.keep = (list(weights), list(grads))   # the tensors must outlive the arrays


def moara_active_mask(st: State, active):
    """An active mask in the C layout (one uint8 per matrix), reusable across calls."""
    return _active_array(st, active)


MOARA_NOALLOC_SCRATCH_BYTES = 1024 << 20


def moara_step(st: State, weights, grads, lr: float, active=None, stream=None, args: StepArgs = None,
               noalloc: bool = False):
    """moara_step of the C ABI (moara_step_noalloc with noalloc=True). With `args` (a
    StepArgs of the same tensors) the pointer arrays are reused and `weights` / `grads` are
    ignored; `active` may be a mask from moara_active_mask."""
    if args is not None:
        w, g = args.w, args.g
    else:
        wd = "bf16" if st.cfg.weight_dtype == MOARA_BF16 else "f32"
        # zero_grad_mode 1 updates the weights of inactive matrices too: check all of them
        w = _ptr_array(st, weights, "weights", wd, None if st.cfg.zero_grad_mode == 1 else active)
        g = _ptr_array(st, grads, "grads", "f32", active)
    act = active if isinstance(active, ctypes.Array) else _active_array(st, active)
    fn = lib().moara_step_noalloc if noalloc else lib().moara_step
    _check(fn(st.handle, w, g, act, ctypes.c_float(lr), _stream_ptr(stream)))


def moara_step_noalloc(st: State, weights, grads, lr: float, active=None, stream=None, args: StepArgs = None):
    """moara_step_noalloc of the C ABI: moara_step without any device allocation."""
    moara_step(st, weights, grads, lr, active=active, stream=stream, args=args, noalloc=True)


def _tensor_shape(st: State, mat: int, which: int):
    m, n = st.shapes[mat]
    rows, cols, r, side, k = st.info[mat]
    s = m if side == MOARA_SIDE_LEFT else n
    if which == MOARA_T_P:
        return (s, r)
    if which in (MOARA_T_EXP_AVG, MOARA_T_EXP_AVG_SQ):
        return (r, n) if side == MOARA_SIDE_LEFT else (m, r)
    if which in (MOARA_T_MAG_AVG, MOARA_T_MAG_AVG_SQ):
        return (m, k)
    raise ValueError(which)


def moara_get_tensor(st: State, mat: int, which: int, stream=None):
    if which == MOARA_T_STEP:
        out = np.zeros(1, dtype=np.int64)
    else:
        out = np.zeros(_tensor_shape(st, mat, which), dtype=np.float32)
    _check(lib().moara_get_tensor(st.handle, int(mat), int(which), out.ctypes.data, out.nbytes, _stream_ptr(stream)))
    return int(out[0]) if which == MOARA_T_STEP else out


def moara_set_tensor(st: State, mat: int, which: int, value, stream=None):
    if which == MOARA_T_STEP:
        a = np.asarray([value], dtype=np.int64)
    else:
        a = np.ascontiguousarray(np.asarray(value, dtype=np.float32))
        if a.shape != _tensor_shape(st, mat, which):
            raise ValueError(f"tensor {which} of matrix {mat} must have shape {_tensor_shape(st, mat, which)}")
    _check(lib().moara_set_tensor(st.handle, int(mat), int(which), a.ctypes.data, a.nbytes, _stream_ptr(stream)))


def moara_refresh_info(st: State, mat: int, stream=None) -> dict:
    """moara_refresh_info of the C ABI: the record of the matrix's last refresh."""
    sw, cv, rk, off = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32(), ctypes.c_float()
    _check(lib().moara_refresh_info(st.handle, int(mat), ctypes.byref(sw), ctypes.byref(cv), ctypes.byref(rk),
                                    ctypes.byref(off), _stream_ptr(stream)))
    return {"sweeps": sw.value, "converged": bool(cv.value), "rank": rk.value, "offdiag": off.value}


def moara_set_timing(st: State, enable: bool):
    _check(lib().moara_set_timing(st.handle, 1 if enable else 0))


def moara_kernel_stats(st: State, kernel: int, stream=None):
    n, ms = ctypes.c_int64(), ctypes.c_double()
    _check(lib().moara_kernel_stats(st.handle, int(kernel), ctypes.byref(n), ctypes.byref(ms), _stream_ptr(stream)))
    return n.value, ms.value


def moara_reset_kernel_stats(st: State, stream=None):
    _check(lib().moara_reset_kernel_stats(st.handle, _stream_ptr(stream)))


def moara_matrix_info(st: State, mat: int):
    a, b = ctypes.c_int64(), ctypes.c_int64()
    r, s, k = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    _check(lib().moara_matrix_info(st.handle, int(mat), ctypes.byref(a), ctypes.byref(b), ctypes.byref(r),
                                   ctypes.byref(s), ctypes.byref(k)))
    return a.value, b.value, r.value, s.value, k.value
