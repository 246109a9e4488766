"""ctypes binding of liblora_mi355x.so (the C ABI in include/lora.h).

Argument marshalling only: torch provides device memory and the current HIP
stream; every step of the computation runs in the library's HIP kernels.  The
library must be built (``paper_2601_07376_amd.build.build()``); importing this
module without it raises immediately, there is no fallback.

``Table(..., debug=True)`` binds a table, the plans built on it and every op
called with them to the debug build liblora_mi355x_debug.so (overlap checks of
each op's buffers, bounds checks of plan values in the kernels); tables and
plans of the two libraries do not mix.
"""
import ctypes
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblora_mi355x.so")
DEBUG_LIB_PATH = os.path.join(_HERE, "liblora_mi355x_debug.so")

LORA_F32, LORA_BF16 = 0, 1
LORA_DATA_BAD_ID, LORA_DATA_EMPTY_SLOT, LORA_DATA_BAD_SEGMENTS, LORA_DATA_BOUNDS = 1, 2, 4, 8
LORA_BUILD_DEBUG = 1
LORA_PLAN_PERM, LORA_PLAN_M_PERM, LORA_PLAN_SMALL_ROW = 0, 1, 2
STATUS = {0: "LORA_OK", 1: "LORA_ERR_NULL", 2: "LORA_ERR_SHAPE", 3: "LORA_ERR_DTYPE",
          4: "LORA_ERR_ALIGN", 5: "LORA_ERR_RANK", 6: "LORA_ERR_SLOT", 7: "LORA_ERR_DATA",
          8: "LORA_ERR_WORKSPACE", 9: "LORA_ERR_HIP", 10: "LORA_ERR_VALUE",
          11: "LORA_ERR_ALIAS"}

_vp, _i32, _i64, _sz, _f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_float
_pp = ctypes.POINTER(ctypes.c_void_p)

# name -> (restype, argtypes); every symbol declared in include/lora.h
SIGNATURES = {
    "lora_abi_version": (_i32, []),
    "lora_status_string": (ctypes.c_char_p, [_i32]),
    "lora_last_error": (ctypes.c_char_p, []),
    "lora_build_flags": (_i32, []),
    "lora_debug_plan_poke": (_i32, [_vp, _i32, _i32, _i32, _vp]),
    "lora_table_device_bytes": (_sz, [_i32]),
    "lora_table_create": (_i32, [_i32, _i32, _i32, _i32, _vp, _sz, _pp]),
    "lora_table_set": (_i32, [_vp, _i32, _i32, _f32, _vp, _vp]),
    "lora_table_clear": (_i32, [_vp, _i32]),
    "lora_table_upload": (_i32, [_vp, _vp]),
    "lora_table_destroy": (None, [_vp]),
    "lora_plan_workspace_bytes": (_sz, [_i32, _i32]),
    "lora_plan_build": (_i32, [_vp, _i32, _vp, _vp, _vp, _sz, _vp, _pp]),
    "lora_plan_build_segments": (_i32, [_vp, _i32, _i32, _vp, _vp, _vp, _vp, _sz, _vp, _pp]),
    "lora_policy_init": (None, [_vp]),
    "lora_plan_build_policy": (_i32, [_vp, _i32, _vp, _vp, _vp, _vp, _sz, _vp, _pp]),
    "lora_plan_export": (_i32, [_vp] + [_vp] * 11 + [_vp]),
    "lora_plan_check": (_i32, [_vp, _vp, _vp]),
    "lora_plan_destroy": (None, [_vp]),
    "lora_shrink": (_i32, [_vp, _vp, _i32, _i64, _vp, _i64, _vp]),
    "lora_expand": (_i32, [_vp, _vp, _i64, _vp, _i32, _i64, _vp]),
    "lora_apply_workspace_bytes": (_sz, [_vp]),
    "lora_apply": (_i32, [_vp, _vp, _i32, _i64, _vp, _i32, _i64, _vp, _sz, _vp]),
    "lora_apply_noalloc": (_i32, [_vp, _vp, _i32, _i64, _vp, _i32, _i64, _vp]),
    "lora_apply_ids_workspace_bytes": (_sz, [_vp, _i32]),
    "lora_apply_ids": (_i32, [_vp, _i32, _vp, _vp, _i32, _i64, _vp, _i32, _i64, _vp, _sz, _vp]),
    "lora_linear_workspace_bytes": (_sz, [_vp]),
    "lora_linear": (_i32, [_vp, _vp, _i32, _i64, _vp, _i32, _i64, _vp, _i32, _i64, _vp, _sz, _vp]),
    "lora_calibrate_mfma": (_i32, [_i32, _i32, _vp, _vp]),
    "lora_grad_workspace_bytes": (_sz, [_vp]),
    "lora_grad": (_i32, [_vp, _vp, _i32, _i64, _vp, _i32, _i64, _vp, _i64, _vp, _vp, _i32,
                         _vp, _sz, _vp]),
    "lora_grad_x_workspace_bytes": (_sz, [_vp]),
    "lora_grad_x": (_i32, [_vp, _vp, _i32, _i64, _vp, _i32, _i64, _vp, _sz, _vp]),
    "lora_adamw_step": (_i32, [_vp, _i32, _vp]),
    "lora_backward_workspace_bytes": (_sz, [_vp]),
    "lora_backward": (_i32, [_vp, _vp, _i32, _i64, _vp, _i32, _i64, _vp, _i64, _vp, _vp, _i32, _vp,
                             _i32, _i64, _vp, _sz, _vp]),
    "lora_token_loss": (_i32, [_i32, _i32, _i32, _vp, _i32, _i64, _vp, _vp, _vp, _vp, _vp, _vp,
                               ctypes.c_float, ctypes.c_float, _vp, _vp, _vp, _i32, _i64, _vp]),
}

_libs = {}


def lib(debug=False):
    """Load the shared library, or its debug build (raises if it has not been
    built)."""
    path = DEBUG_LIB_PATH if debug else LIB_PATH
    if path not in _libs:
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with "
                               "paper_2601_07376_amd.build.build() (hipcc, gfx950)")
        L = ctypes.CDLL(path)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _libs[path] = L
    return _libs[path]


class LoraError(RuntimeError):
    def __init__(self, status, detail):
        super().__init__(f"{STATUS.get(status, status)}: {detail}")
        self.status = status


def _check(status, L=None):
    """Raise for a nonzero status, with the detail of the library that returned it."""
    if status != 0:
        raise LoraError(status, (L or lib()).lora_last_error().decode())


def _dtype(t):
    if t.dtype == torch.bfloat16:
        return LORA_BF16
    if t.dtype == torch.float32:
        return LORA_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _used_on(stream, *tensors):
    """Tensors allocated here on torch's current stream but used by kernels on
    another stream: tell the caching allocator, so that their memory is not
    handed out again before that stream's work on it has finished."""
    if stream is None:
        return
    if stream.cuda_stream == torch.cuda.current_stream(stream.device).cuda_stream:
        return
    for t in tensors:
        if t is not None:
            t.record_stream(stream)


class Policy(ctypes.Structure):
    """lora_policy (include/lora.h): path selection for testing and tuning;
    -1 keeps the library's choice."""
    _fields_ = [("small_max", ctypes.c_int32), ("small_split", ctypes.c_int32),
                ("split_slices", ctypes.c_int32), ("small_chunks", ctypes.c_int32),
                ("fork", ctypes.c_int32), ("grad_splits", ctypes.c_int32),
                ("block_rows", ctypes.c_int32)]

    def __init__(self, **kw):
        super().__init__()
        lib().lora_policy_init(ctypes.byref(self))
        for k, v in kw.items():
            if v is not None:
                setattr(self, k, int(v))


def _rowmajor(t, name):
    if t.dim() != 2:
        raise ValueError(f"{name} must be a 2-D tensor")
    if t.shape[0] == 0:                  # never touched: any valid leading dimension
        return (t.shape[1] + 7) // 8 * 8
    if t.stride(1) != 1:
        raise ValueError(f"{name} must be a 2-D tensor with unit column stride")
    return t.stride(0)


class Table:
    """Adapter table of one adapted layer (slot -> rank, scale, A, B)."""

    def __init__(self, num_slots, d_in, d_out, w_dtype=torch.bfloat16, device="cuda", debug=False):
        L = self.lib = lib(debug)
        self.num_slots, self.d_in, self.d_out = num_slots, d_in, d_out
        self.w_dtype = w_dtype
        self.device = torch.device(device)
        nbytes = L.lora_table_device_bytes(num_slots)
        self.meta = torch.zeros(max(nbytes, 16), dtype=torch.uint8, device=self.device)
        h = ctypes.c_void_p()
        _check(L.lora_table_create(num_slots, d_in, d_out,
                                   LORA_BF16 if w_dtype == torch.bfloat16 else LORA_F32,
                                   _ptr(self.meta), nbytes, ctypes.byref(h)), L)
        self.handle = h
        self.ranks = [0] * num_slots
        self.scales = [0.0] * num_slots
        self._weights = [None] * num_slots      # keeps A / B alive

    def set(self, slot, A, B, scale):
        """A: [rank, d_in], B: [d_out, rank], contiguous, dtype w_dtype, on device."""
        if not (A.is_contiguous() and B.is_contiguous()):
            raise ValueError("A and B must be contiguous")
        if A.dtype != self.w_dtype or B.dtype != self.w_dtype:
            raise TypeError("A and B must use the table's weight dtype")
        r = A.shape[0]
        if A.shape != (r, self.d_in) or B.shape != (self.d_out, r):
            raise ValueError(f"shapes {tuple(A.shape)}, {tuple(B.shape)} do not match "
                             f"[r, {self.d_in}], [{self.d_out}, r]")
        _check(self.lib.lora_table_set(self.handle, slot, r, float(scale), _ptr(A), _ptr(B)),
               self.lib)
        self.ranks[slot], self.scales[slot] = r, float(scale)
        self._weights[slot] = (A, B)

    def clear(self, slot):
        _check(self.lib.lora_table_clear(self.handle, slot), self.lib)
        self.ranks[slot], self.scales[slot] = 0, 0.0
        self._weights[slot] = None

    def upload(self, stream=None):
        _check(self.lib.lora_table_upload(self.handle, _stream(stream)), self.lib)

    def __del__(self):
        h, L = getattr(self, "handle", None), getattr(self, "lib", None)
        if h is not None and L is not None:
            L.lora_table_destroy(h)
            self.handle = None


class Plan:
    """Row grouping of one batch (built on the device, no host synchronisation)."""

    def __init__(self, table, idx=None, mask=None, seg_offsets=None, seg_adapter=None, n=None,
                 stream=None, policy=None):
        L = self.lib = table.lib
        self.table = table
        if idx is not None:
            n = idx.numel()
        elif n is None:
            raise ValueError("segment plans need n")
        self.n = int(n)
        self.ws = torch.empty(max(L.lora_plan_workspace_bytes(self.n, table.num_slots), 16),
                              dtype=torch.uint8, device=table.device)
        _used_on(stream, self.ws)
        self._keep = (idx, mask, seg_offsets, seg_adapter)
        h = ctypes.c_void_p()
        if policy is not None and idx is None:
            raise ValueError("a policy applies to plans built from ids")
        if idx is not None and policy is not None:
            pol = policy if isinstance(policy, Policy) else Policy(**policy)
            _check(L.lora_plan_build_policy(table.handle, self.n, _ptr(idx), _ptr(mask),
                                            ctypes.byref(pol), _ptr(self.ws), self.ws.numel(),
                                            _stream(stream), ctypes.byref(h)), L)
        elif idx is not None:
            _check(L.lora_plan_build(table.handle, self.n, _ptr(idx), _ptr(mask), _ptr(self.ws),
                                     self.ws.numel(), _stream(stream), ctypes.byref(h)), L)
        else:
            _check(L.lora_plan_build_segments(table.handle, self.n, seg_adapter.numel(),
                                              _ptr(seg_offsets), _ptr(seg_adapter), _ptr(mask),
                                              _ptr(self.ws), self.ws.numel(), _stream(stream),
                                              ctypes.byref(h)), L)
        self.handle = h

    def export(self, stream=None):
        S, n = self.table.num_slots, self.n
        arrs = {k: np.zeros(S, np.int32) for k in ("counts", "m_counts")}
        arrs.update({k: np.zeros(S + 1, np.int32) for k in ("offsets", "m_offsets")})
        arrs.update({k: np.zeros(max(n, 1), np.int32)
                     for k in ("perm", "run_start", "run_len", "run_adapter", "m_perm")})
        n_runs = ctypes.c_int32()
        flags = ctypes.c_uint32()
        p = lambda k: arrs[k].ctypes.data_as(ctypes.c_void_p)
        _check(self.lib.lora_plan_export(self.handle, p("counts"), p("offsets"), p("perm"),
                                         ctypes.byref(n_runs), p("run_start"), p("run_len"),
                                         p("run_adapter"), p("m_counts"), p("m_offsets"),
                                         p("m_perm"), ctypes.byref(flags), _stream(stream)),
               self.lib)
        n_act, m_n_act, nr = int(arrs["offsets"][-1]), int(arrs["m_offsets"][-1]), n_runs.value
        return dict(counts=arrs["counts"], offsets=arrs["offsets"], perm=arrs["perm"][:n_act],
                    n_runs=nr, run_start=arrs["run_start"][:nr], run_len=arrs["run_len"][:nr],
                    run_adapter=arrs["run_adapter"][:nr], m_counts=arrs["m_counts"],
                    m_offsets=arrs["m_offsets"], m_perm=arrs["m_perm"][:m_n_act],
                    data_flags=flags.value)

    def check(self, stream=None):
        """Data-error flags (LORA_DATA_* bits); 0 when clean."""
        flags = ctypes.c_uint32()
        st = self.lib.lora_plan_check(self.handle, ctypes.byref(flags), _stream(stream))
        if st not in (0, 7):
            _check(st, self.lib)
        return flags.value

    def debug_poke(self, array, index, value, stream=None):
        """Debug library only: overwrite one row id of the plan (a test hook
        for the kernels' bounds checks; array LORA_PLAN_*)."""
        _check(self.lib.lora_debug_plan_poke(self.handle, int(array), int(index), int(value),
                                             _stream(stream)), self.lib)

    def __del__(self):
        h, L = getattr(self, "handle", None), getattr(self, "lib", None)
        if h is not None and L is not None:
            L.lora_plan_destroy(h)
            self.handle = None


def shrink(plan, X, H=None, stream=None):
    """H[t, :r_a] = X[t] A_a^T (float32 H; untouched elsewhere)."""
    if H is None:
        r = max(max(plan.table.ranks), 1)
        H = torch.zeros(plan.n, (r + 7) // 8 * 8, dtype=torch.float32, device=X.device)
        _used_on(stream, H)
    _check(plan.lib.lora_shrink(plan.handle, _ptr(X), _dtype(X), _rowmajor(X, "X"), _ptr(H),
                                _rowmajor(H, "H"), _stream(stream)), plan.lib)
    return H


def expand(plan, H, Y, stream=None):
    """Y[t] += s_a H[t, :r_a] B_a^T in place."""
    _check(plan.lib.lora_expand(plan.handle, _ptr(H), _rowmajor(H, "H"), _ptr(Y), _dtype(Y),
                                _rowmajor(Y, "Y"), _stream(stream)), plan.lib)
    return Y


def apply_workspace(plan):
    return torch.empty(max(plan.lib.lora_apply_workspace_bytes(plan.handle), 16), dtype=torch.uint8,
                       device=plan.table.device)


def apply(plan, X, Y, ws=None, stream=None):
    """Y[t] += s_a (X[t] A_a^T) B_a^T in place."""
    if ws is None:
        ws = apply_workspace(plan)
        _used_on(stream, ws)
    _check(plan.lib.lora_apply(plan.handle, _ptr(X), _dtype(X), _rowmajor(X, "X"), _ptr(Y),
                               _dtype(Y), _rowmajor(Y, "Y"), _ptr(ws), ws.numel(), _stream(stream)), plan.lib)
    return Y


def apply_noalloc(plan, X, Y, stream=None):
    """apply() with the library's fixed per-GPU scratch instead of a workspace:
    allocates nothing (for graph capture and loops that must not allocate)."""
    _check(plan.lib.lora_apply_noalloc(plan.handle, _ptr(X), _dtype(X), _rowmajor(X, "X"), _ptr(Y),
                                       _dtype(Y), _rowmajor(Y, "Y"), _stream(stream)), plan.lib)
    return Y


def apply_ids_workspace(table, n):
    return torch.empty(max(table.lib.lora_apply_ids_workspace_bytes(table.handle, n), 16),
                       dtype=torch.uint8, device=table.device)


def apply_ids(table, idx, X, Y, ws=None, stream=None):
    """apply() for a small batch without a plan: Y[t] += s_a (X[t] A_a^T) B_a^T
    for idx[t] = a, two launches (n <= 1024, bfloat16 X and weights)."""
    n = int(idx.numel())
    if ws is None:
        ws = apply_ids_workspace(table, n)
        _used_on(stream, ws)
    _check(table.lib.lora_apply_ids(table.handle, n, _ptr(idx), _ptr(X), _dtype(X),
                                    _rowmajor(X, "X"), _ptr(Y), _dtype(Y), _rowmajor(Y, "Y"),
                                    _ptr(ws), ws.numel(), _stream(stream)), table.lib)
    return Y


def linear_workspace(plan):
    return torch.empty(max(plan.lib.lora_linear_workspace_bytes(plan.handle), 16), dtype=torch.uint8,
                       device=plan.table.device)


def linear(plan, X, W, Y, ws=None, stream=None):
    """Y = X W^T + s_a (X A_a^T) B_a^T (rows with no adapter: X W^T); Y written."""
    if ws is None:
        ws = linear_workspace(plan)
        _used_on(stream, ws)
    _check(plan.lib.lora_linear(plan.handle, _ptr(X), _dtype(X), _rowmajor(X, "X"), _ptr(W),
                                _dtype(W), _rowmajor(W, "W"), _ptr(Y), _dtype(Y), _rowmajor(Y, "Y"),
                                _ptr(ws), ws.numel(), _stream(stream)), plan.lib)
    return Y


def grad_workspace(plan):
    return torch.empty(max(plan.lib.lora_grad_workspace_bytes(plan.handle), 16), dtype=torch.uint8,
                       device=plan.table.device)


def grad(plan, X, dY, dA=None, dB=None, H_saved=None, accumulate=False, ws=None, stream=None):
    """Masked adapter-local gradients.  dA / dB: lists (per slot) of float32
    tensors or None; allocated for every live slot when not given."""
    t = plan.table
    if dA is None:
        dA = [torch.empty(r, t.d_in, dtype=torch.float32, device=X.device) if r > 0 else None
              for r in t.ranks]
        _used_on(stream, *dA)
    if dB is None:
        dB = [torch.empty(t.d_out, r, dtype=torch.float32, device=X.device) if r > 0 else None
              for r in t.ranks]
        _used_on(stream, *dB)
    if ws is None:
        ws = grad_workspace(plan)
        _used_on(stream, ws)
    pa = (ctypes.c_void_p * t.num_slots)(*[g.data_ptr() if g is not None else None for g in dA])
    pb = (ctypes.c_void_p * t.num_slots)(*[g.data_ptr() if g is not None else None for g in dB])
    ldh = _rowmajor(H_saved, "H_saved") if H_saved is not None else 0
    _check(plan.lib.lora_grad(plan.handle, _ptr(X), _dtype(X), _rowmajor(X, "X"), _ptr(dY),
                              _dtype(dY), _rowmajor(dY, "dY"), _ptr(H_saved), ldh, pa, pb,
                              1 if accumulate else 0, _ptr(ws), ws.numel(), _stream(stream)), plan.lib)
    return dA, dB


def grad_x_workspace(plan):
    return torch.empty(max(plan.lib.lora_grad_x_workspace_bytes(plan.handle), 16), dtype=torch.uint8,
                       device=plan.table.device)


def grad_x(plan, dY, dX, ws=None, stream=None):
    """dX[t] += s_a (dY[t] B_a) A_a in place over the plan's masked rows."""
    if ws is None:
        ws = grad_x_workspace(plan)
        _used_on(stream, ws)
    _check(plan.lib.lora_grad_x(plan.handle, _ptr(dY), _dtype(dY), _rowmajor(dY, "dY"), _ptr(dX),
                                _dtype(dX), _rowmajor(dX, "dX"), _ptr(ws), ws.numel(), _stream(stream)), plan.lib)
    return dX


def backward_workspace(plan):
    return torch.empty(max(plan.lib.lora_backward_workspace_bytes(plan.handle), 16), dtype=torch.uint8,
                       device=plan.table.device)


def backward(plan, X, dY, dX, dA=None, dB=None, H_saved=None, accumulate=False, ws=None,
             stream=None):
    """grad and grad_x of one backward step in one call (the input gradient
    beside the adapter gradients); returns (dA, dB, dX)."""
    t = plan.table
    if dA is None:
        dA = [torch.empty(r, t.d_in, dtype=torch.float32, device=X.device) if r > 0 else None
              for r in t.ranks]
        _used_on(stream, *dA)
    if dB is None:
        dB = [torch.empty(t.d_out, r, dtype=torch.float32, device=X.device) if r > 0 else None
              for r in t.ranks]
        _used_on(stream, *dB)
    if ws is None:
        ws = backward_workspace(plan)
        _used_on(stream, ws)
    pa = (ctypes.c_void_p * t.num_slots)(*[g.data_ptr() if g is not None else None for g in dA])
    pb = (ctypes.c_void_p * t.num_slots)(*[g.data_ptr() if g is not None else None for g in dB])
    ldh = _rowmajor(H_saved, "H_saved") if H_saved is not None else 0
    _check(plan.lib.lora_backward(plan.handle, _ptr(X), _dtype(X), _rowmajor(X, "X"), _ptr(dY),
                                  _dtype(dY), _rowmajor(dY, "dY"), _ptr(H_saved), ldh, pa, pb,
                                  1 if accumulate else 0, _ptr(dX), _dtype(dX), _rowmajor(dX, "dX"),
                                  _ptr(ws), ws.numel(), _stream(stream)), plan.lib)
    return dA, dB, dX


class AdamWTensor(ctypes.Structure):
    """lora_adamw_tensor (include/lora.h)."""
    _fields_ = [("p", ctypes.c_void_p), ("m", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("g", ctypes.c_void_p), ("p_bf16", ctypes.c_void_p), ("n", ctypes.c_int64),
                ("step", ctypes.c_int32), ("lr", ctypes.c_float), ("beta1", ctypes.c_float),
                ("beta2", ctypes.c_float), ("eps", ctypes.c_float),
                ("weight_decay", ctypes.c_float)]


def adamw_step(params, stream=None):
    """One AdamW step over a group of tensors, each with its own state.

    params: sequence of dicts with float32 device tensors ``p``, ``m``, ``v``,
    ``g`` of one size, optional ``p_bf16`` (bfloat16, same size; receives the
    rounded update), and ``step``, ``lr``, ``beta1``, ``beta2``, ``eps``,
    ``weight_decay``.  Tensors are passed as flat arrays, so they must be
    contiguous."""
    recs = (AdamWTensor * max(len(params), 1))()
    for i, q in enumerate(params):
        n = q["p"].numel()
        for k in ("p", "m", "v", "g"):
            t = q[k]
            if t.dtype != torch.float32 or not t.is_contiguous() or t.numel() != n:
                raise ValueError(f"params[{i}].{k}: contiguous float32 of {n} elements expected")
        pb = q.get("p_bf16")
        if pb is not None and (pb.dtype != torch.bfloat16 or not pb.is_contiguous() or pb.numel() != n):
            raise ValueError(f"params[{i}].p_bf16: contiguous bfloat16 of {n} elements expected")
        recs[i] = AdamWTensor(q["p"].data_ptr(), q["m"].data_ptr(), q["v"].data_ptr(),
                              q["g"].data_ptr(), pb.data_ptr() if pb is not None else None, n,
                              int(q["step"]), float(q["lr"]), float(q["beta1"]),
                              float(q["beta2"]), float(q["eps"]), float(q["weight_decay"]))
    _check(lib().lora_adamw_step(ctypes.cast(recs, ctypes.c_void_p), len(params), _stream(stream)))


LOSS_CE, LOSS_IS, LOSS_PPO = 0, 1, 2


def token_loss(kind, logits, target, dlogits, loss, logp=None, weight=None, mask=None,
               old_logp=None, adv=None, corr=None, clip_lo=0.2, clip_hi=0.2, stream=None):
    """Masked token-level loss (kind LOSS_CE / LOSS_IS / LOSS_PPO): per-token
    ``loss`` and ``logp`` and the gradient ``dlogits`` = dL/dlogits, in place."""
    n, vocab = logits.shape
    _check(lib().lora_token_loss(int(kind), n, vocab, _ptr(logits), _dtype(logits),
                                 _rowmajor(logits, "logits"), _ptr(target), _ptr(weight), _ptr(mask),
                                 _ptr(old_logp), _ptr(adv), _ptr(corr), float(clip_lo),
                                 float(clip_hi), _ptr(loss), _ptr(logp), _ptr(dlogits),
                                 _dtype(dlogits), _rowmajor(dlogits, "dlogits"), _stream(stream)))
    return loss, logp, dlogits
