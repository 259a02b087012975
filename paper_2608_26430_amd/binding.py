"""ctypes binding of libframeft.so: argument marshalling only.

Every computation happens in the HIP library; this module turns torch
tensors into device pointers and the current torch stream into the hipStream_t
of the C ABI (include/frameft.h).  There is no fallback: if the library is not
built, or a call fails, a FrameFTError is raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libframeft.so")
_lib = None

FF_F32, FF_BF16 = 0, 1
_STATUS = {0: "FF_OK", 1: "FF_EINVAL", 2: "FF_ENOTFF", 3: "FF_EUNSUPPORTED", 4: "FF_ENOMEM",
           5: "FF_EDEVICE"}


class FrameFTError(RuntimeError):
    """A libframeft call returned an error status (or the library is missing)."""

    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status
        self.name = _STATUS.get(status, str(status))


def library_path() -> str:
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise FrameFTError(5, f"{_LIB_PATH} is not built (python -m paper_2608_26430_amd.build)")
    lib = ctypes.CDLL(_LIB_PATH)
    i64, i32, f32, vp = ctypes.c_int64, ctypes.c_int, ctypes.c_float, ctypes.c_void_p
    dp = ctypes.POINTER(ctypes.c_double)
    sig = {
        "ff_status_string": (ctypes.c_char_p, [i32]),
        "ff_last_error": (ctypes.c_char_p, []),
        "ff_abi_version": (i32, []),
        "ff_tff_host": (i32, [i64, i64, i64, i64, i64, dp]),
        "ff_framegen": (i32, [i64, i64, i64, ctypes.POINTER(vp)]),
        "ff_frame_export": (i32, [vp, i64, i64, dp]),
        "ff_frame_info": (i32, [vp, ctypes.POINTER(i64), ctypes.POINTER(i64), ctypes.POINTER(i64)]),
        "ff_frame_destroy": (None, [vp]),
        "ff_plan_create": (i32, [vp, vp, i64, vp, vp, i64, i64, ctypes.POINTER(vp)]),
        "ff_plan_destroy": (None, [vp]),
        "ff_plan_query": (i32, [vp, i32, ctypes.POINTER(i64)]),
        "ff_plan_order": (i32, [vp, ctypes.POINTER(i64)]),
        "ff_adapter_fwd": (i32, [vp, i64, i32, vp, i64, vp, f32, f32, vp, i64, vp]),
        "ff_adapter_bwd": (i32, [vp, i64, i32, vp, i64, vp, i64, vp, f32, f32, vp, i64, i32, vp, vp]),
        "ff_adapter_fwd_save": (i32, [vp, i64, i32, vp, i64, vp, f32, f32, vp, i64, vp, vp]),
        "ff_adapter_bwd_saved": (i32, [vp, i64, i32, vp, i64, vp, i64, vp, vp, f32, f32, vp, i64, i32, vp, vp]),
        "ff_merge_delta": (i32, [vp, vp, f32, i32, f32, vp, i64, vp]),
        "ff_adapter_fwd_batched": (i32, [vp, i64, i64, i32, vp, i64, vp, f32, f32, vp, i64, vp]),
        "ff_adapter_bwd_batched": (i32, [vp, i64, i64, i32, vp, i64, vp, i64, vp, f32, f32, vp, i64, i32,
                                         vp, vp]),
        "ff_time_next_kernel": (i32, [vp, vp]),
        "ff_adapter_bwd_noalloc": (i32, [vp, i64, i32, vp, i64, vp, i64, vp, f32, f32, vp, i64, i32, vp, vp]),
        "ff_plan_group_create": (i32, [i64, vp, ctypes.POINTER(vp)]),
        "ff_plan_group_destroy": (None, [vp]),
        "ff_adapter_fwd_group": (i32, [vp, i64, vp, i32, vp, i64, vp, f32, f32, vp, i64, vp]),
        "ff_adapter_bwd_group": (i32, [vp, i64, vp, i32, vp, i64, vp, i64, vp, f32, f32, vp, i64, i32, vp, vp]),
        "ff_adamw_step": (i32, [i64, vp, vp, vp, vp, f32, f32, f32, f32, f32, i64, vp]),
        "ff_adamw_step_batched": (i32, [i64, i64, vp, vp, vp, vp, f32, f32, f32, f32, f32, i64, vp]),
        "ff_lr_linear_warmup": (ctypes.c_double, [i64, i64, i64, ctypes.c_double]),
        "ff_coef_to_plan": (i32, [vp, vp, vp, vp]),
        "ff_coef_to_user": (i32, [vp, vp, vp, i32, vp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int):
    if status != 0:
        msg = _load().ff_last_error().decode()
        raise FrameFTError(status, msg)


# ------------------------------------------------------------------ frames

def tff_host(d: int, k: int, rho: int, col0: int = 0, ncols: Optional[int] = None) -> np.ndarray:
    """Columns col0.. of the real (k, rho, d) tight fusion frame from the library's host construction."""
    lib = _load()
    if ncols is None:
        ncols = k * rho - col0
    out = np.zeros((d, max(ncols, 0)), dtype=np.float64)
    _check(lib.ff_tff_host(d, k, rho, col0, ncols, out.ctypes.data_as(ctypes.POINTER(ctypes.c_double))))
    return out


class Frame:
    """A frame on the current device (ff_framegen)."""

    def __init__(self, handle: int, d: int, k: int, rho: int):
        self._h = ctypes.c_void_p(handle)
        self.d, self.k, self.rho = d, k, rho

    @property
    def handle(self):
        return self._h

    def export(self, col0: int = 0, ncols: Optional[int] = None) -> np.ndarray:
        """Columns of P as the kernels see them (fp32 block read back), fp64 d x ncols."""
        if ncols is None:
            ncols = self.k * self.rho - col0
        out = np.zeros((self.d, ncols), dtype=np.float64)
        _check(_load().ff_frame_export(self._h, col0, ncols,
                                       out.ctypes.data_as(ctypes.POINTER(ctypes.c_double))))
        return out

    def close(self):
        if self._h:
            _load().ff_frame_destroy(self._h)
            self._h = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def framegen(d: int, k: int, rho: int) -> Frame:
    """TFF(k, rho, d) on the current device (Algorithm 1, step 2)."""
    lib = _load()
    h = ctypes.c_void_p()
    _check(lib.ff_framegen(d, k, rho, ctypes.byref(h)))
    return Frame(h.value, d, k, rho)


# ------------------------------------------------------------------ plans

class Plan:
    """Support of C on a pair of frames, with device tables and workspace."""

    def __init__(self, f_in: Frame, f_out: Frame, rows, cols, max_tokens: int, max_batch: int = 1):
        lib = _load()
        rows = np.ascontiguousarray(rows, dtype=np.int32)
        cols = np.ascontiguousarray(cols, dtype=np.int32)
        if rows.shape != cols.shape or rows.ndim != 1:
            raise ValueError("rows and cols must be 1-D of equal length")
        h = ctypes.c_void_p()
        _check(lib.ff_plan_create(f_in.handle, f_out.handle, rows.size,
                                  rows.ctypes.data if rows.size else None,
                                  cols.ctypes.data if cols.size else None,
                                  max_tokens, max_batch, ctypes.byref(h)))
        self._h = h
        self.f_in, self.f_out = f_in, f_out
        self.n, self.m = f_in.d, f_out.d
        self.nnz = int(rows.size)
        self.max_tokens, self.max_batch = max_tokens, max_batch
        self._order = None

    @property
    def handle(self):
        return self._h

    def query(self, key: int) -> int:
        v = ctypes.c_int64()
        _check(_load().ff_plan_query(self._h, key, ctypes.byref(v)))
        return v.value

    def tile_tokens(self, dtype: str) -> int:
        return self.query(FF_BF16 if dtype == "bf16" else FF_F32)

    @property
    def workspace_bytes(self) -> int:
        return self.query(2)

    @property
    def fast128(self) -> bool:
        """True when bf16 calls run the fused kernels for 128-wide frame blocks."""
        return bool(self.query(4))

    @property
    def coef_slots(self) -> int:
        """Length L of every c / dC array of this plan (nnz plus padding slots)."""
        return self.query(5)

    @property
    def saved_floats(self) -> int:
        """Length of the c_saved arrays of adapter_fwd(save=...) / adapter_bwd(saved=...) (0: none needed)."""
        return self.query(6)

    @property
    def bwd_tile_tokens(self) -> int:
        """Tokens per workgroup tile of the fused 128-wide backward (16 or 8; 0 without it)."""
        return self.query(7)

    @property
    def radix(self):
        """(input, output) frame application: 4 for the factored radix-4 form, 1 for dense blocks."""
        return self.query(8), self.query(9)

    @property
    def gen_chunks(self) -> int:
        """Input-side chunks of a generic-kernel tile (1: the whole input side at once)."""
        return self.query(10)

    def gen_tile_tokens(self, dtype: str) -> int:
        """Most tokens per generic-kernel tile with those chunks."""
        return self.query(12 if dtype == "bf16" else 11)

    @property
    def gen_token_groups(self) -> bool:
        """True when bf16 generic-kernel tiles keep four tokens of a coefficient together."""
        return bool(self.query(13))

    def new_saved(self, device=None):
        """A c_saved array for one adapter of this plan (None when the plan needs none)."""
        torch = _torch()
        n = self.saved_floats
        return torch.empty((n,), dtype=torch.float32, device=device or "cuda") if n else None

    @property
    def order(self) -> np.ndarray:
        """User index of the support entry in each coefficient slot, -1 for padding:
        c_plan[j] = c_user[order[j]] where order[j] >= 0, dC_user[order[j]] = dC_plan[j]."""
        if self._order is None:
            o = np.empty(self.coef_slots, dtype=np.int64)
            _check(_load().ff_plan_order(self._h, o.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))))
            self._order = o
        return self._order

    def to_plan(self, c_user) -> np.ndarray:
        """Host user-order coefficients (nnz) -> plan layout (L, fp32, zero padding)."""
        c_user = np.asarray(c_user)
        o = self.order
        out = np.zeros(o.size, dtype=np.float32)
        keep = o >= 0
        out[keep] = c_user[o[keep]]
        return out

    def to_user(self, c_plan) -> np.ndarray:
        """Host plan-layout array (L) -> user order (nnz)."""
        c_plan = np.asarray(c_plan)
        o = self.order
        out = np.empty(self.nnz, dtype=c_plan.dtype)
        keep = o >= 0
        out[o[keep]] = c_plan[keep]
        return out

    def close(self):
        if self._h:
            _load().ff_plan_destroy(self._h)
            self._h = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def plan_create(f_in: Frame, f_out: Frame, rows, cols, max_tokens: int, max_batch: int = 1) -> Plan:
    return Plan(f_in, f_out, rows, cols, max_tokens, max_batch)


# ------------------------------------------------------------------ hot path

def _torch():
    import torch
    return torch


def _act_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return FF_BF16
    if t.dtype == torch.float32:
        return FF_F32
    raise TypeError(f"unsupported activation dtype {t.dtype}")


def _mat(t, name):
    if t.dim() != 2 or t.stride(1) != 1 or not t.is_cuda:
        raise ValueError(f"{name} must be a 2-D device tensor with unit column stride")
    return t.data_ptr(), t.stride(0)


def _vec(t, name, length=None):
    torch = _torch()
    if t.dtype != torch.float32 or not t.is_contiguous() or not t.is_cuda:
        raise ValueError(f"{name} must be a contiguous fp32 device tensor")
    if length is not None and t.numel() != length:
        raise ValueError(f"{name} must hold the plan's {length} coefficient slots (Plan.coef_slots)")
    return t.data_ptr()


def _stream(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def adapter_fwd(plan: Plan, X, c_vals, scale: float, Y=None, beta: float = 0.0, stream=None, save=None):
    """Y = beta*Y + scale * P_out C P_in^T x for each token row of X; returns Y.  With `save` (a
    c_saved array, Plan.new_saved) the forward also stores the coefficients in the backward's
    order, for adapter_bwd(saved=...) with the same c_vals (ff_adapter_fwd_save)."""
    torch = _torch()
    T = X.shape[0]
    if Y is None:
        if beta != 0.0:
            raise ValueError("beta != 0 needs an existing Y")
        Y = torch.empty((T, plan.m), dtype=X.dtype, device=X.device)
    xp, ldx = _mat(X, "X")
    yp, ldy = _mat(Y, "Y")
    if Y.dtype != X.dtype or Y.shape[0] != T:
        raise ValueError("Y must match X in dtype and token count")
    cp = _vec(c_vals, "c_vals", plan.coef_slots)
    if save is not None:
        _check(_load().ff_adapter_fwd_save(plan.handle, T, _act_code(X), xp, ldx, cp, scale, beta, yp, ldy,
                                           _vec(save, "save", plan.saved_floats), _stream(stream)))
    else:
        _check(_load().ff_adapter_fwd(plan.handle, T, _act_code(X), xp, ldx, cp, scale, beta, yp, ldy,
                                      _stream(stream)))
    return Y


def adapter_bwd(plan: Plan, X, G, c_vals, scale: float, dX=None, dC=None, beta_dx: float = 0.0,
                accumulate_dc: bool = False, want_dx: bool = True, want_dc: bool = True, stream=None,
                saved=None):
    """Backward of adapter_fwd for upstream gradient G: returns (dX, dC) (None where not wanted).
    `saved`: the c_saved array of adapter_fwd(save=...) with the same c_vals (ff_adapter_bwd_saved)."""
    torch = _torch()
    T = G.shape[0]
    act = _act_code(G)
    if want_dx and dX is None:
        if beta_dx != 0.0:
            raise ValueError("beta_dx != 0 needs an existing dX")
        dX = torch.empty((T, plan.n), dtype=G.dtype, device=G.device)
    if want_dc and dC is None:
        if accumulate_dc:
            raise ValueError("accumulate_dc needs an existing dC")
        dC = torch.empty((plan.coef_slots,), dtype=torch.float32, device=G.device)
    gp, ldg = _mat(G, "G")
    xp, ldx = _mat(X, "X") if X is not None else (None, plan.n)
    dxp, lddx = _mat(dX, "dX") if want_dx else (None, plan.n)
    dcp = _vec(dC, "dC", plan.coef_slots) if want_dc else None
    cp = _vec(c_vals, "c_vals", plan.coef_slots) if c_vals is not None else None
    if saved is not None:
        _check(_load().ff_adapter_bwd_saved(plan.handle, T, act, xp, ldx, gp, ldg, cp,
                                            _vec(saved, "saved", plan.saved_floats), scale, beta_dx,
                                            dxp, lddx, int(accumulate_dc), dcp, _stream(stream)))
    else:
        _check(_load().ff_adapter_bwd(plan.handle, T, act, xp, ldx, gp, ldg, cp, scale, beta_dx,
                                      dxp, lddx, int(accumulate_dc), dcp, _stream(stream)))
    return (dX if want_dx else None), (dC if want_dc else None)


def adapter_bwd_noalloc(plan: Plan, X, G, c_vals, scale: float, dX, dC, beta_dx: float = 0.0,
                        accumulate_dc: bool = False, stream=None):
    """adapter_bwd through ff_adapter_bwd_noalloc: the library allocates nothing and uses its static
    scratch.  The outputs dX and dC (either may be None to skip it) are the caller's."""
    T = G.shape[0]
    gp, ldg = _mat(G, "G")
    xp, ldx = _mat(X, "X") if X is not None else (None, plan.n)
    dxp, lddx = _mat(dX, "dX") if dX is not None else (None, plan.n)
    dcp = _vec(dC, "dC", plan.coef_slots) if dC is not None else None
    cp = _vec(c_vals, "c_vals", plan.coef_slots) if c_vals is not None else None
    _check(_load().ff_adapter_bwd_noalloc(plan.handle, T, _act_code(G), xp, ldx, gp, ldg, cp, scale, beta_dx,
                                          dxp, lddx, int(accumulate_dc), dcp, _stream(stream)))
    return dX, dC


def _fvec(t, name, n=None):
    torch = _torch()
    if t.dtype != torch.float32 or not t.is_contiguous() or not t.is_cuda or (n is not None and t.numel() != n):
        raise ValueError(f"{name} must be a contiguous fp32 device tensor of {n} elements")
    return t.data_ptr()


def adamw_step(c, g, m, v, lr: float, step: int, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
               weight_decay: float = 0.0, stream=None):
    """One AdamW step on device fp32 vectors c, m, v (in place) with gradient g (ff_adamw_step)."""
    n = c.numel()
    _check(_load().ff_adamw_step(n, _fvec(c, "c", n), _fvec(g, "g", n), _fvec(m, "m", n), _fvec(v, "v", n),
                                 lr, beta1, beta2, eps, weight_decay, step, _stream(stream)))
    return c


def adamw_step_batched(cs: Sequence, gs: Sequence, ms: Sequence, vs: Sequence, lr: float, step: int,
                       beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8, weight_decay: float = 0.0,
                       stream=None):
    """adamw_step over equally long vectors of many adapters in one launch (ff_adamw_step_batched)."""
    n, dev = cs[0].numel(), cs[0].device
    for group, name in ((cs, "c"), (gs, "g"), (ms, "m"), (vs, "v")):
        for t in group:
            _fvec(t, name, n)
            if t.data_ptr() % 16:
                raise ValueError(f"{name} arrays must be 16-byte aligned")
    ptrs = [pointer_array(x, dev) for x in (cs, gs, ms, vs)]
    _check(_load().ff_adamw_step_batched(len(cs), n, *[p.data_ptr() for p in ptrs], lr, beta1, beta2, eps,
                                         weight_decay, step, _stream(stream)))
    return cs


def lr_linear_warmup(step: int, warmup: int, total: int, base_lr: float) -> float:
    """Learning rate of optimizer step `step` (0-based) under the linear schedule with warmup."""
    return float(_load().ff_lr_linear_warmup(step, warmup, total, base_lr))


def coef_to_plan(plan: Plan, c_user, c_plan=None, stream=None):
    """Device user-order coefficients (nnz fp32) -> plan layout (Plan.coef_slots, zero padding),
    on the device (ff_coef_to_plan); returns c_plan."""
    torch = _torch()
    if c_plan is None:
        c_plan = torch.empty((plan.coef_slots,), dtype=torch.float32, device=c_user.device)
    _check(_load().ff_coef_to_plan(plan.handle, _vec(c_user, "c_user", plan.nnz),
                                   _vec(c_plan, "c_plan", plan.coef_slots), _stream(stream)))
    return c_plan


def coef_to_user(plan: Plan, c_plan, c_user=None, accumulate: bool = False, stream=None):
    """Device plan-layout array (Plan.coef_slots) -> user order (nnz), added to c_user when
    accumulate (ff_coef_to_user); returns c_user."""
    torch = _torch()
    if c_user is None:
        if accumulate:
            raise ValueError("accumulate needs an existing c_user")
        c_user = torch.empty((plan.nnz,), dtype=torch.float32, device=c_plan.device)
    _check(_load().ff_coef_to_user(plan.handle, _vec(c_plan, "c_plan", plan.coef_slots),
                                   _vec(c_user, "c_user", plan.nnz), int(accumulate), _stream(stream)))
    return c_user


def merge_delta(plan: Plan, c_vals, scale: float, W, beta: float = 1.0, stream=None):
    """W = beta*W + scale * P_out C P_in^T in place; returns W."""
    torch = _torch()
    wp, ldw = _mat(W, "W")
    if W.dtype not in (torch.float32, torch.bfloat16) or tuple(W.shape) != (plan.m, plan.n):
        raise ValueError("W must be m x n fp32 or bf16")
    code = FF_BF16 if W.dtype == torch.bfloat16 else FF_F32
    _check(_load().ff_merge_delta(plan.handle, _vec(c_vals, "c_vals", plan.coef_slots), scale, code, beta, wp, ldw,
                                  _stream(stream)))
    return W


def pointer_array(tensors: Sequence, device):
    """Device array of data pointers (int64) for the batched calls."""
    torch = _torch()
    return torch.tensor([t.data_ptr() for t in tensors], dtype=torch.int64, device=device)


def adapter_fwd_batched(plan: Plan, Xs: Sequence, cs: Sequence, scale: float, Ys: Sequence,
                        beta: float = 0.0, stream=None, ptrs=None):
    """adapter_fwd for len(Xs) adapters sharing the plan (one launch).  `ptrs` may hold
    precomputed pointer arrays (X, c, Y) from pointer_array()."""
    count, T = len(Xs), Xs[0].shape[0]
    _, ldx = _mat(Xs[0], "X")
    _, ldy = _mat(Ys[0], "Y")
    dev = Xs[0].device
    px, pc, py = ptrs if ptrs is not None else (pointer_array(Xs, dev), pointer_array(cs, dev),
                                                 pointer_array(Ys, dev))
    _check(_load().ff_adapter_fwd_batched(plan.handle, count, T, _act_code(Xs[0]), px.data_ptr(), ldx,
                                          pc.data_ptr(), scale, beta, py.data_ptr(), ldy, _stream(stream)))
    return Ys


def adapter_bwd_batched(plan: Plan, Xs: Sequence, Gs: Sequence, cs: Sequence, scale: float,
                        dXs: Optional[Sequence], dCs: Optional[Sequence], beta_dx: float = 0.0,
                        accumulate_dc: bool = False, stream=None, ptrs=None):
    """adapter_bwd for len(Gs) adapters sharing the plan (one fused launch + one reduction)."""
    count, T = len(Gs), Gs[0].shape[0]
    dev = Gs[0].device
    _, ldg = _mat(Gs[0], "G")
    _, ldx = _mat(Xs[0], "X")
    lddx = _mat(dXs[0], "dX")[1] if dXs is not None else plan.n
    if ptrs is not None:
        px, pg, pc, pdx, pdc = ptrs
    else:
        px, pg = pointer_array(Xs, dev), pointer_array(Gs, dev)
        pc = pointer_array(cs, dev) if cs is not None else None     # not needed without dX
        pdx = pointer_array(dXs, dev) if dXs is not None else None
        pdc = pointer_array(dCs, dev) if dCs is not None else None
    _check(_load().ff_adapter_bwd_batched(plan.handle, count, T, _act_code(Gs[0]), px.data_ptr(), ldx,
                                          pg.data_ptr(), ldg, pc.data_ptr() if pc is not None else None,
                                          scale, beta_dx,
                                          pdx.data_ptr() if pdx is not None else None, lddx,
                                          int(accumulate_dc), pdc.data_ptr() if pdc is not None else None,
                                          _stream(stream)))
    return dXs, dCs


class PlanGroup:
    """Adapters over one frame pair with a support each (ff_plan_group_create): plans[i] serves
    adapter i.  Keeps the plans alive."""

    def __init__(self, plans: Sequence[Plan]):
        h = ctypes.c_void_p()
        arr = (ctypes.c_void_p * len(plans))(*[p.handle.value for p in plans])
        _check(_load().ff_plan_group_create(len(plans), ctypes.cast(arr, ctypes.c_void_p), ctypes.byref(h)))
        self._h = h
        self.plans = list(plans)
        self.count = len(plans)
        self.n, self.m = plans[0].n, plans[0].m

    @property
    def handle(self):
        return self._h

    def close(self):
        if self._h:
            _load().ff_plan_group_destroy(self._h)
            self._h = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def plan_group(plans: Sequence[Plan]) -> PlanGroup:
    return PlanGroup(plans)


def adapter_fwd_group(group: PlanGroup, Xs: Sequence, cs: Sequence, scale: float, Ys: Sequence, beta: float = 0.0,
                      tokens=None, T: Optional[int] = None, stream=None, ptrs=None):
    """Forward of adapter i on plans[i] (one launch).  `tokens`: optional device int32 tensor of
    per-adapter token counts (each clamped to T, the launch size, default Xs[0].shape[0]).  `ptrs`
    may hold precomputed pointer arrays (X, c, Y) from pointer_array()."""
    T = Xs[0].shape[0] if T is None else T
    _, ldx = _mat(Xs[0], "X")
    _, ldy = _mat(Ys[0], "Y")
    dev = Xs[0].device
    px, pc, py = ptrs if ptrs is not None else (pointer_array(Xs, dev), pointer_array(cs, dev),
                                                 pointer_array(Ys, dev))
    tp = _tokens_ptr(tokens, group.count)
    _check(_load().ff_adapter_fwd_group(group.handle, T, tp, _act_code(Xs[0]), px.data_ptr(), ldx, pc.data_ptr(),
                                        scale, beta, py.data_ptr(), ldy, _stream(stream)))
    return Ys


def adapter_bwd_group(group: PlanGroup, Xs: Sequence, Gs: Sequence, cs: Optional[Sequence], scale: float,
                      dXs: Optional[Sequence], dCs: Optional[Sequence], beta_dx: float = 0.0,
                      accumulate_dc: bool = False, tokens=None, T: Optional[int] = None, stream=None, ptrs=None):
    """Backward of adapter i on plans[i] (dX and/or dC; one launch plus the dC reduction).  `ptrs`
    may hold precomputed pointer arrays (X, G, c, dX, dC)."""
    T = Gs[0].shape[0] if T is None else T
    dev = Gs[0].device
    _, ldg = _mat(Gs[0], "G")
    _, ldx = _mat(Xs[0], "X")
    lddx = _mat(dXs[0], "dX")[1] if dXs is not None else group.n
    if ptrs is not None:
        px, pg, pc, pdx, pdc = ptrs
    else:
        px, pg = pointer_array(Xs, dev), pointer_array(Gs, dev)
        pc = pointer_array(cs, dev) if cs is not None else None
        pdx = pointer_array(dXs, dev) if dXs is not None else None
        pdc = pointer_array(dCs, dev) if dCs is not None else None
    tp = _tokens_ptr(tokens, group.count)
    _check(_load().ff_adapter_bwd_group(group.handle, T, tp, _act_code(Gs[0]), px.data_ptr(), ldx, pg.data_ptr(),
                                        ldg, pc.data_ptr() if pc is not None else None, scale, beta_dx,
                                        pdx.data_ptr() if pdx is not None else None, lddx, int(accumulate_dc),
                                        pdc.data_ptr() if pdc is not None else None, _stream(stream)))
    return dXs, dCs


def _tokens_ptr(tokens, count):
    if tokens is None:
        return None
    torch = _torch()
    if tokens.dtype != torch.int32 or not tokens.is_cuda or not tokens.is_contiguous() or tokens.numel() != count:
        raise ValueError("tokens must be a contiguous int32 device tensor with one count per adapter")
    return tokens.data_ptr()


def time_next_kernel(ev_start, ev_stop):
    """Arm the next hot-path call to record torch.cuda.Events around its main kernel."""
    for ev in (ev_start, ev_stop):
        if ev is not None and not ev.cuda_event:
            ev.record()          # torch creates the underlying hipEvent_t on first use
    _check(_load().ff_time_next_kernel(ctypes.c_void_p(ev_start.cuda_event if ev_start else None),
                                       ctypes.c_void_p(ev_stop.cuda_event if ev_stop else None)))
