"""Exact top-k gradient sparsification with error feedback and the sparse
aggregate + multi-tensor SGD update on AMD MI355X (gfx950).

Thin ctypes binding over ``lib/libtkef.so`` (C ABI in ``include/tkef.h``).
This module only marshals arguments: every step of the computation runs in
the library's HIP kernels. PyTorch supplies device memory and streams.

    plan = SparsifyPlan(numels, mode=GLOBAL, rho=0.001)
    plan.bind(grads, residuals)            # once per set of buffers
    idx, val = plan.execute()              # every step

    up = UpdatePlan(numels, P=128, stride=k)
    up.bind(params, momentum)              # once
    up.execute(idx_all, val_all, lr=0.1, mu=0.9, wd=5e-5)
"""
from __future__ import annotations

# torch first: it loads the HIP runtime that this library must share
import torch  # noqa: E402

import ctypes
import os
from typing import Optional, Sequence, Tuple

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "lib", "libtkef.so")

GLOBAL = 0
PER_TENSOR = 1
APPROX = 2          # MSTopK (Alg. 1) over the concatenated list
STATUS_NAN = 1
STATUS_UNSORTED = 2
STATUS_INDEX_RANGE = 4
STATUS_TIMEOUT = 8
STATUS_NONFINITE = 16
VAL_F32 = 0
VAL_F16 = 1

OK, EINVAL, ERANGE, EWORKSPACE, EHIP, ESTATE, ENOMEM = 0, -1, -2, -3, -4, -5, -6


class TkefError(RuntimeError):
    def __init__(self, fn: str, code: int, msg: str):
        super().__init__(f"{fn}: {msg} ({code})")
        self.code = code


class TkefStatusError(RuntimeError):
    """A call finished with bits set in its device status word."""

    NAMES = {STATUS_NAN: "NaN in g + r (selection unspecified)",
             STATUS_UNSORTED: "an index list is not ascending",
             STATUS_INDEX_RANGE: "an index lies outside [0, d)",
             STATUS_TIMEOUT: "a wait between workgroups gave up (results invalid)",
             STATUS_NONFINITE: "MSTopK saw a non-finite value (it took the first k positions)"}

    def __init__(self, fn: str, bits: int):
        what = "; ".join(m for b, m in self.NAMES.items() if bits & b) or "unknown bits"
        super().__init__(f"{fn}: device status {bits:#x}: {what}")
        self.bits = bits


_lib: Optional[ctypes.CDLL] = None


def _declare(lib: ctypes.CDLL) -> ctypes.CDLL:
    vp, i32, i64, f32, f64, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                  ctypes.c_float, ctypes.c_double, ctypes.c_size_t)
    P = ctypes.POINTER
    sig = {
        "tkef_version": ([], ctypes.c_int),
        "tkef_strerror": ([ctypes.c_int], ctypes.c_char_p),
        "tkef_k_from_rho": ([i64, f64], i64),
        "tkef_sparsify_plan_create": ([P(i64), i32, i32, f64, i64, P(vp)], ctypes.c_int),
        "tkef_sparsify_plan_destroy": ([vp], ctypes.c_int),
        "tkef_sparsify_plan_info": ([vp, P(sz), P(i64), P(i64), P(i32), P(i32)], ctypes.c_int),
        "tkef_sparsify_plan_group_k": ([vp, P(i64), i32], ctypes.c_int),
        "tkef_sparsify_plan_bind": ([vp, P(vp), P(vp), vp, sz, vp], ctypes.c_int),
        "tkef_sparsify_execute": ([vp, vp, sz, vp, vp, vp, vp], ctypes.c_int),
        "tkef_sparsify_plan_set_events": ([vp, P(vp), i32], ctypes.c_int),
        "tkef_sparsify_plan_launch_name": ([vp, i32], ctypes.c_char_p),
        "tkef_sparsify_plan_set_value_format": ([vp, i32], ctypes.c_int),
        "tkef_sparsify_plan_set_approx": ([vp, i32, ctypes.c_uint64], ctypes.c_int),
        "tkef_sparsify_approx_result": ([vp, vp, P(f64), P(i64), vp], ctypes.c_int),
        "tkef_sparsify_workspace": ([P(i64), i32, i32, f64, i64, P(sz), P(i64)], ctypes.c_int),
        "tkef_sparsify": ([P(vp), P(vp), P(i64), i32, i32, f64, i64, i32, vp, vp, P(i64), vp,
                           sz, vp, vp], ctypes.c_int),
        "tkef_sparsify1": ([vp, vp, i64, i64, vp, vp, vp, sz, vp, vp], ctypes.c_int),
        "tkef_sparsify1_static": ([vp, vp, i64, i64, vp, vp, vp, vp], ctypes.c_int),
        "tkef_aggregate_workspace": ([P(i64), i32, i32, P(sz)], ctypes.c_int),
        "tkef_aggregate_update": ([P(vp), P(vp), P(i64), i32, P(vp), P(vp), P(i64), i32, f32,
                                   f32, f32, vp, sz, vp, vp], ctypes.c_int),
        "tkef_update_plan_create": ([P(i64), i32, i32, i64, P(vp)], ctypes.c_int),
        "tkef_update_plan_destroy": ([vp], ctypes.c_int),
        "tkef_update_plan_info": ([vp, P(sz), P(i64), P(i32)], ctypes.c_int),
        "tkef_update_plan_bind": ([vp, P(vp), P(vp), vp, sz, vp], ctypes.c_int),
        "tkef_update_execute": ([vp, vp, vp, vp, f32, f32, f32, vp, sz, vp, vp], ctypes.c_int),
        "tkef_update_plan_set_events": ([vp, P(vp), i32], ctypes.c_int),
        "tkef_update_plan_launch_name": ([vp, i32], ctypes.c_char_p),
        "tkef_update_plan_set_value_format": ([vp, i32], ctypes.c_int),
        "tkef_update_plan_set_deterministic": ([vp, i32], ctypes.c_int),
        "tkef_aggregate_execute": ([vp, vp, vp, vp, vp, sz, vp, vp], ctypes.c_int),
        "tkef_sparse_aggregate": ([P(vp), P(i64), i32, vp, vp, i32, i32, i64, vp, vp, sz, vp,
                                   vp], ctypes.c_int),
        "tkef_update_workspace": ([P(i64), i32, i32, i64, P(sz)], ctypes.c_int),
        "tkef_lars_update_execute": ([vp, vp, vp, vp, f64, f64, f64, f32, vp, vp, sz, vp, vp],
                                     ctypes.c_int),
        "tkef_update_plan_bind_grads": ([vp, P(vp), vp, sz, vp], ctypes.c_int),
        "tkef_lars_rates_execute": ([vp, f64, f64, f64, vp, vp, sz, vp], ctypes.c_int),
        "tkef_lars_launch_name": ([i32, i32], ctypes.c_char_p),
        "tkef_sparse_aggregate_update": ([P(vp), P(vp), P(i64), i32, vp, vp, i32, i64, vp, f32,
                                          f32, f32, vp, sz, vp, vp], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


def lib() -> ctypes.CDLL:
    """The loaded HIP library. Raises if it has not been built: there is no
    fallback implementation."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        _lib = _declare(ctypes.CDLL(LIB_PATH))
    return _lib


def _check(fn: str, rc: int) -> None:
    if rc != OK:
        raise TkefError(fn, rc, lib().tkef_strerror(rc).decode())


def _new_status(dev) -> torch.Tensor:
    return torch.zeros(1, dtype=torch.int32, device=dev)


def _raise_on_status(fn: str, status: torch.Tensor, stream=None) -> None:
    """Synchronizes the stream and raises TkefStatusError if any status bit is
    set."""
    (stream or torch.cuda.current_stream()).synchronize()
    bits = int(status.item()) & 0xFFFFFFFF
    if bits:
        raise TkefStatusError(fn, bits)


def strerror(code: int) -> str:
    return lib().tkef_strerror(code).decode()


def k_from_rho(d: int, rho: float) -> int:
    return int(lib().tkef_k_from_rho(d, rho))


def _i64_array(vals: Sequence[int]):
    return (ctypes.c_int64 * max(1, len(vals)))(*[int(v) for v in vals])


def _ptr_array(ts: Sequence[Optional[torch.Tensor]]):
    return (ctypes.c_void_p * max(1, len(ts)))(*[(t.data_ptr() if t is not None else None)
                                                 for t in ts])


def _stream_handle(stream: Optional[torch.cuda.Stream]) -> Optional[int]:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream or None


def _check_f32_tensors(ts: Sequence[torch.Tensor], what: str) -> None:
    for t in ts:
        if t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{what}: expected contiguous float32 CUDA tensors")


def _val_format(dtype) -> int:
    if dtype == torch.float32:
        return VAL_F32
    if dtype == torch.float16:
        return VAL_F16
    raise ValueError("values are float32 or float16")


def _events(events: Optional[Sequence[torch.cuda.Event]]):
    """Raw event handles of torch events (each recorded once so it exists)."""
    if not events:
        return None, 0
    for e in events:
        if e.cuda_event == 0:
            e.record()
    arr = (ctypes.c_void_p * len(events))(*[e.cuda_event for e in events])
    return arr, len(events)


# ----------------------------------------------------------------------------
class SparsifyPlan:
    """Plan for sparsifying a fixed list of tensor sizes (see tkef.h)."""

    def __init__(self, numels: Sequence[int], mode: int = GLOBAL, rho: Optional[float] = None,
                 k: Optional[int] = None, val_dtype=torch.float32, n_search: int = 30,
                 check: bool = False):
        """check=True: every execute without a caller status word uses its
        own, synchronizes and raises TkefStatusError on any status bit."""
        self.check = bool(check)
        self._numels = [int(n) for n in numels]
        self._h = ctypes.c_void_p()
        L = lib()
        _check("tkef_sparsify_plan_create", L.tkef_sparsify_plan_create(
            _i64_array(self._numels), len(self._numels), int(mode),
            float(rho) if rho is not None else 0.0, int(k) if k else 0, ctypes.byref(self._h)))
        self.val_dtype = val_dtype
        _check("tkef_sparsify_plan_set_value_format",
               L.tkef_sparsify_plan_set_value_format(self._h, _val_format(val_dtype)))
        self.mode, self.n_search = int(mode), int(n_search)
        if self.mode == APPROX:
            _check("tkef_sparsify_plan_set_approx",
                   L.tkef_sparsify_plan_set_approx(self._h, self.n_search, 0))
        ws, kt, d, ng, nl = (ctypes.c_size_t(), ctypes.c_int64(), ctypes.c_int64(),
                             ctypes.c_int32(), ctypes.c_int32())
        _check("tkef_sparsify_plan_info", L.tkef_sparsify_plan_info(
            self._h, ctypes.byref(ws), ctypes.byref(kt), ctypes.byref(d), ctypes.byref(ng),
            ctypes.byref(nl)))
        self.ws_bytes, self.k_total, self.d = ws.value, kt.value, d.value
        self.ngroups, self.nlaunch = ng.value, nl.value
        self.ws: Optional[torch.Tensor] = None
        self._bound = None
        self._events = None

    def __del__(self):
        if getattr(self, "_h", None) and self._h.value and _lib is not None:
            _lib.tkef_sparsify_plan_destroy(self._h)
            self._h = ctypes.c_void_p()

    def group_k(self):
        arr = (ctypes.c_int64 * self.ngroups)()
        _check("tkef_sparsify_plan_group_k", lib().tkef_sparsify_plan_group_k(
            self._h, arr, self.ngroups))
        return list(arr)

    def launch_names(self):
        return [lib().tkef_sparsify_plan_launch_name(self._h, i).decode()
                for i in range(self.nlaunch)]

    def bind(self, grads: Sequence[torch.Tensor], residuals: Sequence[torch.Tensor],
             ws: Optional[torch.Tensor] = None, stream=None) -> "SparsifyPlan":
        if len(grads) != len(self._numels) or len(residuals) != len(self._numels):
            raise ValueError("tensor count does not match the plan")
        _check_f32_tensors(list(grads) + list(residuals), "bind")
        for g, r, n in zip(grads, residuals, self._numels):
            if g.numel() != n or r.numel() != n:
                raise ValueError("tensor size does not match the plan")
        dev = grads[0].device
        if ws is None:
            ws = torch.empty(max(self.ws_bytes, 256), dtype=torch.uint8, device=dev)
        self.ws = ws
        _check("tkef_sparsify_plan_bind", lib().tkef_sparsify_plan_bind(
            self._h, _ptr_array(grads), _ptr_array(residuals), ws.data_ptr(), ws.numel(),
            _stream_handle(stream)))
        self._bound = (list(grads), list(residuals))
        return self

    def set_events(self, events: Optional[Sequence[torch.cuda.Event]]) -> None:
        arr, n = _events(events)
        self._events = (arr, list(events) if events else None)
        _check("tkef_sparsify_plan_set_events",
               lib().tkef_sparsify_plan_set_events(self._h, arr, n))

    def execute(self, idx_out: Optional[torch.Tensor] = None,
                val_out: Optional[torch.Tensor] = None,
                status: Optional[torch.Tensor] = None, stream=None,
                window_word: Optional[int] = None) -> Tuple[torch.Tensor, torch.Tensor]:
        """window_word (APPROX plans): the 64-bit value the band offset of
        this and later executions is drawn from."""
        if self._bound is None or self.ws is None:
            raise RuntimeError("plan is not bound")
        if window_word is not None:
            if self.mode != APPROX:
                raise ValueError("window_word applies to APPROX plans only")
            _check("tkef_sparsify_plan_set_approx", lib().tkef_sparsify_plan_set_approx(
                self._h, self.n_search, int(window_word) & ((1 << 64) - 1)))
        dev = self.ws.device
        if idx_out is None:
            idx_out = torch.empty(max(self.k_total, 1), dtype=torch.int32, device=dev)
        if val_out is None:
            val_out = torch.empty(max(self.k_total, 1), dtype=self.val_dtype, device=dev)
        if idx_out.numel() < self.k_total or val_out.numel() < self.k_total:
            raise ValueError("output buffers too small")
        if idx_out.dtype != torch.int32 or val_out.dtype != self.val_dtype:
            raise ValueError("idx_out must be int32 and val_out of the plan's value dtype")
        own = self.check and status is None
        if own:
            status = _new_status(dev)
        _check("tkef_sparsify_execute", lib().tkef_sparsify_execute(
            self._h, self.ws.data_ptr(), self.ws.numel(), idx_out.data_ptr(),
            val_out.data_ptr(), status.data_ptr() if status is not None else None,
            _stream_handle(stream)))
        if own:
            _raise_on_status("tkef_sparsify_execute", status, stream)
        return idx_out[: self.k_total], val_out[: self.k_total]


    def approx_result(self, stream=None) -> dict:
        """Search result of the last APPROX execution (synchronizes the
        stream): mean, u, k1, k2, offset, take, key1, key2."""
        out = (ctypes.c_double * 2)()
        cnt = (ctypes.c_int64 * 6)()
        _check("tkef_sparsify_approx_result", lib().tkef_sparsify_approx_result(
            self._h, self.ws.data_ptr() if self.ws is not None else None, out, cnt,
            _stream_handle(stream)))
        return {"mean": out[0], "u": out[1], "k1": cnt[0], "k2": cnt[1], "offset": cnt[2],
                "take": cnt[3], "key1": cnt[4], "key2": cnt[5]}


LARS_LAUNCHES = ["seg", "lars_norm", "lars_rates", "lars_step"]
LARS_DENSE_LAUNCHES = ["lars_norm_dense", "lars_rates"]


class UpdatePlan:
    """Plan for the sparse aggregate + SGD update of a fixed parameter list."""

    def __init__(self, numels: Sequence[int], P: int, stride: int, val_dtype=torch.float32,
                 check: bool = False, deterministic: bool = False):
        """check=True: every execute / aggregate / lars_execute without a
        caller status word uses its own, synchronizes and raises
        TkefStatusError on any status bit. deterministic=True: each
        position's entries are summed in worker order, then list order
        (bitwise reproducible; tkef_update_plan_set_deterministic)."""
        self.check = bool(check)
        self._numels = [int(n) for n in numels]
        self.P, self.stride = int(P), int(stride)
        self._h = ctypes.c_void_p()
        L = lib()
        _check("tkef_update_plan_create", L.tkef_update_plan_create(
            _i64_array(self._numels), len(self._numels), self.P, self.stride,
            ctypes.byref(self._h)))
        self.val_dtype = val_dtype
        _check("tkef_update_plan_set_value_format",
               L.tkef_update_plan_set_value_format(self._h, _val_format(val_dtype)))
        self.deterministic = bool(deterministic)
        _check("tkef_update_plan_set_deterministic",
               L.tkef_update_plan_set_deterministic(self._h, int(self.deterministic)))
        ws, d, nl = ctypes.c_size_t(), ctypes.c_int64(), ctypes.c_int32()
        _check("tkef_update_plan_info", L.tkef_update_plan_info(
            self._h, ctypes.byref(ws), ctypes.byref(d), ctypes.byref(nl)))
        self.ws_bytes, self.d, self.nlaunch = ws.value, d.value, nl.value
        self.ws: Optional[torch.Tensor] = None
        self._bound = None
        self._events = None

    def __del__(self):
        if getattr(self, "_h", None) and self._h.value and _lib is not None:
            _lib.tkef_update_plan_destroy(self._h)
            self._h = ctypes.c_void_p()

    def launch_names(self):
        return [lib().tkef_update_plan_launch_name(self._h, i).decode()
                for i in range(self.nlaunch)]

    def bind(self, params: Sequence[torch.Tensor],
             momentum: Optional[Sequence[torch.Tensor]] = None,
             ws: Optional[torch.Tensor] = None, stream=None) -> "UpdatePlan":
        if len(params) != len(self._numels):
            raise ValueError("tensor count does not match the plan")
        _check_f32_tensors(list(params) + list(momentum or []), "bind")
        for i, (w, n) in enumerate(zip(params, self._numels)):
            if w.numel() != n or (momentum is not None and momentum[i].numel() != n):
                raise ValueError("tensor size does not match the plan")
        if ws is None:
            ws = torch.empty(max(self.ws_bytes, 256), dtype=torch.uint8, device=params[0].device)
        self.ws = ws
        mom = _ptr_array(momentum) if momentum is not None else None
        _check("tkef_update_plan_bind", lib().tkef_update_plan_bind(
            self._h, _ptr_array(params), mom, ws.data_ptr(), ws.numel(),
            _stream_handle(stream)))
        self._bound = (list(params), list(momentum) if momentum is not None else None)
        return self

    def set_events(self, events: Optional[Sequence[torch.cuda.Event]]) -> None:
        arr, n = _events(events)
        self._events = (arr, list(events) if events else None)
        _check("tkef_update_plan_set_events", lib().tkef_update_plan_set_events(self._h, arr, n))

    def _check_lists(self, idx, val, nnz):
        if self._bound is None or self.ws is None:
            raise RuntimeError("plan is not bound")
        if idx.dtype != torch.int32 or val.dtype != self.val_dtype:
            raise ValueError("idx must be int32 and val of the plan's value dtype")
        if not (idx.is_cuda and val.is_cuda and idx.is_contiguous() and val.is_contiguous()):
            raise ValueError("idx and val must be contiguous CUDA tensors")
        if idx.numel() < self.P * self.stride or val.numel() < self.P * self.stride:
            raise ValueError("idx / val hold fewer than P * stride entries")
        if nnz is not None and (nnz.dtype != torch.int32 or nnz.numel() < self.P or not nnz.is_cuda):
            raise ValueError("nnz must be a CUDA int32 tensor of P counts")

    def _status(self, status):
        own = self.check and status is None
        return (_new_status(self.ws.device) if own else status), own

    def execute(self, idx: torch.Tensor, val: torch.Tensor, lr: float, mu: float = 0.0,
                wd: float = 0.0, nnz: Optional[torch.Tensor] = None,
                status: Optional[torch.Tensor] = None, stream=None) -> None:
        self._check_lists(idx, val, nnz)
        status, own = self._status(status)
        _check("tkef_update_execute", lib().tkef_update_execute(
            self._h, idx.data_ptr(), val.data_ptr(),
            nnz.data_ptr() if nnz is not None else None, float(lr), float(mu), float(wd),
            self.ws.data_ptr(), self.ws.numel(),
            status.data_ptr() if status is not None else None, _stream_handle(stream)))
        if own:
            _raise_on_status("tkef_update_execute", status, stream)

    def lars_execute(self, idx: torch.Tensor, val: torch.Tensor, gamma: float, eta: float,
                     eps: float, mu: float = 0.0, nnz: Optional[torch.Tensor] = None,
                     status: Optional[torch.Tensor] = None,
                     rates: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
        """Sum the lists and apply the LARS step (Eq. lars rates) to the bound
        tensors. Returns the per-tensor rates (float64)."""
        self._check_lists(idx, val, nnz)
        if rates is None:
            rates = torch.empty(len(self._numels), dtype=torch.float64, device=self.ws.device)
        status, own = self._status(status)
        _check("tkef_lars_update_execute", lib().tkef_lars_update_execute(
            self._h, idx.data_ptr(), val.data_ptr(),
            nnz.data_ptr() if nnz is not None else None, float(gamma), float(eta), float(eps),
            float(mu), rates.data_ptr(), self.ws.data_ptr(), self.ws.numel(),
            status.data_ptr() if status is not None else None, _stream_handle(stream)))
        if own:
            _raise_on_status("tkef_lars_update_execute", status, stream)
        return rates

    def bind_grads(self, grads: Sequence[torch.Tensor], stream=None) -> "UpdatePlan":
        """Dense gradients (same sizes as the bound parameters) for lars_rates."""
        if self._bound is None or self.ws is None:
            raise RuntimeError("plan is not bound")
        if len(grads) != len(self._numels):
            raise ValueError("tensor count does not match the plan")
        _check_f32_tensors(list(grads), "bind_grads")
        for g, n in zip(grads, self._numels):
            if g.numel() != n:
                raise ValueError("tensor size does not match the plan")
        _check("tkef_update_plan_bind_grads", lib().tkef_update_plan_bind_grads(
            self._h, _ptr_array(grads), self.ws.data_ptr(), self.ws.numel(),
            _stream_handle(stream)))
        self._grads = list(grads)
        return self

    def lars_rates(self, gamma: float, eta: float, eps: float,
                   rates: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
        """Layer-wise rates of Eq. (lars) from the bound parameters and the
        dense gradients of bind_grads (float64, one per tensor)."""
        if rates is None:
            rates = torch.empty(len(self._numels), dtype=torch.float64, device=self.ws.device)
        _check("tkef_lars_rates_execute", lib().tkef_lars_rates_execute(
            self._h, float(gamma), float(eta), float(eps), rates.data_ptr(), self.ws.data_ptr(),
            self.ws.numel(), _stream_handle(stream)))
        return rates

    def aggregate(self, idx: torch.Tensor, val: torch.Tensor, nnz: Optional[torch.Tensor] = None,
                  status: Optional[torch.Tensor] = None, stream=None) -> None:
        """Writes the sum of the P lists into the bound tensors (every
        position; zero where no list names it)."""
        self._check_lists(idx, val, nnz)
        status, own = self._status(status)
        _check("tkef_aggregate_execute", lib().tkef_aggregate_execute(
            self._h, idx.data_ptr(), val.data_ptr(),
            nnz.data_ptr() if nnz is not None else None, self.ws.data_ptr(), self.ws.numel(),
            status.data_ptr() if status is not None else None, _stream_handle(stream)))
        if own:
            _raise_on_status("tkef_aggregate_execute", status, stream)


# ----------------------------------------------------------------------------
# one-shot calls: each calls the C one-shot of the same name. Without a caller
# status word they use their own, synchronize and raise TkefStatusError when
# the device reports a problem; with one, checking it is the caller's.

def _ws(nbytes: int, dev) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=dev)


def _finish(fn: str, status: Optional[torch.Tensor], own: bool) -> None:
    if own:
        _raise_on_status(fn, status)


def sparsify(grads: Sequence[torch.Tensor], residuals: Sequence[torch.Tensor],
             rho: Optional[float] = None, mode: int = GLOBAL, k: Optional[int] = None,
             status: Optional[torch.Tensor] = None, val_dtype=torch.float32,
             return_counts: bool = False):
    """x = g + r; top-k of |x| (ties to the lower position); r <- x with the
    selected entries zeroed. Returns (idx int32, val of val_dtype: float32,
    or float16 rounded to nearest even), and with return_counts the k of each
    selection group."""
    if len(grads) != len(residuals) or not grads:
        raise ValueError("grads and residuals: equal, non-empty lists")
    _check_f32_tensors(list(grads) + list(residuals), "sparsify")
    numels = [t.numel() for t in grads]
    if [t.numel() for t in residuals] != numels:
        raise ValueError("residual sizes differ from the gradients'")
    L = lib()
    arr = _i64_array(numels)
    rho_v, k_v = float(rho) if rho is not None else 0.0, int(k) if k else 0
    nbytes, kt = ctypes.c_size_t(), ctypes.c_int64()
    _check("tkef_sparsify_workspace", L.tkef_sparsify_workspace(
        arr, len(numels), int(mode), rho_v, k_v, ctypes.byref(nbytes), ctypes.byref(kt)))
    dev = grads[0].device
    ngroups = len(numels) if mode == PER_TENSOR else 1
    counts = (ctypes.c_int64 * ngroups)()
    idx = torch.empty(max(kt.value, 1), dtype=torch.int32, device=dev)
    val = torch.empty(max(kt.value, 1), dtype=val_dtype, device=dev)
    own = status is None
    if own:
        status = _new_status(dev)
    _check("tkef_sparsify", L.tkef_sparsify(
        _ptr_array(grads), _ptr_array(residuals), arr, len(numels), int(mode), rho_v, k_v,
        _val_format(val_dtype), idx.data_ptr(), val.data_ptr(), counts,
        _ws(nbytes.value, dev).data_ptr(), max(nbytes.value, 256), status.data_ptr(),
        _stream_handle(None)))
    _finish("tkef_sparsify", status, own)
    out = (idx[: kt.value], val[: kt.value])
    return (*out, list(counts)) if return_counts else out


def sparsify1(g: torch.Tensor, r: torch.Tensor, k: int,
              status: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """One flat tensor, explicit k (tkef_sparsify1). Returns (idx, val)."""
    _check_f32_tensors([g, r], "sparsify1")
    d = g.numel()
    if r.numel() != d:
        raise ValueError("g and r differ in size")
    L = lib()
    nbytes = ctypes.c_size_t()
    _check("tkef_sparsify_workspace", L.tkef_sparsify_workspace(
        _i64_array([d]), 1, GLOBAL, 0.0, int(k), ctypes.byref(nbytes), None))
    idx = torch.empty(max(int(k), 1), dtype=torch.int32, device=g.device)
    val = torch.empty(max(int(k), 1), dtype=torch.float32, device=g.device)
    own = status is None
    if own:
        status = _new_status(g.device)
    _check("tkef_sparsify1", L.tkef_sparsify1(
        g.data_ptr(), r.data_ptr(), d, int(k), idx.data_ptr(), val.data_ptr(),
        _ws(nbytes.value, g.device).data_ptr(), max(nbytes.value, 256), status.data_ptr(),
        _stream_handle(None)))
    _finish("tkef_sparsify1", status, own)
    return idx[: int(k)], val[: int(k)]


STATIC_MAX_D = 1 << 26
STATIC_MAX_K = 1 << 17


def sparsify1_static(g: torch.Tensor, r: torch.Tensor, k: int,
                     idx_out: Optional[torch.Tensor] = None,
                     val_out: Optional[torch.Tensor] = None,
                     status: Optional[torch.Tensor] = None, stream=None
                     ) -> Tuple[torch.Tensor, torch.Tensor]:
    """tkef_sparsify1 with the library's fixed scratch (tkef_sparsify1_static,
    for callers that cannot allocate): no workspace, no synchronization.
    With idx_out / val_out / status given, this function allocates nothing
    either; the status word, when given, is the caller's to check."""
    _check_f32_tensors([g, r], "sparsify1_static")
    d = g.numel()
    if r.numel() != d:
        raise ValueError("g and r differ in size")
    if idx_out is None:
        idx_out = torch.empty(max(int(k), 1), dtype=torch.int32, device=g.device)
    if val_out is None:
        val_out = torch.empty(max(int(k), 1), dtype=torch.float32, device=g.device)
    if idx_out.numel() < k or val_out.numel() < k or idx_out.dtype != torch.int32 or \
            val_out.dtype != torch.float32:
        raise ValueError("idx_out (int32) and val_out (float32) must hold k entries")
    _check("tkef_sparsify1_static", lib().tkef_sparsify1_static(
        g.data_ptr(), r.data_ptr(), d, int(k), idx_out.data_ptr(), val_out.data_ptr(),
        status.data_ptr() if status is not None else None, _stream_handle(stream)))
    return idx_out[: int(k)], val_out[: int(k)]


def aggregate_update(params: Sequence[torch.Tensor],
                     lists: Sequence[Tuple[torch.Tensor, torch.Tensor]], lr: float,
                     momentum: Optional[Sequence[torch.Tensor]] = None, mu: float = 0.0,
                     wd: float = 0.0, status: Optional[torch.Tensor] = None) -> None:
    """Sum P separate worker lists [(idx_p int32, val_p float32), ...] (each
    ascending) and apply w -= lr * (sum [+ wd * w], through momentum if
    mu != 0): tkef_aggregate_update."""
    _check_f32_tensors(list(params) + list(momentum or []), "aggregate_update")
    numels = [t.numel() for t in params]
    P = len(lists)
    if P < 1:
        raise ValueError("at least one worker list")
    for i, v in lists:
        if i.dtype != torch.int32 or v.dtype != torch.float32 or i.numel() != v.numel():
            raise ValueError("each list: int32 idx and float32 val of one length")
        if i.numel() and not (i.is_cuda and v.is_cuda and i.is_contiguous() and v.is_contiguous()):
            raise ValueError("lists must be contiguous CUDA tensors")
    L = lib()
    arr = _i64_array(numels)
    nbytes = ctypes.c_size_t()
    _check("tkef_aggregate_workspace", L.tkef_aggregate_workspace(
        arr, len(numels), P, ctypes.byref(nbytes)))
    dev = params[0].device
    own = status is None
    if own:
        status = _new_status(dev)
    ip = (ctypes.c_void_p * P)(*[(i.data_ptr() if i.numel() else None) for i, _ in lists])
    vp = (ctypes.c_void_p * P)(*[(v.data_ptr() if v.numel() else None) for _, v in lists])
    _check("tkef_aggregate_update", L.tkef_aggregate_update(
        _ptr_array(params), _ptr_array(momentum) if momentum is not None else None, arr,
        len(numels), ip, vp, _i64_array([i.numel() for i, _ in lists]), P, float(lr),
        float(mu), float(wd), _ws(nbytes.value, dev).data_ptr(), max(nbytes.value, 256),
        status.data_ptr(), _stream_handle(None)))
    _finish("tkef_aggregate_update", status, own)


def _gathered(idx: torch.Tensor, val: torch.Tensor):
    if idx.dim() == 1:
        idx, val = idx.view(1, -1), val.view(1, -1)
    if idx.shape != val.shape or idx.dtype != torch.int32:
        raise ValueError("idx (int32) and val: (P, stride) of one shape")
    return idx.contiguous(), val.contiguous(), idx.shape[0], idx.shape[1]


def sparse_aggregate_update(params: Sequence[torch.Tensor], idx: torch.Tensor,
                            val: torch.Tensor, lr: float,
                            momentum: Optional[Sequence[torch.Tensor]] = None,
                            mu: float = 0.0, wd: float = 0.0,
                            nnz: Optional[torch.Tensor] = None,
                            status: Optional[torch.Tensor] = None) -> None:
    """Sum P workers' sparse gradients (idx, val: (P, stride) gathered layout)
    and apply w -= lr * (sum [+ wd * w], through momentum if mu != 0):
    tkef_sparse_aggregate_update."""
    _check_f32_tensors(list(params) + list(momentum or []), "sparse_aggregate_update")
    idx, val, P, stride = _gathered(idx, val)
    if val.dtype != torch.float32:
        raise ValueError("values are float32 (binary16 lists: UpdatePlan)")
    numels = [t.numel() for t in params]
    L = lib()
    arr = _i64_array(numels)
    nbytes = ctypes.c_size_t()
    _check("tkef_update_workspace", L.tkef_update_workspace(
        arr, len(numels), P, stride, ctypes.byref(nbytes)))
    dev = params[0].device
    own = status is None
    if own:
        status = _new_status(dev)
    _check("tkef_sparse_aggregate_update", L.tkef_sparse_aggregate_update(
        _ptr_array(params), _ptr_array(momentum) if momentum is not None else None, arr,
        len(numels), idx.data_ptr(), val.data_ptr(), P, stride,
        nnz.data_ptr() if nnz is not None else None, float(lr), float(mu), float(wd),
        _ws(nbytes.value, dev).data_ptr(), max(nbytes.value, 256), status.data_ptr(),
        _stream_handle(None)))
    _finish("tkef_sparse_aggregate_update", status, own)


def sparse_aggregate(outs: Sequence[torch.Tensor], idx: torch.Tensor, val: torch.Tensor,
                     nnz: Optional[torch.Tensor] = None,
                     status: Optional[torch.Tensor] = None) -> None:
    """outs <- sum of P workers' sparse lists (idx, val: (P, stride) gathered
    layout), densely: every position written, zero where no list names it
    (tkef_sparse_aggregate; float32 or float16 values)."""
    _check_f32_tensors(list(outs), "sparse_aggregate")
    idx, val, P, stride = _gathered(idx, val)
    numels = [t.numel() for t in outs]
    L = lib()
    arr = _i64_array(numels)
    nbytes = ctypes.c_size_t()
    _check("tkef_update_workspace", L.tkef_update_workspace(
        arr, len(numels), P, stride, ctypes.byref(nbytes)))
    dev = outs[0].device
    own = status is None
    if own:
        status = _new_status(dev)
    _check("tkef_sparse_aggregate", L.tkef_sparse_aggregate(
        _ptr_array(outs), arr, len(numels), idx.data_ptr(), val.data_ptr(),
        _val_format(val.dtype), P, stride, nnz.data_ptr() if nnz is not None else None,
        _ws(nbytes.value, dev).data_ptr(), max(nbytes.value, 256), status.data_ptr(),
        _stream_handle(None)))
    _finish("tkef_sparse_aggregate", status, own)
