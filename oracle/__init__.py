"""CPU oracle (test infrastructure only).

Plain, slow reference for what the GPU library computes; see
``tkef_oracle.c`` for the definitions and their sources in the paper. Only the
tests, the smoke check and the CPU-baseline leg of the benchmark import this
package. It shares no code with the GPU library and never imports it.

The C part is built with gcc into ``oracle/liboracle.so`` (``build()``); the
list handling around it (concatenating a tensor list, per-tensor groups) is
plain numpy. The approximate selector of Alg. 1 (MSTopK) is plain numpy in
float64, in ``oracle/mstopk.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import List, Optional, Sequence, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "tkef_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
          "-fno-fast-math", "-Wall", "-Wextra"]

ORC_OK, ORC_EINVAL, ORC_ENAN, ORC_ENOMEM, ORC_ERANGE = 0, 1, 2, 3, 4

GLOBAL, PER_TENSOR = 0, 1


class OracleError(RuntimeError):
    pass


def build(src: str = SRC, out: str = LIB, extra: Sequence[str] = ()) -> str:
    """Compile the oracle with gcc (always recompiles)."""
    cmd = ["gcc", *CFLAGS, *extra, src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


_P = ctypes.POINTER


def _bind(lib: ctypes.CDLL) -> ctypes.CDLL:
    i64, i32, f32, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_void_p
    lib.oracle_version.restype = ctypes.c_int
    lib.oracle_k_from_rho.argtypes = [i64, ctypes.c_double]
    lib.oracle_k_from_rho.restype = i64
    lib.oracle_ef_add.argtypes = [vp, vp, vp, i64]
    lib.oracle_ef_add.restype = None
    lib.oracle_topk_select.argtypes = [vp, i64, i64, vp]
    lib.oracle_topk_select.restype = ctypes.c_int
    lib.oracle_sparsify.argtypes = [vp, vp, i64, i64, i64, vp, vp, vp]
    lib.oracle_sparsify.restype = ctypes.c_int
    lib.oracle_rank.argtypes = [vp, i64, i64]
    lib.oracle_rank.restype = i64
    lib.oracle_update.argtypes = [vp, vp, i64, i32, vp, vp, i64, vp, f32, f32, f32]
    lib.oracle_update.restype = ctypes.c_int
    lib.oracle_aggregate.argtypes = [vp, i64, i32, vp, vp, i64, vp]
    lib.oracle_aggregate.restype = ctypes.c_int
    return lib


_lib: Optional[ctypes.CDLL] = None


def load(path: str = LIB) -> ctypes.CDLL:
    """Load the built oracle, building it first only if nothing is built."""
    global _lib
    if path == LIB and _lib is not None:
        return _lib
    if not os.path.exists(path):
        if path != LIB:
            raise FileNotFoundError(path)
        build()
    lib = _bind(ctypes.CDLL(path))
    if path == LIB:
        _lib = lib
    return lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


def f16_rne(x) -> np.ndarray:
    """Values on the wire in 16-bit floating point (Sec. 5.3 sends FP16
    elements): binary32 -> binary16, round to nearest, ties to even, overflow
    to infinity, subnormals kept (numpy's IEEE conversion)."""
    with np.errstate(over="ignore"):
        return np.ascontiguousarray(x, dtype=np.float32).astype(np.float16)


class Oracle:
    """numpy-facing wrapper around one build of the C oracle."""

    def __init__(self, lib: Optional[ctypes.CDLL] = None):
        self.lib = lib if lib is not None else load()

    # -- pieces ------------------------------------------------------------
    def k_from_rho(self, d: int, rho: float) -> int:
        return int(self.lib.oracle_k_from_rho(d, rho))

    def ef_add(self, g, r) -> np.ndarray:
        g, r = _f32(g), _f32(r)
        x = np.empty_like(g)
        self.lib.oracle_ef_add(_ptr(g), _ptr(r), _ptr(x), g.size)
        return x

    def topk_select(self, x, k: int) -> np.ndarray:
        x = _f32(x)
        sel = np.empty(max(k, 1), dtype=np.int64)
        rc = self.lib.oracle_topk_select(_ptr(x), x.size, k, _ptr(sel))
        if rc != ORC_OK:
            raise OracleError(f"oracle_topk_select rc={rc}")
        return sel[:k]

    def rank(self, x, i: int) -> int:
        x = _f32(x)
        return int(self.lib.oracle_rank(_ptr(x), x.size, i))

    # -- sparsify ----------------------------------------------------------
    def sparsify_flat(self, g, r, k: int, index_base: int = 0
                      ) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
        g, r = _f32(g), _f32(r)
        n = g.size
        idx = np.empty(max(k, 1), dtype=np.int32)
        val = np.empty(max(k, 1), dtype=np.float32)
        r_out = np.empty(n, dtype=np.float32)
        rc = self.lib.oracle_sparsify(_ptr(g), _ptr(r), n, k, index_base,
                                      _ptr(idx), _ptr(val), _ptr(r_out))
        if rc != ORC_OK:
            raise OracleError(f"oracle_sparsify rc={rc}")
        return idx[:k], val[:k], r_out

    def sparsify(self, grads: Sequence[np.ndarray], residuals: Sequence[np.ndarray],
                 rho: Optional[float] = None, mode: int = GLOBAL, k: Optional[int] = None
                 ) -> Tuple[np.ndarray, np.ndarray, List[np.ndarray], List[int]]:
        """Tensor-list sparsify. GLOBAL: one selection over the concatenation
        in list order (k from rho over the total size, or explicit k).
        PER_TENSOR: one selection per tensor with k_t from rho over its size;
        outputs concatenated in tensor order. Indices are global positions in
        the concatenation. Returns (idx, val, new residuals, group sizes)."""
        sizes = [int(np.asarray(a).size) for a in grads]
        offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
        if mode == GLOBAL:
            g = np.concatenate([_f32(a).ravel() for a in grads]) if grads else np.empty(0, np.float32)
            r = np.concatenate([_f32(a).ravel() for a in residuals]) if residuals else np.empty(0, np.float32)
            kk = int(k) if k is not None else self.k_from_rho(int(g.size), rho)
            idx, val, r_out = self.sparsify_flat(g, r, kk)
            outs = [r_out[offs[t]:offs[t + 1]].reshape(np.shape(residuals[t]))
                    for t in range(len(sizes))]
            return idx, val, outs, [kk]
        if mode != PER_TENSOR:
            raise ValueError("mode")
        if k is not None:
            raise ValueError("explicit k only in GLOBAL mode")
        idxs, vals, outs, ks = [], [], [], []
        for t, (ga, ra) in enumerate(zip(grads, residuals)):
            n = sizes[t]
            kt = self.k_from_rho(n, rho)
            i, v, ro = self.sparsify_flat(_f32(ga).ravel(), _f32(ra).ravel(), kt,
                                          index_base=int(offs[t]))
            idxs.append(i)
            vals.append(v)
            outs.append(ro.reshape(np.shape(ra)))
            ks.append(kt)
        return (np.concatenate(idxs) if idxs else np.empty(0, np.int32),
                np.concatenate(vals) if vals else np.empty(0, np.float32), outs, ks)

    # -- aggregate + update ------------------------------------------------
    def aggregate(self, d: int, idx, val, nnz=None) -> np.ndarray:
        """Dense sum of the lists (Alg. 2 accumulation), worker order. idx,
        val: (P, stride) gathered layout (float16 values are widened exactly)."""
        idx = np.ascontiguousarray(idx, dtype=np.int32)
        val = np.ascontiguousarray(np.asarray(val).astype(np.float32))
        if idx.ndim == 1:
            idx, val = idx[None, :], val[None, :]
        P, stride = idx.shape
        nnz = np.full(P, stride, np.int64) if nnz is None else np.ascontiguousarray(nnz, np.int64)
        # NaN-filled, so that a position the C code never writes shows up
        out = np.full(max(d, 1), np.nan, dtype=np.float32)
        rc = self.lib.oracle_aggregate(_ptr(out), d, P, _ptr(idx), _ptr(val), stride, _ptr(nnz))
        if rc != ORC_OK:
            raise OracleError(f"oracle_aggregate rc={rc}")
        return out[:d]

    def update(self, w, b, idx, val, nnz=None, lr=0.1, mu=0.0, wd=0.0
               ) -> Tuple[np.ndarray, Optional[np.ndarray]]:
        """w, b: flat float32 (copies are updated and returned). idx, val:
        (P, stride) arrays in the gathered layout; nnz: per-worker counts
        (default: all of each row)."""
        w = np.array(w, dtype=np.float32, copy=True).ravel()
        bb = None if b is None else np.array(b, dtype=np.float32, copy=True).ravel()
        idx = np.ascontiguousarray(idx, dtype=np.int32)
        val = np.ascontiguousarray(val, dtype=np.float32)
        if idx.ndim == 1:
            idx, val = idx[None, :], val[None, :]
        P, stride = idx.shape
        nnz = np.full(P, stride, np.int64) if nnz is None else np.ascontiguousarray(nnz, np.int64)
        rc = self.lib.oracle_update(_ptr(w), 0 if bb is None else _ptr(bb), w.size, P,
                                    _ptr(idx), _ptr(val), stride, _ptr(nnz),
                                    np.float32(lr), np.float32(mu), np.float32(wd))
        if rc != ORC_OK:
            raise OracleError(f"oracle_update rc={rc}")
        return w, bb
