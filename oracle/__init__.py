"""CPU oracle for the Polyglot window-ranking LM step -- TEST INFRASTRUCTURE.

Only the test suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg
of ``bench.py`` may import this package.  The product path (the HIP library
and its Python binding) never imports, links or calls anything here, and this
package imports nothing from the product.

The arithmetic lives in ``oracle.cpp`` (plain single-threaded C++, float64
arithmetic, built with g++ -O2 and no fast-math).  This module only loads the
shared library with ctypes and marshals numpy arrays.

Model (the reading of the paper's SENNA-like ranking LM, §1 Introduction):
``s(x) = w2 . tanh(W1 x + b1) + b2``, hinge ``max(0, 1 - s(x) + s(x~))``
against the window with its centre word replaced, mean over the batch,
plain SGD.  The embedding gradient is the row scatter-add that §4.2 (Table 1)
profiles and §4.3 optimises.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.cpp")
_LIB = os.path.join(_HERE, "liboracle.so")

# Error codes returned by the C entry points.
OK, EINVAL, ENULL, EID = 0, -1, -2, -5


class OracleError(RuntimeError):
    def __init__(self, rc: int, what: str):
        super().__init__(f"oracle {what} failed with code {rc}")
        self.rc = rc


def build(force: bool = True) -> str:
    """Compile liboracle.so with g++ (-O2, no fast-math, single-threaded)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(
            ["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-fno-fast-math",
             "-o", tmp, _SRC],
            check=True,
        )
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        i32, dbl, lng = ctypes.c_int, ctypes.c_double, ctypes.c_long
        p = ctypes.c_void_p
        lib.oracle_train_step_f32.argtypes = [i32] * 5 + [p] * 7 + [dbl, p]
        lib.oracle_train_step_f64.argtypes = [i32] * 5 + [p] * 7 + [dbl, p]
        lib.oracle_gradients_f64.argtypes = [i32] * 5 + [p] * 7 + [p] * 6
        lib.oracle_loss_f64.argtypes = [i32] * 5 + [p] * 7 + [p]
        lib.oracle_score_f32.argtypes = [i32] * 5 + [p] * 6 + [p]
        lib.oracle_score_f64.argtypes = [i32] * 5 + [p] * 6 + [p]
        lib.oracle_gather_f32.argtypes = [i32] * 4 + [p] * 5
        lib.oracle_touched_rows.argtypes = [i32] * 3 + [p, p, p, ctypes.c_int32, p]
        lib.oracle_scatter_add_f32.argtypes = [i32, i32, p, p, p, lng, dbl]
        lib.oracle_scatter_add_f64.argtypes = [i32, i32, p, p, p, lng, dbl]
        lib.oracle_scatter_add_ex.argtypes = [i32, i32, p, i32, p, i32, p, lng, dbl, i32]
        lib.oracle_encode.argtypes = [i32, p, lng, p]
        lib.oracle_decode.argtypes = [i32, p, lng, p]
        for name in ("oracle_train_step_f32", "oracle_train_step_f64", "oracle_gradients_f64",
                     "oracle_loss_f64", "oracle_score_f32", "oracle_score_f64",
                     "oracle_gather_f32", "oracle_touched_rows", "oracle_scatter_add_f32",
                     "oracle_scatter_add_f64", "oracle_scatter_add_ex", "oracle_encode",
                     "oracle_decode"):
            getattr(lib, name).restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _arr(a, dtype):
    a = np.asarray(a)
    if a.dtype != dtype or not a.flags.c_contiguous:
        raise TypeError(f"expected C-contiguous {np.dtype(dtype).name}, got {a.dtype}")
    return a


def _check(rc, what):
    if rc != OK:
        raise OracleError(rc, what)


def _dims(params, windows):
    E, W1 = params["E"], params["W1"]
    V, d = E.shape
    H = W1.shape[0]
    B, win = windows.shape
    return V, d, win, H, B


def train_step(params: dict, windows, corrupt, lr: float) -> float:
    """One SGD step in place on ``params`` (dict E, W1, b1, w2, b2; all
    float32 or all float64).  Returns the mean hinge loss before the update."""
    dt = params["E"].dtype
    if dt not in (np.float32, np.float64):
        raise TypeError("params must be float32 or float64")
    for k in ("E", "W1", "b1", "w2", "b2"):
        _arr(params[k], dt)
    windows = _arr(windows, np.int32)
    corrupt = _arr(corrupt, np.int32)
    V, d, win, H, B = _dims(params, windows)
    loss = ctypes.c_double()
    fn = _load().oracle_train_step_f32 if dt == np.float32 else _load().oracle_train_step_f64
    rc = fn(V, d, win, H, B, *[_ptr(params[k]) for k in ("E", "W1", "b1", "w2", "b2")],
            _ptr(windows), _ptr(corrupt), float(lr), ctypes.byref(loss))
    _check(rc, "train_step")
    return loss.value


def gradients(params: dict, windows, corrupt):
    """Mean loss and gradients (float64 params only).  dE is dense [V][d]."""
    for k in ("E", "W1", "b1", "w2", "b2"):
        _arr(params[k], np.float64)
    windows = _arr(windows, np.int32)
    corrupt = _arr(corrupt, np.int32)
    V, d, win, H, B = _dims(params, windows)
    loss = ctypes.c_double()
    db2 = ctypes.c_double()
    g = {"E": np.zeros((V, d)), "W1": np.zeros((H, win * d)), "b1": np.zeros(H),
         "w2": np.zeros(H)}
    rc = _load().oracle_gradients_f64(
        V, d, win, H, B, *[_ptr(params[k]) for k in ("E", "W1", "b1", "w2", "b2")],
        _ptr(windows), _ptr(corrupt), ctypes.byref(loss), _ptr(g["E"]), _ptr(g["W1"]),
        _ptr(g["b1"]), _ptr(g["w2"]), ctypes.byref(db2))
    _check(rc, "gradients")
    g["b2"] = np.array([db2.value])
    return loss.value, g


def loss(params: dict, windows, corrupt) -> float:
    """Mean hinge loss (float64 params only)."""
    for k in ("E", "W1", "b1", "w2", "b2"):
        _arr(params[k], np.float64)
    windows = _arr(windows, np.int32)
    corrupt = _arr(corrupt, np.int32)
    V, d, win, H, B = _dims(params, windows)
    out = ctypes.c_double()
    rc = _load().oracle_loss_f64(V, d, win, H, B,
                                 *[_ptr(params[k]) for k in ("E", "W1", "b1", "w2", "b2")],
                                 _ptr(windows), _ptr(corrupt), ctypes.byref(out))
    _check(rc, "loss")
    return out.value


def score(params: dict, windows) -> np.ndarray:
    """Scores s(x) of the true windows, float64."""
    dt = params["E"].dtype
    for k in ("E", "W1", "b1", "w2", "b2"):
        _arr(params[k], dt)
    windows = _arr(windows, np.int32)
    V, d, win, H, B = _dims(params, windows)
    out = np.zeros(B, np.float64)
    fn = _load().oracle_score_f32 if dt == np.float32 else _load().oracle_score_f64
    rc = fn(V, d, win, H, B, *[_ptr(params[k]) for k in ("E", "W1", "b1", "w2", "b2")],
            _ptr(windows), _ptr(out))
    _check(rc, "score")
    return out


def gather(E, windows, corrupt):
    """X[B][win*d] and Xc[B][d]: plain copies of the embedding rows."""
    E = _arr(E, np.float32)
    windows = _arr(windows, np.int32)
    corrupt = _arr(corrupt, np.int32)
    V, d = E.shape
    B, win = windows.shape
    X = np.empty((B, win * d), np.float32)
    Xc = np.empty((B, d), np.float32)
    rc = _load().oracle_gather_f32(V, d, win, B, _ptr(E), _ptr(windows), _ptr(corrupt),
                                   _ptr(X), _ptr(Xc))
    _check(rc, "gather")
    return X, Xc


def touched_rows(V: int, windows, corrupt) -> np.ndarray:
    """Sorted distinct rows touched by one step."""
    windows = _arr(windows, np.int32)
    corrupt = _arr(corrupt, np.int32)
    B, win = windows.shape
    cap = B * (win + 1)
    out = np.empty(max(cap, 1), np.int32)
    n = ctypes.c_int32()
    rc = _load().oracle_touched_rows(V, win, B, _ptr(windows), _ptr(corrupt), _ptr(out), cap,
                                     ctypes.byref(n))
    _check(rc, "touched_rows")
    return out[: n.value].copy()


def scatter_add(table, idx, Y, alpha: float = 1.0) -> None:
    """In place: for k in order, table[idx[k]] += alpha * Y[k] (float64 carry)."""
    dt = table.dtype
    table = _arr(table, dt)
    Y = _arr(Y, dt)
    idx = _arr(idx, np.int32)
    rows, d = table.shape
    N = idx.shape[0]
    if Y.shape != (N, d):
        raise ValueError("Y must be [len(idx)][d]")
    fn = _load().oracle_scatter_add_f32 if dt == np.float32 else _load().oracle_scatter_add_f64
    rc = fn(rows, d, _ptr(table), _ptr(idx), _ptr(Y), N, float(alpha))
    _check(rc, "scatter_add")


# storage formats and ops of the general advanced-indexing op
F32, BF16, F16 = 0, 1, 2
OP_INC, OP_SET = 0, 1


def _dtype_code(arr, bf16):
    if bf16:
        if arr.dtype != np.uint16:
            raise ValueError("bfloat16 arrays are passed as their uint16 bit patterns")
        return BF16
    if arr.dtype == np.float32:
        return F32
    if arr.dtype == np.float16:
        return F16
    raise ValueError("table must be float32, float16, or bfloat16 bits (uint16, bf16=True)")


def scatter_add_ex(table, idx, Y, alpha: float = 1.0, op: int = OP_INC, bf16: bool = False) -> None:
    """In place, the general op: op=OP_INC does table[idx[k]] += alpha*Y[k]
    for k in order (rows carried in float64, rounded once to the storage
    format, to nearest even); op=OP_SET does table[idx[k]] = Y[k] (last
    wins).  table/Y: float32, float16, or bfloat16 bit patterns as uint16 with
    bf16=True; idx: int32 or int64."""
    code = _dtype_code(table, bf16)
    if Y.dtype != table.dtype:
        raise ValueError("Y must have the table's storage format")
    if not (table.flags.c_contiguous and Y.flags.c_contiguous):
        raise ValueError("table and Y must be C-contiguous")
    idx = np.ascontiguousarray(idx)
    if idx.dtype not in (np.int32, np.int64):
        raise ValueError("idx must be int32 or int64")
    rows, d = table.shape
    N = idx.shape[0]
    if Y.shape != (N, d):
        raise ValueError("Y must be [len(idx)][d]")
    rc = _load().oracle_scatter_add_ex(rows, d, _ptr(table), code, _ptr(idx), idx.dtype.itemsize,
                                       _ptr(Y), N, float(alpha), int(op))
    _check(rc, "scatter_add_ex")


def encode(x, dtype: int) -> np.ndarray:
    """float64 values rounded to a storage format (F32 -> float32 array,
    BF16 / F16 -> uint16 bit patterns)."""
    x = np.ascontiguousarray(x, np.float64)
    out = np.empty(x.shape, np.float32 if dtype == F32 else np.uint16)
    _check(_load().oracle_encode(int(dtype), _ptr(x), x.size, _ptr(out)), "encode")
    return out


def decode(a, dtype: int) -> np.ndarray:
    """Storage-format values (as produced by encode) to float64."""
    a = np.ascontiguousarray(a)
    x = np.empty(a.shape, np.float64)
    _check(_load().oracle_decode(int(dtype), _ptr(a), a.size, _ptr(x)), "decode")
    return x
