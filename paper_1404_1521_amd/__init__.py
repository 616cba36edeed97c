"""Python binding of libpolyglot.so, the MI355X (gfx950) HIP library for the
minibatch SGD step of the Polyglot window-ranking language model
(Kulkarni et al., arXiv:1404.1521; model per §1 Introduction, embedding
scatter-add per §4.2-§4.3).

This module only marshals arguments: it checks tensor dtypes, devices and
shapes, passes raw device pointers and the HIP stream to the C ABI of
include/polyglot.h, and raises on a nonzero return code.  Every step of the
computation runs in the library's HIP kernels.  PyTorch supplies device
memory and streams.  There is no fallback: if the library is not built, or no
GPU is present, the calls raise.
"""
from __future__ import annotations

import ctypes
import os

import torch  # loaded first: the library then binds to torch's HIP runtime

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpolyglot.so")

OK, EINVAL, ENULL, EBATCH, EHIP, EID, ESTATE = 0, -1, -2, -3, -4, -5, -6
SCATTER_SORTED, SCATTER_ATOMIC = 0, 1
F32, BF16, F16 = 0, 1, 2      # storage formats of scatter_update
OP_INC, OP_SET = 0, 1         # its operations
_CODE_NAMES = {EINVAL: "EINVAL", ENULL: "ENULL", EBATCH: "EBATCH", EHIP: "EHIP", EID: "EID",
               ESTATE: "ESTATE"}

# Every entry point declared in include/polyglot.h.
EXPORTS = ("polyglot_init", "polyglot_destroy", "polyglot_set_stream", "polyglot_train_step",
           "polyglot_train_step_sync", "polyglot_train_steps", "polyglot_score", "polyglot_gather", "polyglot_scatter_add",
           "polyglot_scatter_update", "polyglot_scatter_add_noalloc",
           "polyglot_touched_rows", "polyglot_status", "polyglot_last_error",
           "polyglot_set_timing", "polyglot_kernel_times")
KERNEL_NAMES = ("fwdbwd", "sort", "update", "gather", "scatter", "score", "segfix", "wide_dw1",
                "wide_g")


class PolyglotError(RuntimeError):
    def __init__(self, rc: int, msg: str):
        super().__init__(f"{_CODE_NAMES.get(rc, rc)}: {msg}")
        self.rc = rc


class Config(ctypes.Structure):
    _fields_ = [("V", ctypes.c_int32), ("d", ctypes.c_int32), ("win", ctypes.c_int32),
                ("H", ctypes.c_int32), ("max_batch", ctypes.c_int32),
                ("scatter_mode", ctypes.c_int32), ("max_scatter", ctypes.c_int32),
                ("max_rows", ctypes.c_int32)]


_lib = None


def load_library():
    """Loads libpolyglot.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run paper_1404_1521_amd.build.build()")
    lib = ctypes.CDLL(LIB_PATH)
    p, i32, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
    sig = {
        "polyglot_init": [ctypes.POINTER(Config), p, ctypes.POINTER(p)],
        "polyglot_destroy": [p],
        "polyglot_set_stream": [p, p],
        "polyglot_train_step": [p] + [p] * 7 + [i32, f32, p],
        "polyglot_train_step_sync": [p] + [p] * 7 + [i32, f32, ctypes.POINTER(f32)],
        "polyglot_train_steps": [p] + [p] * 7 + [i32, i32, f32, p],
        "polyglot_score": [p] + [p] * 6 + [i32, p],
        "polyglot_gather": [p, p, p, p, i32, p, p],
        "polyglot_scatter_add": [p, p, i32, i32, p, p, i32, f32, i32],
        "polyglot_scatter_update": [p, p, i32, i32, i32, p, i32, p, i32, f32, i32, i32],
        "polyglot_scatter_add_noalloc": [p, i32, i32, p, p, i32, f32, p, p],
        "polyglot_touched_rows": [p, p, i32, p],
        "polyglot_status": [p],
        "polyglot_last_error": [p],
        "polyglot_set_timing": [p, ctypes.c_int],
        "polyglot_kernel_times": [p, p, p],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_char_p if name == "polyglot_last_error" else ctypes.c_int
    _lib = lib
    return lib


def _dev_tensor(t, dtype, name, shape=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device (cuda) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return ctypes.c_void_p(t.data_ptr())


NOALLOC_MAX_N = 8192  # POLYGLOT_NOALLOC_MAX_N


def scatter_add_noalloc(table, idx, Y, alpha: float = 1.0, status=None, stream=None) -> None:
    """table[idx[k]] += alpha * Y[k] (sorted mode) through the entry point that
    allocates nothing and needs no context (N <= NOALLOC_MAX_N).  status: an
    optional int32 device tensor of one element that receives OK or EID on
    the device.  Asynchronous on `stream` (default: torch's current stream)."""
    lib = load_library()
    rows, d = table.shape
    N = idx.shape[0]
    st = stream if stream is not None else torch.cuda.current_stream()
    sp = None if status is None else _dev_tensor(status, torch.int32, "status", (1,))
    rc = lib.polyglot_scatter_add_noalloc(
        _dev_tensor(table, torch.float32, "table"), rows, d,
        _dev_tensor(idx, torch.int32, "idx", (N,)),
        _dev_tensor(Y, torch.float32, "Y", (N, d)), N, alpha, sp,
        ctypes.c_void_p(st.cuda_stream))
    if rc != OK:
        raise PolyglotError(rc, "scatter_add_noalloc")


class Context:
    """A library context (workspace + stream) for one model shape."""

    def __init__(self, V: int, d: int, win: int, H: int, max_batch: int,
                 scatter_mode: int = SCATTER_SORTED, max_scatter: int = 0, max_rows: int = 0,
                 stream: torch.cuda.Stream | None = None):
        self._lib = load_library()
        if not torch.cuda.is_available():
            raise RuntimeError("no GPU: the Polyglot HIP library needs an MI355X device")
        self.cfg = Config(V, d, win, H, max_batch, scatter_mode, max_scatter, max_rows)
        self.V, self.d, self.win, self.H = V, d, win, H
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        h = ctypes.c_void_p()
        rc = self._lib.polyglot_init(ctypes.byref(self.cfg), ctypes.c_void_p(self.stream.cuda_stream),
                                     ctypes.byref(h))
        if rc != OK:
            raise PolyglotError(rc, "polyglot_init failed")
        self._h = h

    # ------------------------------------------------------------------ helpers
    def _check(self, rc: int, what: str):
        if rc != OK:
            msg = self._lib.polyglot_last_error(self._h)
            raise PolyglotError(rc, f"{what}: {msg.decode() if msg else ''}")

    def _params(self, params: dict):
        V, d, win, H = self.V, self.d, self.win, self.H
        return [_dev_tensor(params["E"], torch.float32, "E", (V, d)),
                _dev_tensor(params["W1"], torch.float32, "W1", (H, win * d)),
                _dev_tensor(params["b1"], torch.float32, "b1", (H,)),
                _dev_tensor(params["w2"], torch.float32, "w2", (H,)),
                _dev_tensor(params["b2"], torch.float32, "b2", (1,))]

    # -------------------------------------------------------------- entry points
    def train_step(self, params: dict, windows, corrupt, lr: float, loss_out=None) -> None:
        """One SGD step in place on params (asynchronous on the context stream)."""
        B = windows.shape[0]
        args = self._params(params)
        w = _dev_tensor(windows, torch.int32, "windows", (B, self.win))
        c = _dev_tensor(corrupt, torch.int32, "corrupt", (B,))
        lo = None if loss_out is None else _dev_tensor(loss_out, torch.float32, "loss_out")
        self._check(self._lib.polyglot_train_step(self._h, *args, w, c, B, lr, lo), "train_step")

    def train_step_sync(self, params: dict, windows, corrupt, lr: float) -> float:
        """One SGD step in place on params; synchronises the context stream and
        returns the step's mean loss as a Python float."""
        B = windows.shape[0]
        args = self._params(params)
        w = _dev_tensor(windows, torch.int32, "windows", (B, self.win))
        c = _dev_tensor(corrupt, torch.int32, "corrupt", (B,))
        loss = ctypes.c_float(0.0)
        self._check(self._lib.polyglot_train_step_sync(self._h, *args, w, c, B, lr,
                                                       ctypes.byref(loss)), "train_step_sync")
        return loss.value

    def train_steps(self, params: dict, windows, corrupt, lr: float, losses_out=None) -> None:
        """S steps over windows[S][B][win], corrupt[S][B] (graph-replayed)."""
        S, B = windows.shape[0], windows.shape[1]
        args = self._params(params)
        w = _dev_tensor(windows, torch.int32, "windows", (S, B, self.win))
        c = _dev_tensor(corrupt, torch.int32, "corrupt", (S, B))
        lo = None if losses_out is None else _dev_tensor(losses_out, torch.float32, "losses", (S,))
        self._check(self._lib.polyglot_train_steps(self._h, *args, w, c, S, B, lr, lo),
                    "train_steps")

    def score(self, params: dict, windows, out=None):
        B = windows.shape[0]
        if out is None:
            out = torch.empty(B, dtype=torch.float32, device=windows.device)
        args = self._params(params)
        w = _dev_tensor(windows, torch.int32, "windows", (B, self.win))
        o = _dev_tensor(out, torch.float32, "scores", (B,))
        self._check(self._lib.polyglot_score(self._h, *args, w, B, o), "score")
        return out

    def gather(self, E, windows, corrupt, X=None, Xc=None):
        B = windows.shape[0]
        if X is None:
            X = torch.empty(B, self.win * self.d, dtype=torch.float32, device=E.device)
        if Xc is None:
            Xc = torch.empty(B, self.d, dtype=torch.float32, device=E.device)
        self._check(self._lib.polyglot_gather(
            self._h, _dev_tensor(E, torch.float32, "E", (self.V, self.d)),
            _dev_tensor(windows, torch.int32, "windows", (B, self.win)),
            _dev_tensor(corrupt, torch.int32, "corrupt", (B,)), B,
            _dev_tensor(X, torch.float32, "X", (B, self.win * self.d)),
            _dev_tensor(Xc, torch.float32, "Xc", (B, self.d))), "gather")
        return X, Xc

    def scatter_add(self, table, idx, Y, alpha: float = 1.0, mode: int = SCATTER_SORTED) -> None:
        """table[idx[k]] += alpha * Y[k] for every k (repeated indices accumulate)."""
        rows, d = table.shape
        N = idx.shape[0]
        self._check(self._lib.polyglot_scatter_add(
            self._h, _dev_tensor(table, torch.float32, "table"), rows, d,
            _dev_tensor(idx, torch.int32, "idx", (N,)),
            _dev_tensor(Y, torch.float32, "Y", (N, d)), N, alpha, mode), "scatter_add")

    def scatter_update(self, table, idx, Y, alpha: float = 1.0, op: int = OP_INC,
                       mode: int = SCATTER_SORTED) -> None:
        """The general advanced-indexing op on a float32, bfloat16 or float16
        table (Y in the same dtype) with int32 or int64 indices: op=OP_INC
        adds alpha * Y[k] into row idx[k]; op=OP_SET assigns Y[k] (the last
        k of a row wins)."""
        codes = {torch.float32: F32, torch.bfloat16: BF16, torch.float16: F16}
        if table.dtype not in codes:
            raise TypeError(f"table must be float32, bfloat16 or float16, got {table.dtype}")
        if idx.dtype not in (torch.int32, torch.int64):
            raise TypeError(f"idx must be int32 or int64, got {idx.dtype}")
        rows, d = table.shape
        N = idx.shape[0]
        self._check(self._lib.polyglot_scatter_update(
            self._h, _dev_tensor(table, table.dtype, "table"), codes[table.dtype], rows, d,
            _dev_tensor(idx, idx.dtype, "idx", (N,)), idx.element_size(),
            _dev_tensor(Y, table.dtype, "Y", (N, d)), N, alpha, op, mode), "scatter_update")

    def touched_rows(self):
        n = ctypes.c_int32()
        self._check(self._lib.polyglot_touched_rows(self._h, None, 0, ctypes.byref(n)),
                    "touched_rows")
        buf = (ctypes.c_int32 * max(n.value, 1))()
        self._check(self._lib.polyglot_touched_rows(self._h, buf, n.value, ctypes.byref(n)),
                    "touched_rows")
        return list(buf)[: n.value]

    def set_timing(self, enable: bool) -> None:
        self._check(self._lib.polyglot_set_timing(self._h, int(enable)), "set_timing")

    def kernel_times(self) -> dict:
        """{kernel name: (total ms, launches)} since the last call; synchronises."""
        ms = (ctypes.c_double * len(KERNEL_NAMES))()
        n = (ctypes.c_int32 * len(KERNEL_NAMES))()
        self._check(self._lib.polyglot_kernel_times(self._h, ms, n), "kernel_times")
        return {name: (ms[i], n[i]) for i, name in enumerate(KERNEL_NAMES)}

    def status(self) -> int:
        """Synchronises; returns OK or EID (the sticky device flag), clearing it."""
        return self._lib.polyglot_status(self._h)

    def close(self):
        if getattr(self, "_h", None):
            self._lib.polyglot_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
