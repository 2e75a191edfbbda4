"""Thin ctypes binding over the engine's C ABI (include/xlh.h).

Argument marshalling only: every step of evaluation runs in the library's
HIP kernels.  PyTorch provides the device workspace and the stream.  The
library must have been built (``python -m paper_2609_27203_amd.build``);
there is no fallback of any kind when it is missing.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libxlh.so")

XL_OK = 0
STATUS = ["XL_OK", "XL_INVALID_ARGUMENT", "XL_TYPE_MISMATCH", "XL_UNSUPPORTED",
          "XL_RESOURCE_EXHAUSTED", "XL_CAPACITY_EXCEEDED", "XL_CONVERGENCE_FAILURE",
          "XL_DEVICE_ERROR", "XL_PARSE_ERROR"]
XL_I32, XL_F32, XL_U32, XL_I64, XL_U64, XL_F64, XL_BOOL = 1, 2, 3, 4, 5, 6, 7
_TYPES = {"i32": XL_I32, "f32": XL_F32, "u32": XL_U32, "i64": XL_I64, "u64": XL_U64, "f64": XL_F64,
          "bool": XL_BOOL}
_NP = {"i32": np.int32, "f32": np.float32, "u32": np.uint32, "i64": np.int64, "u64": np.uint64,
       "f64": np.float64, "bool": np.bool_}


def _torch_dtype(t: str):
    import torch
    return {"i32": torch.int32, "f32": torch.float32, "u32": torch.uint32, "i64": torch.int64,
            "u64": torch.uint64, "f64": torch.float64, "bool": torch.bool}[t]
STATS_ROUNDS = 256


class XlError(RuntimeError):
    def __init__(self, status: int, message: str):
        self.status = status
        self.status_name = STATUS[status] if 0 <= status < len(STATUS) else str(status)
        super().__init__(f"{self.status_name}: {message}")


class xl_fixpoint_stats(C.Structure):
    _fields_ = [
        ("status", C.c_int32), ("iterations", C.c_int32), ("strata", C.c_int32),
        ("rounds_recorded", C.c_int32), ("delta_rows", C.c_int64 * STATS_ROUNDS),
        ("candidates_total", C.c_int64), ("new_tuples_total", C.c_int64),
        ("derived_tuples", C.c_int64), ("peak_workspace_bytes", C.c_int64),
        ("control_bytes_read", C.c_int64), ("table_grows", C.c_int64), ("index_builds", C.c_int64), ("index_reuses", C.c_int64),
        ("ms_total", C.c_double),
        ("emit_ms", C.c_double), ("emit_launches", C.c_int64), ("emit_source_rows", C.c_int64),
        ("emit_candidates", C.c_int64), ("emit_new", C.c_int64),
        ("front_ms", C.c_double), ("front_launches", C.c_int64), ("front_candidates", C.c_int64),
        ("front_new", C.c_int64),
        ("pull_ms", C.c_double), ("pull_launches", C.c_int64), ("pull_candidates", C.c_int64),
        ("pull_new", C.c_int64),
        ("wcoj_ms", C.c_double), ("wcoj_launches", C.c_int64), ("wcoj_candidates", C.c_int64),
        ("wcoj_new", C.c_int64),
        ("gather_ms", C.c_double), ("gather_launches", C.c_int64), ("gather_candidates", C.c_int64),
        ("gather_new", C.c_int64),
    ]

    def as_dict(self) -> dict:
        n = min(self.rounds_recorded, STATS_ROUNDS)
        return {
            "status": STATUS[self.status], "iterations": self.iterations, "strata": self.strata,
            "rounds_recorded": self.rounds_recorded, "delta_rows": list(self.delta_rows[:n]),
            "candidates_total": self.candidates_total, "new_tuples_total": self.new_tuples_total,
            "derived_tuples": self.derived_tuples, "peak_workspace_bytes": self.peak_workspace_bytes,
            "control_bytes_read": self.control_bytes_read, "table_grows": self.table_grows,
            "index_builds": self.index_builds, "index_reuses": self.index_reuses,
            "ms_total": self.ms_total, "emit_ms": self.emit_ms, "emit_launches": self.emit_launches,
            "emit_source_rows": self.emit_source_rows, "emit_candidates": self.emit_candidates,
            "emit_new": self.emit_new, "front_ms": self.front_ms, "front_launches": self.front_launches,
            "front_candidates": self.front_candidates, "front_new": self.front_new,
            "pull_ms": self.pull_ms, "pull_launches": self.pull_launches,
            "pull_candidates": self.pull_candidates, "pull_new": self.pull_new,
            "wcoj_ms": self.wcoj_ms, "wcoj_launches": self.wcoj_launches,
            "wcoj_candidates": self.wcoj_candidates, "wcoj_new": self.wcoj_new,
            "gather_ms": self.gather_ms, "gather_launches": self.gather_launches,
            "gather_candidates": self.gather_candidates, "gather_new": self.gather_new,
        }


_lib = None
EXPORTS = ["xl_context_create", "xl_context_create_static", "xl_context_set_option", "xl_relation_create", "xl_relation_load",
           "xl_relation_clear", "xl_relation_size", "xl_relation_read", "xl_rule_compile",
           "xl_program_explain", "xl_fixpoint_run", "xl_last_error", "xl_status_string",
           "xl_program_destroy", "xl_relation_destroy", "xl_context_destroy"]


def lib() -> C.CDLL:
    """Load libxlh.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_27203_amd.build`")
    import torch  # noqa: F401  -- loads the HIP runtime the library is linked against
    L = C.CDLL(LIB_PATH)
    vp, i64, i32 = C.c_void_p, C.c_int64, C.c_int
    L.xl_context_create.argtypes = [i32, vp, vp, C.c_size_t, C.POINTER(vp)]
    L.xl_context_create_static.argtypes = [i32, vp, C.POINTER(vp)]
    L.xl_context_set_option.argtypes = [vp, C.c_char_p, i64]
    L.xl_relation_create.argtypes = [vp, C.c_char_p, i32, C.POINTER(C.c_int), i64, C.POINTER(vp)]
    L.xl_relation_load.argtypes = [vp, C.POINTER(vp), i64, i32]
    L.xl_relation_clear.argtypes = [vp]
    L.xl_relation_size.argtypes = [vp, C.POINTER(i64)]
    L.xl_relation_read.argtypes = [vp, C.POINTER(vp), i64, C.POINTER(i64), i32]
    L.xl_rule_compile.argtypes = [vp, C.c_char_p, C.POINTER(vp)]
    L.xl_program_explain.argtypes = [vp, C.c_char_p, C.c_size_t, C.POINTER(C.c_size_t)]
    L.xl_fixpoint_run.argtypes = [vp, i64, C.POINTER(xl_fixpoint_stats)]
    L.xl_last_error.argtypes = [vp]
    L.xl_last_error.restype = C.c_char_p
    L.xl_status_string.argtypes = [i32]
    L.xl_status_string.restype = C.c_char_p
    for f in ("xl_program_destroy", "xl_relation_destroy", "xl_context_destroy"):
        getattr(L, f).argtypes = [vp]
        getattr(L, f).restype = None
    for f in EXPORTS:
        if f not in ("xl_last_error", "xl_status_string") and getattr(L, f).restype is not None:
            getattr(L, f).restype = C.c_int
    _lib = L
    return L


class Context:
    """xl_context over a torch-allocated workspace on one device (or planning-only)."""

    def __init__(self, device: int = 0, workspace_bytes: int = 1 << 30, stream=None,
                 static: bool = False):
        """static=True: xl_context_create_static (the library's static 64 MiB
        device workspace, no allocation by the library or here)."""
        L = lib()
        self._h = C.c_void_p()
        self.device = device
        self.workspace = None
        self.stream = None
        if static:
            import torch
            if not torch.cuda.is_available():
                raise RuntimeError("no GPU visible: the engine runs only on the device")
            self.stream = stream if stream is not None else torch.cuda.current_stream(device)
            st = L.xl_context_create_static(device, C.c_void_p(self.stream.cuda_stream), C.byref(self._h))
            if st != XL_OK:
                raise XlError(st, "xl_context_create_static failed")
        elif device >= 0:
            import torch
            if not torch.cuda.is_available():
                raise RuntimeError("no GPU visible: the engine runs only on the device")
            self.workspace = torch.empty(workspace_bytes, dtype=torch.uint8, device=f"cuda:{device}")
            self.stream = stream if stream is not None else torch.cuda.current_stream(device)
            st = L.xl_context_create(device, C.c_void_p(self.stream.cuda_stream),
                                     C.c_void_p(self.workspace.data_ptr()), workspace_bytes,
                                     C.byref(self._h))
        else:
            st = L.xl_context_create(-1, None, None, 0, C.byref(self._h))
        if st != XL_OK:
            raise XlError(st, "xl_context_create failed")
        self.relations = {}
        self._programs = []

    def _check(self, st: int):
        if st != XL_OK:
            raise XlError(st, lib().xl_last_error(self._h).decode())

    def set_option(self, key: str, value: int):
        self._check(lib().xl_context_set_option(self._h, key.encode(), int(value)))

    def relation(self, name: str, types, max_rows: int = 0) -> "Relation":
        arr = (C.c_int * len(types))(*[_TYPES[t] for t in types])
        h = C.c_void_p()
        self._check(lib().xl_relation_create(self._h, name.encode(), len(types), arr, max_rows,
                                             C.byref(h)))
        r = Relation(self, h, name, tuple(types))
        self.relations[name] = r
        return r

    def compile(self, text: str) -> "Program":
        h = C.c_void_p()
        self._check(lib().xl_rule_compile(self._h, text.encode(), C.byref(h)))
        p = Program(self, h)
        self._programs.append(p)
        return p

    def close(self):
        if self._h:
            lib().xl_context_destroy(self._h)
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Relation:
    def __init__(self, ctx: Context, h, name: str, types):
        self.ctx, self._h, self.name, self.types = ctx, h, name, types

    def load(self, cols):
        """Load column arrays (numpy arrays, or torch tensors on the context's device)."""
        import torch
        n = len(cols[0]) if len(cols) else 0
        on_dev = isinstance(cols[0], torch.Tensor) and cols[0].is_cuda
        keep = []
        ptrs = (C.c_void_p * len(self.types))()
        for j, (t, c) in enumerate(zip(self.types, cols)):
            if on_dev:
                c = c.contiguous()
                want = _torch_dtype(t)
                # bool columns also take raw bytes (uint8), checked by the library
                if c.dtype != want and not (t == "bool" and c.dtype == torch.uint8):
                    raise TypeError(f"column {j} of {self.name} must be {want}")
                ptrs[j] = c.data_ptr()
            else:
                if t == "bool" and getattr(c, "dtype", None) == np.uint8:
                    c = np.ascontiguousarray(c)
                else:
                    c = np.ascontiguousarray(c, dtype=_NP[t])
                ptrs[j] = c.ctypes.data
            keep.append(c)
        self.ctx._check(lib().xl_relation_load(self._h, ptrs, n, 1 if on_dev else 0))

    def clear(self):
        self.ctx._check(lib().xl_relation_clear(self._h))

    def size(self) -> int:
        n = C.c_int64()
        self.ctx._check(lib().xl_relation_size(self._h, C.byref(n)))
        return n.value

    def read(self):
        """Rows in canonical order as numpy arrays (one per column)."""
        n = self.size()
        out = [np.empty(n, _NP[t]) for t in self.types]
        ptrs = (C.c_void_p * len(self.types))(*[o.ctypes.data for o in out])
        got = C.c_int64()
        self.ctx._check(lib().xl_relation_read(self._h, ptrs, n, C.byref(got), 0))
        return out

    def read_device(self):
        """Rows in canonical order as torch tensors on the context's device."""
        import torch
        n = self.size()
        dev = f"cuda:{self.ctx.device}"
        out = [torch.empty(max(n, 1), dtype=_torch_dtype(t), device=dev) for t in self.types]
        ptrs = (C.c_void_p * len(self.types))(*[o.data_ptr() for o in out])
        got = C.c_int64()
        self.ctx._check(lib().xl_relation_read(self._h, ptrs, n, C.byref(got), 1))
        return [o[:n] for o in out]


class Program:
    def __init__(self, ctx: Context, h):
        self.ctx, self._h = ctx, h

    def explain(self) -> str:
        need = C.c_size_t()
        lib().xl_program_explain(self._h, None, 0, C.byref(need))
        buf = C.create_string_buffer(need.value)
        lib().xl_program_explain(self._h, buf, need.value, C.byref(need))
        return buf.value.decode()

    def run(self, max_iterations: int = 10_000) -> dict:
        st = xl_fixpoint_stats()
        self.ctx._check(lib().xl_fixpoint_run(self._h, max_iterations, C.byref(st)))
        return st.as_dict()

    def run_status(self, max_iterations: int = 10_000):
        """Like run() but returns (status name, stats) instead of raising."""
        st = xl_fixpoint_stats()
        s = lib().xl_fixpoint_run(self._h, max_iterations, C.byref(st))
        return STATUS[s], st.as_dict()
