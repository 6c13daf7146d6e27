"""GETT dense tensor contraction on AMD Instinct MI355X (gfx950).

Python binding of ``lib/libgett.so`` (ctypes).  The functions below carry the
names of the C interface in ``include/gett.h`` and only marshal arguments;
every step of the contraction runs in the library's HIP kernels.  torch is
used for device memory and streams only.

    import torch, paper_1607_00145_amd as gett
    p = gett.Plan("C[a,b,c] = A[a,k,c] * B[k,b]", C=c, A=a, B=b)
    p(a, b, c, alpha=1.0, beta=0.0)          # enqueued on torch's current stream
"""
from __future__ import annotations

import ctypes
import json
import os
import re
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
# GETT_LIBRARY may name another build of the same sources (the sanitizer
# build, lib/libgett_asan.so); there is no fallback when it is missing.
LIB_PATH = os.environ.get("GETT_LIBRARY") or os.path.join(_HERE, "lib", "libgett.so")

GETT_FLOAT32 = 0
GETT_FLOAT64 = 1
GETT_FLAG_NONE = 0
GETT_FLAG_NO_SWAP = 1
GETT_FLAG_SCALAR = 2
GETT_FLAG_NO_SPLIT = 4
GETT_FLAG_WHOLE_TILES = 8
GETT_FLAG_DETERMINISTIC = GETT_FLAG_WHOLE_TILES   # former name
GETT_MAX_RANK = 16
GETT_METHOD_GETT = 0
GETT_METHOD_TTGT = 1
GETT_METHOD_LOG = 2
GETT_SUCCESS = 0
GETT_ERROR_INVALID_VALUE = 1
GETT_ERROR_INVALID_INDICES = 2
GETT_ERROR_NOT_SUPPORTED = 3
GETT_ERROR_HIP = 4
GETT_ERROR_ALLOC = 5

STATUS = {0: "GETT_SUCCESS", 1: "GETT_ERROR_INVALID_VALUE", 2: "GETT_ERROR_INVALID_INDICES",
          3: "GETT_ERROR_NOT_SUPPORTED", 4: "GETT_ERROR_HIP", 5: "GETT_ERROR_ALLOC"}

_lib = None


class GettError(RuntimeError):
    def __init__(self, status: int, what: str = ""):
        name = STATUS.get(status, str(status))
        super().__init__(f"{what}: {name}" if what else name)
        self.status = status


def load_library() -> ctypes.CDLL:
    """Load libgett.so; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_1607_00145_amd.build` (hipcc, gfx950)")
    lib = ctypes.CDLL(LIB_PATH)
    i64p = ctypes.POINTER(ctypes.c_int64)
    lib.gett_plan.restype = ctypes.c_int
    lib.gett_plan.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_int,
                              ctypes.c_char_p, i64p, i64p,
                              ctypes.c_char_p, i64p, i64p,
                              ctypes.c_char_p, i64p, i64p, ctypes.c_uint32]
    lib.gett_contract.restype = ctypes.c_int
    lib.gett_contract.argtypes = [ctypes.c_void_p, ctypes.c_double, ctypes.c_void_p,
                                  ctypes.c_void_p, ctypes.c_double, ctypes.c_void_p,
                                  ctypes.c_void_p]
    lib.gett_contract_noalloc.restype = ctypes.c_int
    lib.gett_contract_noalloc.argtypes = lib.gett_contract.argtypes
    lib.gett_plan_tune.restype = ctypes.c_int
    lib.gett_plan_tune.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.gett_destroy.restype = ctypes.c_int
    lib.gett_destroy.argtypes = [ctypes.c_void_p]
    lib.gett_transpose.restype = ctypes.c_int
    lib.gett_transpose.argtypes = [ctypes.c_int, ctypes.c_int, i64p, i64p, i64p, ctypes.c_double,
                                   ctypes.c_void_p, ctypes.c_double, ctypes.c_void_p,
                                   ctypes.c_void_p]
    lib.gett_ttgt_plan.restype = ctypes.c_int
    lib.gett_ttgt_plan.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_int,
                                   ctypes.c_char_p, i64p, i64p,
                                   ctypes.c_char_p, i64p, i64p,
                                   ctypes.c_char_p, i64p, i64p, ctypes.c_int64]
    lib.gett_ttgt_workspace_size.restype = ctypes.c_int
    lib.gett_ttgt_workspace_size.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_uint64)]
    lib.gett_ttgt_contract.restype = ctypes.c_int
    lib.gett_ttgt_contract.argtypes = [ctypes.c_void_p, ctypes.c_double, ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_double, ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p]
    lib.gett_ttgt_destroy.restype = ctypes.c_int
    lib.gett_ttgt_destroy.argtypes = [ctypes.c_void_p]
    lib.gett_ttgt_describe.restype = ctypes.c_char_p
    lib.gett_ttgt_describe.argtypes = [ctypes.c_void_p]
    lib.gett_log_plan.restype = ctypes.c_int
    lib.gett_log_plan.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_int,
                                  ctypes.c_char_p, i64p, i64p,
                                  ctypes.c_char_p, i64p, i64p,
                                  ctypes.c_char_p, i64p, i64p]
    lib.gett_log_contract.restype = ctypes.c_int
    lib.gett_log_contract.argtypes = [ctypes.c_void_p, ctypes.c_double, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_double, ctypes.c_void_p,
                                      ctypes.c_void_p]
    lib.gett_log_destroy.restype = ctypes.c_int
    lib.gett_log_destroy.argtypes = [ctypes.c_void_p]
    lib.gett_log_describe.restype = ctypes.c_char_p
    lib.gett_log_describe.argtypes = [ctypes.c_void_p]
    lib.gett_select_plan.restype = ctypes.c_int
    lib.gett_select_plan.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_int,
                                     ctypes.c_char_p, i64p, i64p, ctypes.c_char_p, i64p, i64p,
                                     ctypes.c_char_p, i64p, i64p, ctypes.c_uint32,
                                     ctypes.c_int64]
    lib.gett_select_workspace_size.restype = ctypes.c_int
    lib.gett_select_workspace_size.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_uint64)]
    lib.gett_select_tune.restype = ctypes.c_int
    lib.gett_select_tune.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                     ctypes.c_uint64, ctypes.c_void_p]
    lib.gett_select_force.restype = ctypes.c_int
    lib.gett_select_force.argtypes = [ctypes.c_void_p, ctypes.c_int]
    lib.gett_select_method.restype = ctypes.c_int
    lib.gett_select_method.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int)]
    lib.gett_select_contract.restype = ctypes.c_int
    lib.gett_select_contract.argtypes = [ctypes.c_void_p, ctypes.c_double, ctypes.c_void_p,
                                         ctypes.c_void_p, ctypes.c_double, ctypes.c_void_p,
                                         ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p]
    lib.gett_select_destroy.restype = ctypes.c_int
    lib.gett_select_destroy.argtypes = [ctypes.c_void_p]
    lib.gett_select_describe.restype = ctypes.c_char_p
    lib.gett_select_describe.argtypes = [ctypes.c_void_p]
    lib.gett_status_string.restype = ctypes.c_char_p
    lib.gett_status_string.argtypes = [ctypes.c_int]
    lib.gett_plan_describe.restype = ctypes.c_char_p
    lib.gett_plan_describe.argtypes = [ctypes.c_void_p]
    _lib = lib
    return lib


def _arr(values: Optional[Sequence[int]]):
    if values is None:
        return None
    vals = [int(v) for v in values]
    return (ctypes.c_int64 * max(1, len(vals)))(*vals)


# ----------------------------------------------------------- C interface ---

def gett_plan(dtype: int, modes_C: str, extent_C, stride_C, modes_A: str, extent_A, stride_A,
              modes_B: str, extent_B, stride_B, flags: int = 0):
    """Returns (status, plan handle or None).  Strides may be None (Fortran layout)."""
    lib = load_library()
    h = ctypes.c_void_p()
    st = lib.gett_plan(ctypes.byref(h), int(dtype),
                       modes_C.encode(), _arr(extent_C), _arr(stride_C),
                       modes_A.encode(), _arr(extent_A), _arr(stride_A),
                       modes_B.encode(), _arr(extent_B), _arr(stride_B), int(flags))
    return st, (h.value if st == 0 else None)


def gett_contract(plan, alpha: float, A: int, B: int, beta: float, C: int, stream: int = 0) -> int:
    """Device pointers as integers; stream as a hipStream_t integer (0 = default)."""
    return load_library().gett_contract(plan, float(alpha), A or None, B or None, float(beta),
                                        C or None, stream or None)


def gett_contract_noalloc(plan, alpha: float, A: int, B: int, beta: float, C: int,
                          stream: int = 0) -> int:
    """gett_contract with the partial-tile workspace taken from the library's
    fixed static buffer (no device allocation).  Arguments as gett_contract."""
    return load_library().gett_contract_noalloc(plan, float(alpha), A or None, B or None,
                                                float(beta), C or None, stream or None)


def gett_plan_tune(plan, max_candidates: int, A: int, B: int, C: int, stream: int = 0) -> int:
    """Times the plan's best `max_candidates` candidates on (A, B, C) and keeps the
    fastest; C is overwritten.  Device pointers and stream as integers."""
    return load_library().gett_plan_tune(plan, int(max_candidates), A or None, B or None,
                                         C or None, stream or None)


def gett_destroy(plan) -> int:
    return load_library().gett_destroy(plan)


def gett_transpose(dtype: int, extent, stride_in, stride_out, alpha: float, src: int,
                   beta: float, dst: int, stream: int = 0) -> int:
    """Eq. 4 over the iteration space `extent`; the permutation is carried by
    the output strides.  Device pointers and stream as integers."""
    return load_library().gett_transpose(int(dtype), len(extent), _arr(extent), _arr(stride_in),
                                         _arr(stride_out), float(alpha), src or None,
                                         float(beta), dst or None, stream or None)


def gett_ttgt_plan(dtype: int, modes_C: str, extent_C, stride_C, modes_A: str, extent_A,
                   stride_A, modes_B: str, extent_B, stride_B, max_workspace_bytes: int = -1):
    """Returns (status, TTGT plan handle or None)."""
    lib = load_library()
    h = ctypes.c_void_p()
    st = lib.gett_ttgt_plan(ctypes.byref(h), int(dtype),
                            modes_C.encode(), _arr(extent_C), _arr(stride_C),
                            modes_A.encode(), _arr(extent_A), _arr(stride_A),
                            modes_B.encode(), _arr(extent_B), _arr(stride_B),
                            int(max_workspace_bytes))
    return st, (h.value if st == 0 else None)


def gett_ttgt_workspace_size(plan):
    """Returns (status, bytes)."""
    n = ctypes.c_uint64()
    st = load_library().gett_ttgt_workspace_size(plan, ctypes.byref(n))
    return st, int(n.value)


def gett_ttgt_contract(plan, alpha: float, A: int, B: int, beta: float, C: int, workspace: int,
                       workspace_bytes: int, stream: int = 0) -> int:
    return load_library().gett_ttgt_contract(plan, float(alpha), A or None, B or None,
                                             float(beta), C or None, workspace or None,
                                             int(workspace_bytes), stream or None)


def gett_ttgt_destroy(plan) -> int:
    return load_library().gett_ttgt_destroy(plan)


def gett_ttgt_describe(plan) -> str:
    return load_library().gett_ttgt_describe(plan).decode()


def gett_log_plan(dtype: int, modes_C: str, extent_C, stride_C, modes_A: str, extent_A,
                  stride_A, modes_B: str, extent_B, stride_B):
    """Returns (status, LoG plan handle or None); status 3 when LoG does not apply."""
    lib = load_library()
    h = ctypes.c_void_p()
    st = lib.gett_log_plan(ctypes.byref(h), int(dtype),
                           modes_C.encode(), _arr(extent_C), _arr(stride_C),
                           modes_A.encode(), _arr(extent_A), _arr(stride_A),
                           modes_B.encode(), _arr(extent_B), _arr(stride_B))
    return st, (h.value if st == 0 else None)


def gett_log_contract(plan, alpha: float, A: int, B: int, beta: float, C: int,
                      stream: int = 0) -> int:
    return load_library().gett_log_contract(plan, float(alpha), A or None, B or None,
                                            float(beta), C or None, stream or None)


def gett_log_destroy(plan) -> int:
    return load_library().gett_log_destroy(plan)


def gett_log_describe(plan) -> str:
    return load_library().gett_log_describe(plan).decode()


def gett_select_plan(dtype: int, modes_C: str, extent_C, stride_C, modes_A: str, extent_A,
                     stride_A, modes_B: str, extent_B, stride_B, flags: int = 0,
                     max_workspace_bytes: int = -1):
    """Returns (status, selection plan handle or None)."""
    lib = load_library()
    h = ctypes.c_void_p()
    st = lib.gett_select_plan(ctypes.byref(h), int(dtype),
                              modes_C.encode(), _arr(extent_C), _arr(stride_C),
                              modes_A.encode(), _arr(extent_A), _arr(stride_A),
                              modes_B.encode(), _arr(extent_B), _arr(stride_B),
                              int(flags), int(max_workspace_bytes))
    return st, (h.value if st == 0 else None)


def gett_select_workspace_size(plan):
    """Returns (status, bytes)."""
    n = ctypes.c_uint64()
    st = load_library().gett_select_workspace_size(plan, ctypes.byref(n))
    return st, int(n.value)


def gett_select_tune(plan, max_candidates: int, A: int, B: int, C: int, workspace: int,
                     workspace_bytes: int, stream: int = 0) -> int:
    return load_library().gett_select_tune(plan, int(max_candidates), A or None, B or None,
                                           C or None, workspace or None, int(workspace_bytes),
                                           stream or None)


def gett_select_force(plan, method: int) -> int:
    return load_library().gett_select_force(plan, int(method))


def gett_select_method(plan):
    """Returns (status, method)."""
    m = ctypes.c_int()
    st = load_library().gett_select_method(plan, ctypes.byref(m))
    return st, int(m.value)


def gett_select_contract(plan, alpha: float, A: int, B: int, beta: float, C: int, workspace: int,
                         workspace_bytes: int, stream: int = 0) -> int:
    return load_library().gett_select_contract(plan, float(alpha), A or None, B or None,
                                               float(beta), C or None, workspace or None,
                                               int(workspace_bytes), stream or None)


def gett_select_destroy(plan) -> int:
    return load_library().gett_select_destroy(plan)


def gett_select_describe(plan) -> str:
    return load_library().gett_select_describe(plan).decode()


def gett_status_string(status: int) -> str:
    return load_library().gett_status_string(int(status)).decode()


def gett_plan_describe(plan) -> str:
    return load_library().gett_plan_describe(plan).decode()


# ------------------------------------------------------ torch convenience ---

_EXPR = re.compile(r"^\s*(\w+)\s*\[([^\]]*)\]\s*=\s*(\w+)\s*\[([^\]]*)\]\s*\*\s*(\w+)\s*\[([^\]]*)\]\s*$")


def parse_expression(expr: str):
    """'C[a,b,i,j] = A[i,m,a] * B[m,j,b]' (the input format of Listing 9) ->
    (modes_C, modes_A, modes_B) as comma-separated strings."""
    m = _EXPR.match(expr)
    if not m:
        raise ValueError(f"cannot parse contraction {expr!r}")
    norm = lambda s: ",".join(x.strip() for x in s.split(",") if x.strip()) + \
        ("," if len([x for x in s.split(",") if x.strip()]) == 1 else "")
    return norm(m.group(2)), norm(m.group(4)), norm(m.group(6))


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return GETT_FLOAT32
    if t.dtype == torch.float64:
        return GETT_FLOAT64
    raise TypeError(f"unsupported dtype {t.dtype}: float32 or float64 only")


class Plan:
    """A plan bound to the shapes and strides of given torch tensors."""

    def __init__(self, expr_or_modes, C, A, B, flags: int = 0):
        if isinstance(expr_or_modes, str):
            mc, ma, mb = parse_expression(expr_or_modes)
        else:
            mc, ma, mb = expr_or_modes
        self.modes = (mc, ma, mb)
        self.dtype = _dtype_code(C)
        if _dtype_code(A) != self.dtype or _dtype_code(B) != self.dtype:
            raise TypeError("A, B and C must have one dtype")
        self.sig = tuple((tuple(t.shape), tuple(t.stride())) for t in (C, A, B))
        st, h = gett_plan(self.dtype, mc, list(C.shape), list(C.stride()),
                          ma, list(A.shape), list(A.stride()),
                          mb, list(B.shape), list(B.stride()), flags)
        if st != 0:
            raise GettError(st, "gett_plan")
        self._h = h

    def describe(self) -> dict:
        return json.loads(gett_plan_describe(self._h))

    def __call__(self, A, B, C, alpha: float = 1.0, beta: float = 0.0, stream=None):
        import torch
        for name, t in (("A", A), ("B", B), ("C", C)):
            if not t.is_cuda:
                raise ValueError(f"{name} must be a device tensor")
        if tuple((tuple(t.shape), tuple(t.stride())) for t in (C, A, B)) != self.sig:
            raise ValueError("tensor shapes/strides differ from the plan's")
        s = stream if stream is not None else torch.cuda.current_stream()
        st = gett_contract(self._h, alpha, A.data_ptr(), B.data_ptr(), beta, C.data_ptr(),
                           s.cuda_stream)
        if st != 0:
            raise GettError(st, "gett_contract")
        return C

    def tune(self, A, B, C, max_candidates: int = 16, stream=None):
        """Runs the best `max_candidates` kernels of the performance model's ranking
        on these tensors and keeps the fastest (C is overwritten)."""
        import torch
        for name, t in (("A", A), ("B", B), ("C", C)):
            if not t.is_cuda:
                raise ValueError(f"{name} must be a device tensor")
        if tuple((tuple(t.shape), tuple(t.stride())) for t in (C, A, B)) != self.sig:
            raise ValueError("tensor shapes/strides differ from the plan's")
        s = stream if stream is not None else torch.cuda.current_stream()
        st = gett_plan_tune(self._h, max_candidates, A.data_ptr(), B.data_ptr(), C.data_ptr(),
                            s.cuda_stream)
        if st != 0:
            raise GettError(st, "gett_plan_tune")
        return self.describe()

    def close(self):
        if getattr(self, "_h", None):
            gett_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def contract(expr: str, A, B, C=None, alpha: float = 1.0, beta: float = 0.0, out_shape=None):
    """One-shot contraction on torch device tensors.  When C is None a new
    column-major C is allocated (beta must then be 0)."""
    import torch
    mc, ma, mb = parse_expression(expr)
    if C is None:
        if beta != 0:
            raise ValueError("beta != 0 needs C")
        ext = {}
        for modes, t in ((ma, A), (mb, B)):
            for n, s in zip([x for x in modes.split(",") if x], t.shape):
                ext[n] = s
        shape = [ext[n] for n in mc.split(",") if n]
        C = torch.empty(list(reversed(shape)), dtype=A.dtype, device=A.device).permute(
            *reversed(range(len(shape)))) if shape else torch.empty((), dtype=A.dtype,
                                                                    device=A.device)
    p = Plan((mc, ma, mb), C, A, B)
    p(A, B, C, alpha, beta)
    return C
