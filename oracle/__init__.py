"""Oracle for the GETT contraction C <- alpha * A * B + beta * C.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark import this package.  It shares no code with the
GPU library (``paper_1607_00145_amd``) and imports nothing from it.

The arithmetic lives in ``gett_oracle.c`` (plain C, fp64, the definition of
Eq. 3 evaluated as the naive loop nest of Listing 3, and the transposition of
Eq. 4); this module only builds that file with gcc and marshals numpy arrays
into it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gett_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_LIB_ASAN = os.path.join(_HERE, "liboracle_asan.so")
_lib = None

ERRORS = {0: "ok", -1: "invalid value", -2: "parse error", -3: "invalid indices", -4: "point out of range"}


class OracleError(RuntimeError):
    def __init__(self, code: int):
        super().__init__(f"oracle: {ERRORS.get(code, code)}")
        self.code = code


def build(force: bool = True, sanitize: bool = False) -> str:
    """Compile gett_oracle.c into liboracle.so (gcc -O2 -fopenmp, no fast-math),
    or, sanitize, into liboracle_asan.so with AddressSanitizer and
    UndefinedBehaviorSanitizer (clang, whose runtime the sanitized library
    shares; tests/run_sanitized.sh)."""
    out = _LIB_ASAN if sanitize else _LIB
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(_SRC):
        tmp = out + f".tmp{os.getpid()}"
        if sanitize:
            cmd = ["/opt/rocm/llvm/bin/clang", "-O1", "-g", "-fsanitize=address,undefined",
                   "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-fopenmp",
                   "-fPIC", "-shared", "-std=c99", "-Wall", "-o", tmp, _SRC, "-lm"]
        else:
            cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-Wall", "-o", tmp,
                   _SRC, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, out)
    return out


def _open(path: str):
    """ctypes handle of a built oracle library with its signatures set."""
    lib = ctypes.CDLL(path)
    i64p = ctypes.POINTER(ctypes.c_int64)
    lib.oracle_contract.restype = ctypes.c_int
    lib.oracle_contract.argtypes = [
        ctypes.c_int,
        ctypes.c_char_p, i64p, i64p,
        ctypes.c_char_p, i64p, i64p,
        ctypes.c_char_p, i64p, i64p,
        ctypes.c_double, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_double,
        ctypes.c_void_p, ctypes.c_int64, i64p,
        ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double), ctypes.c_int]
    lib.oracle_max_threads.restype = ctypes.c_int
    lib.oracle_transpose.restype = ctypes.c_int
    lib.oracle_transpose.argtypes = [
        ctypes.c_int, ctypes.c_int, i64p, i64p, i64p, ctypes.c_double, ctypes.c_void_p,
        ctypes.c_double, ctypes.c_void_p, i64p,
        ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
    return lib


def _load():
    global _lib
    if _lib is None:
        # ORACLE_LIBRARY may name another build of gett_oracle.c (the sanitizer build)
        path = os.environ.get("ORACLE_LIBRARY")
        if not path:
            path = build(force=False)
        _lib = _open(path)
    return _lib


class using_library:
    """Context manager: route every call to another build of the oracle's
    source (the mutation tests build copies with a planted mistake and check
    that the pins catch it)."""

    def __init__(self, path: str):
        self.path = path

    def __enter__(self):
        global _lib
        self.saved = _load()
        _lib = _open(self.path)
        return self

    def __exit__(self, *exc):
        global _lib
        _lib = self.saved
        return False


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def _i64(seq):
    arr = (ctypes.c_int64 * max(1, len(seq)))(*[int(v) for v in seq])
    return arr


def _view(arr: np.ndarray, dtype):
    """Base pointer, extents and element strides of an ndarray view."""
    if arr.dtype != dtype:
        raise TypeError(f"expected {dtype}, got {arr.dtype}")
    item = arr.itemsize
    if any(s % item for s in arr.strides):
        raise ValueError("strides must be whole elements")
    if any(s < 0 for s in arr.strides):
        raise ValueError("negative strides are not supported")
    return arr.ctypes.data, list(arr.shape), [s // item for s in arr.strides]


@dataclass
class Result:
    out64: np.ndarray   # alpha * t + beta * C_in, unrounded fp64
    den64: np.ndarray   # |alpha| * sum |a||b| + |beta| * |C_in|


def contract(modes_C: str, modes_A: str, modes_B: str, A: np.ndarray, B: np.ndarray,
             alpha: float = 1.0, beta: float = 0.0, C: np.ndarray | None = None,
             shape_C=None, points=None, nthreads: int = 0) -> Result:
    """Evaluate the contraction with the oracle.

    ``A``, ``B`` and ``C`` are numpy arrays whose axes follow the mode strings
    (any positive strides).  ``C`` is read only when ``beta != 0``; without it
    ``shape_C`` gives C's extents.  ``points`` are positions in C's
    column-major logical order (first mode fastest); None means all of C,
    returned with C's shape in Fortran order.
    """
    if A.dtype not in (np.float32, np.float64):
        raise TypeError("float32 or float64 only")
    dt = A.dtype
    dcode = 0 if dt == np.float32 else 1
    pa, ea, sa = _view(A, dt)
    pb, eb, sb = _view(B, dt)
    if C is not None:
        pc, ec, sc = _view(C, dt)
    else:
        if shape_C is None:
            raise ValueError("shape_C is needed when C is not given")
        ec = [int(v) for v in shape_C]
        sc = list(np.cumprod([1] + ec[:-1])) if ec else []
        pc = None
    size_c = int(np.prod(ec)) if ec else 1
    if points is None:
        npts = size_c
        pts_ptr = None
    else:
        pts = np.ascontiguousarray(points, dtype=np.int64)
        npts = int(pts.size)
        pts_ptr = pts.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))
    out = np.empty(max(npts, 1), dtype=np.float64)
    den = np.empty(max(npts, 1), dtype=np.float64)
    rc = _load().oracle_contract(
        dcode,
        modes_C.encode(), _i64(ec), _i64(sc),
        modes_A.encode(), _i64(ea), _i64(sa),
        modes_B.encode(), _i64(eb), _i64(sb),
        float(alpha), pa, pb, float(beta), pc if beta != 0 else None,
        npts, pts_ptr,
        out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
        den.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), int(nthreads))
    if rc != 0:
        raise OracleError(rc)
    out, den = out[:npts], den[:npts]
    if points is None:
        out = out.reshape(ec, order="F") if ec else out.reshape(())
        den = den.reshape(ec, order="F") if ec else den.reshape(())
    return Result(out, den)


def transpose(A: np.ndarray, perm, alpha: float = 1.0, beta: float = 0.0,
              B: np.ndarray | None = None) -> Result:
    """Eq. 4: B[Pi(i)] <- alpha * A[i] + beta * B[Pi(i)], where output mode j is
    input mode perm[j].  ``A`` and ``B`` may have any positive strides; ``B``
    (shape A.shape[perm]) is read only when beta != 0.  Returns fp64 arrays
    of the output's shape."""
    if A.dtype not in (np.float32, np.float64):
        raise TypeError("float32 or float64 only")
    dt = A.dtype
    perm = [int(p) for p in perm]
    if len(perm) != A.ndim:
        raise ValueError("perm must name every mode of A once")
    pa, ea, sa = _view(A, dt)
    out_shape = [ea[p] for p in perm]
    pb, sb = None, None
    if beta != 0:
        if B is None or list(B.shape) != out_shape:
            raise ValueError("B of shape A.shape[perm] is needed when beta != 0")
        pb, _, sb = _view(B, dt)
    n = int(np.prod(out_shape)) if out_shape else 1
    out = np.zeros(max(n, 1), dtype=np.float64)
    den = np.zeros(max(n, 1), dtype=np.float64)
    rc = _load().oracle_transpose(
        0 if dt == np.float32 else 1, len(ea), _i64(ea), _i64(sa), _i64(perm), float(alpha), pa,
        float(beta), pb, _i64(sb) if sb is not None else None,
        out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
        den.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    if rc != 0:
        raise OracleError(rc)
    shape = out_shape if out_shape else ()
    return Result(out[:n].reshape(shape, order="F"), den[:n].reshape(shape, order="F"))


def rel_error(got, ref: Result) -> float:
    """max |got - out64| / den64, where den64 == 0 demands equality.

    This is the error measure of the parity bar: the difference from the
    unrounded fp64 result, relative to the sum of |a||b| over the contracted
    indices (scaled by |alpha|) plus |beta||C_in|.
    """
    got = np.asarray(got, dtype=np.float64).reshape(-1)
    out = np.asarray(ref.out64, dtype=np.float64).reshape(-1)
    den = np.asarray(ref.den64, dtype=np.float64).reshape(-1)
    if got.size != out.size or den.size != out.size:
        raise ValueError(f"sizes differ: got {got.size}, out64 {out.size}, den64 {den.size}")
    # den64 is a sum of magnitudes: a negative or NaN value means a broken
    # reference, and dividing by it would let any result pass
    if np.any(~(den >= 0)):
        raise ValueError("den64 must be >= 0 everywhere")
    if got.size == 0:
        return 0.0
    diff = np.abs(got - out)
    zero = den == 0
    if np.any(zero & (diff != 0)):
        return float("inf")
    if np.any(~np.isfinite(got)):
        return float("inf")
    with np.errstate(invalid="ignore", divide="ignore"):
        r = np.where(zero, 0.0, diff / np.where(zero, 1.0, den))
    return float(r.max())
