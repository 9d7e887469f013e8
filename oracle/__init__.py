"""CPU oracle for the tiled GEMM C = A B -- TEST INFRASTRUCTURE ONLY.

The arithmetic lives in ``oracle_gemm.c``: the plain fp64 triple loop that
defines the matrix product (paper, Background, "General Matrix
Multiplication"), over operands given as raw fp16 / bf16 bit patterns that it
decodes itself.  This module only builds that C file with gcc and marshals
numpy arrays into it.

Only the test suite, ``__graft_entry__.smoke()`` and the benchmark's
``cpu_baseline`` leg may import this package.  It shares no code with the GPU
library and the GPU library never calls it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import tempfile

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "oracle_gemm.c")
LIBRARY = os.path.join(_HERE, "liboracle.so")

DTYPES = {"f16": 0, "bf16": 1}

_lib = None


def build(out_path: str = LIBRARY, defines: tuple[str, ...] = ()) -> str:
    """Compile ``oracle_gemm.c`` into a shared library with gcc and OpenMP.

    ``defines`` adds ``-D`` macros; the pin self-test uses it to build copies
    with a planted mistake into a temporary directory.
    """
    tmp = out_path + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-fno-fast-math",
           "-ffp-contract=off", SOURCE, "-o", tmp, "-lm"]
    cmd[1:1] = ["-D" + d for d in defines]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out_path)
    return out_path


def _bind(lib: ctypes.CDLL) -> ctypes.CDLL:
    i64, i32 = ctypes.c_int64, ctypes.c_int
    p = ctypes.c_void_p
    lib.oracle_gemm_rows.argtypes = [i64, i64, i64, p, p, i32, i64, p, p, p, i32]
    lib.oracle_gemm_rows.restype = i32
    lib.oracle_gemm.argtypes = [i64, i64, i64, p, p, i32, p, p, i32]
    lib.oracle_gemm.restype = i32
    lib.oracle_decode.argtypes = [p, i64, i32, p]
    lib.oracle_decode.restype = i32
    lib.oracle_max_threads.argtypes = []
    lib.oracle_max_threads.restype = i32
    return lib


def load(path: str | None = None) -> ctypes.CDLL:
    """Load the built oracle (building it first only if no library exists)."""
    global _lib
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(LIBRARY):
            build()
        _lib = _bind(ctypes.CDLL(LIBRARY))
    return _lib


def _u16(x) -> np.ndarray:
    a = np.ascontiguousarray(x)
    if a.dtype != np.uint16:
        a = np.ascontiguousarray(a.view(np.uint16)) if a.dtype.itemsize == 2 else None
    if a is None:
        raise TypeError("operands must be 16-bit bit patterns")
    return a


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def decode(bits, dtype: str, lib: ctypes.CDLL | None = None) -> np.ndarray:
    """Decode fp16 / bf16 bit patterns to float64 (same shape)."""
    lib = lib or load()
    b = _u16(bits)
    out = np.empty(b.shape, dtype=np.float64)
    rc = lib.oracle_decode(_ptr(b), b.size, DTYPES[dtype], _ptr(out))
    if rc != 0:
        raise ValueError("oracle_decode failed (%d)" % rc)
    return out


def gemm_rows(A_bits, B_bits, dtype: str, rows, nthreads: int = 0,
              lib: ctypes.CDLL | None = None, with_abs: bool = True):
    """Rows ``rows`` of C = A B and of |A| |B|, both float64 (len(rows) x N)."""
    lib = lib or load()
    A = _u16(A_bits)
    B = _u16(B_bits)
    if A.ndim != 2 or B.ndim != 2 or A.shape[1] != B.shape[0]:
        raise ValueError("shape mismatch: A %s, B %s" % (A.shape, B.shape))
    M, K = A.shape
    N = B.shape[1]
    r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    C = np.empty((r.size, N), dtype=np.float64)
    S = np.empty((r.size, N), dtype=np.float64) if with_abs else None
    rc = lib.oracle_gemm_rows(M, N, K, _ptr(A), _ptr(B), DTYPES[dtype], r.size, _ptr(r),
                              _ptr(C), _ptr(S) if S is not None else None, nthreads)
    if rc != 0:
        raise ValueError("oracle_gemm_rows failed (%d)" % rc)
    return C, S


def gemm(A_bits, B_bits, dtype: str, nthreads: int = 0, lib: ctypes.CDLL | None = None,
         with_abs: bool = True):
    """C = A B and |A| |B| in float64 for all M rows."""
    A = _u16(A_bits)
    return gemm_rows(A, B_bits, dtype, np.arange(A.shape[0]), nthreads, lib, with_abs)


def max_threads(lib: ctypes.CDLL | None = None) -> int:
    return (lib or load()).oracle_max_threads()


def build_variant(defines: tuple[str, ...]) -> ctypes.CDLL:
    """Build and load a throw-away copy with extra macros (planted-mistake tests)."""
    d = tempfile.mkdtemp(prefix="oracle_variant_")
    path = os.path.join(d, "liboracle_variant.so")
    build(path, defines)
    return load(path)
