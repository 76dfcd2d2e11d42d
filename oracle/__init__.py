"""CPU oracle for 8-bit block-wise optimizers (test infrastructure only).

Plain C (``bq_oracle.c``) behind ctypes, operating on numpy arrays.  Only the
test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package; the product path never does.  It shares
no code with the HIP library.

Paper: Dettmers et al., "8-bit Optimizers via Block-wise Quantization".
  - codebooks: Section 2.3 (dynamic tree), Section 3.2 (unsigned dynamic)
  - nearest code: Eq. 3 / Eq. 4
  - block-wise quantize / dequantize: Section 3.1, Section 2.2
  - optimizer update: Eq. 1 (Momentum), Eq. 2 (Adam), AdamW (decoupled decay)
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bq_oracle.c")
# BQ_SANITIZE=1: the build with AddressSanitizer and UndefinedBehaviorSanitizer
# (clang, to share the ASan runtime of the sanitized library; no OpenMP)
SANITIZE = os.environ.get("BQ_SANITIZE") == "1"
_LIB = os.path.join(_HERE, "liboracle_san.so" if SANITIZE else "liboracle.so")

ADAM, ADAMW, MOMENTUM, ADAGRAD, LAMB, LARS = 0, 1, 2, 3, 4, 5
TWO_STATES = (0, 1, 4)
SIGNED, UNSIGNED = 0, 1


def build(sanitize: bool = None) -> str:
    """Compile the oracle with gcc (IEEE binary32, no contraction, OpenMP); with
    sanitize (default: BQ_SANITIZE=1), with clang under AddressSanitizer and
    UndefinedBehaviorSanitizer, single-threaded, to liboracle_san.so."""
    if sanitize is None:
        sanitize = SANITIZE
    if sanitize:
        rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
        out = os.path.join(_HERE, "liboracle_san.so")
        cmd = [os.path.join(rocm, "llvm", "bin", "clang"), "-O1", "-g", "-std=c11", "-fPIC",
               "-shared", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
               "-fno-omit-frame-pointer", "-ffp-contract=off", "-fno-fast-math",
               "-fvisibility=hidden", "-Wall", "-Wextra", "-o", out + ".tmp", _SRC, "-lm"]
    else:
        out = os.path.join(_HERE, "liboracle.so")
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
               "-ffp-contract=off", "-fno-fast-math", "-fvisibility=hidden",
               "-Wall", "-Wextra", "-o", out + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        P, I, I32, I64, F = (ctypes.c_void_p, ctypes.c_int, ctypes.c_int32,
                             ctypes.c_int64, ctypes.c_float)
        L.oracle_dynamic_codebook.argtypes = [I, P]
        L.oracle_dynamic_codebook.restype = I
        L.oracle_codebook.argtypes = [I, P]
        L.oracle_codebook.restype = I
        L.oracle_quantile_codebook.argtypes = [P, ctypes.c_int64, P]
        L.oracle_quantile_codebook.restype = I
        L.oracle_chunked_quantile_codebook.argtypes = [P, ctypes.c_int64, ctypes.c_int64, P]
        L.oracle_chunked_quantile_codebook.restype = I
        L.oracle_nearest_brute.argtypes = [P, F]
        L.oracle_nearest_brute.restype = I
        L.oracle_nearest_bsearch.argtypes = [P, F]
        L.oracle_nearest_bsearch.restype = I
        L.oracle_quantize_blockwise.argtypes = [P, P, I64, I32, P, P, I, I]
        L.oracle_quantize_blockwise.restype = None
        L.oracle_dequantize_blockwise.argtypes = [P, P, P, I64, I32, P, I]
        L.oracle_dequantize_blockwise.restype = None
        L.oracle_half_to_float.argtypes = [P, P, I64]
        L.oracle_half_to_float.restype = None
        L.oracle_step32.argtypes = [I, I64, P, P, I, P, P, F, F, F, F, F, I64, F]
        L.oracle_step32.restype = I
        L.oracle_step8.argtypes = [I, I32, I, I64, P, P, P, P, P, P, P, P,
                                   F, F, F, F, F, I64, I, F]
        L.oracle_step8.restype = I
        L.oracle_max_threads.argtypes = []
        L.oracle_max_threads.restype = I
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _check(a, dtype, name):
    if not (isinstance(a, np.ndarray) and a.dtype == dtype and a.flags.c_contiguous):
        raise TypeError(f"{name} must be a C-contiguous numpy {np.dtype(dtype).name} array")


def dynamic_codebook(kind: int) -> np.ndarray:
    out = np.empty(256, np.float32)
    if lib().oracle_dynamic_codebook(int(kind), out.ctypes.data) != 0:
        raise ValueError(f"unknown codebook kind {kind}")
    return out


def codebook(kind: int) -> np.ndarray:
    """Fixed maps: 0/1 dynamic, 2/3 inverse dynamic, 4/5 linear (signed/unsigned)."""
    out = np.empty(256, np.float32)
    if lib().oracle_codebook(int(kind), out.ctypes.data) != 0:
        raise ValueError(f"unknown codebook kind {kind}")
    return out


def quantile_codebook(sample) -> np.ndarray:
    """Quantile map (App. F.2) of a host sample."""
    x = np.ascontiguousarray(sample, dtype=np.float32).ravel()
    out = np.empty(256, np.float32)
    if lib().oracle_quantile_codebook(x.ctypes.data, x.size, out.ctypes.data) != 0:
        raise ValueError("quantile map: empty or non-finite sample, or all-zero map")
    return out


def chunked_quantile_codebook(sample, chunk: int = 4096) -> np.ndarray:
    """Quantile map from the length-weighted average of per-chunk quantiles (App. G),
    summed in chunk order."""
    x = np.ascontiguousarray(sample, dtype=np.float32).ravel()
    out = np.empty(256, np.float32)
    if lib().oracle_chunked_quantile_codebook(x.ctypes.data, x.size, int(chunk),
                                              out.ctypes.data) != 0:
        raise ValueError("chunked quantile map: empty or non-finite sample")
    return out


def nearest_brute(qmap: np.ndarray, y: float) -> int:
    _check(qmap, np.float32, "qmap")
    return lib().oracle_nearest_brute(qmap.ctypes.data, float(np.float32(y)))


def nearest_bsearch(qmap: np.ndarray, y: float) -> int:
    _check(qmap, np.float32, "qmap")
    return lib().oracle_nearest_bsearch(qmap.ctypes.data, float(np.float32(y)))


def quantize_blockwise(qmap, x, blocksize, brute=False, nthreads=0):
    _check(qmap, np.float32, "qmap")
    _check(x, np.float32, "x")
    n = x.size
    codes = np.empty(n, np.uint8)
    absmax = np.empty((n + blocksize - 1) // blocksize, np.float32)
    lib().oracle_quantize_blockwise(qmap.ctypes.data, x.ctypes.data, n, blocksize,
                                    codes.ctypes.data, absmax.ctypes.data,
                                    int(bool(brute)), int(nthreads))
    return codes, absmax


def dequantize_blockwise(qmap, codes, absmax, blocksize, nthreads=0):
    _check(qmap, np.float32, "qmap")
    _check(codes, np.uint8, "codes")
    _check(absmax, np.float32, "absmax")
    n = codes.size
    if absmax.size < (n + blocksize - 1) // blocksize:
        raise ValueError("absmax too short")
    out = np.empty(n, np.float32)
    lib().oracle_dequantize_blockwise(qmap.ctypes.data, codes.ctypes.data,
                                      absmax.ctypes.data, n, blocksize,
                                      out.ctypes.data, int(nthreads))
    return out


def half_to_float(h: np.ndarray) -> np.ndarray:
    h = np.ascontiguousarray(h).view(np.uint16)
    out = np.empty(h.size, np.float32)
    lib().oracle_half_to_float(h.ctypes.data, out.ctypes.data, h.size)
    return out


def _grad_kind(g):
    if g.dtype == np.float16:
        return 1
    if g.dtype == np.float32:
        return 0
    raise TypeError("grad must be float16 or float32")


def step32(opt, w, g, m, v, lr, beta1, beta2, eps, wd, step, trust=0.0):
    """Update w, m, v (fp32 states, quantization bypassed) in place.  trust is
    LARS's trust coefficient (unused by the other optimizers)."""
    _check(w, np.float32, "w")
    _check(m, np.float32, "m")
    if opt in TWO_STATES:
        _check(v, np.float32, "v")
    g = np.ascontiguousarray(g)
    rc = lib().oracle_step32(int(opt), w.size, w.ctypes.data, g.ctypes.data, _grad_kind(g),
                             m.ctypes.data, _ptr(v), lr, beta1, beta2, eps, wd, int(step),
                             float(trust))
    if rc != 0:
        raise ValueError("oracle_step32: bad argument")


def step8(opt, blocksize, w, g, c1, a1, q1, c2, a2, q2, lr, beta1, beta2, eps, wd,
          step, nthreads=0, trust=0.0):
    """One 8-bit step on one tensor; w, c1, a1, c2, a2 are updated in place."""
    _check(w, np.float32, "w")
    _check(c1, np.uint8, "c1")
    _check(a1, np.float32, "a1")
    _check(q1, np.float32, "q1")
    if opt in TWO_STATES:
        _check(c2, np.uint8, "c2")
        _check(a2, np.float32, "a2")
        _check(q2, np.float32, "q2")
    g = np.ascontiguousarray(g)
    rc = lib().oracle_step8(int(opt), int(blocksize), _grad_kind(g), w.size, w.ctypes.data,
                            g.ctypes.data, c1.ctypes.data, _ptr(c2), a1.ctypes.data,
                            _ptr(a2), q1.ctypes.data, _ptr(q2), lr, beta1, beta2, eps,
                            wd, int(step), int(nthreads), float(trust))
    if rc != 0:
        raise ValueError("oracle_step8: bad argument")


def max_threads() -> int:
    return lib().oracle_max_threads()
