"""Reference oracle -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU library never loads it and
shares no code with it: the two are compared, never combined.

Contents
--------
* ``conv_oracle.c`` -- plain fp64 seven-loop direct convolution (paper,
  Sec. 1 CNN equation and Listing 1, strides restored), built into
  ``liboracle.so`` with gcc and called through ctypes here.
* ``conv_lib`` -- the same definition evaluated by a library routine
  (PyTorch's CPU convolution in fp64), for comparing every output of the
  full-size workloads in seconds; pinned element by element to the loop nest
  above by the CPU tests.
* ``eq1`` -- the paper's data-movement cost, Eq. (1), its relaxed form
  Eq. (4), the Case 1a closed form and Table 1 (Sec. 2.1), written out in
  Python.

Inputs are passed as the exact stored values: float32 arrays, or bfloat16
bit patterns held in uint16 arrays; both are widened exactly to float64
before the fp64 arithmetic.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "conv_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile ``conv_oracle.c`` into ``liboracle.so`` (gcc, OpenMP).

    ``-ffp-contract=off`` keeps each multiply and add as written, so the
    oracle's arithmetic is exactly the loop nest in the source.
    """
    if not force and os.path.exists(_LIB):
        return _LIB
    tmp = _LIB + ".tmp"
    cmd = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
           "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build()
    lib = ctypes.CDLL(_LIB)
    i64 = ctypes.c_longlong
    dp = ctypes.POINTER(ctypes.c_double)
    lib.cnn_oracle_fwd.argtypes = [dp, dp, dp, dp] + [i64] * 9
    lib.cnn_oracle_fwd.restype = ctypes.c_int
    lib.cnn_oracle_points.argtypes = [dp, dp, ctypes.POINTER(i64), i64, dp, dp] + [i64] * 9
    lib.cnn_oracle_points.restype = ctypes.c_int
    lib.cnn_oracle_threads.argtypes = []
    lib.cnn_oracle_threads.restype = ctypes.c_int
    lib.cnn_oracle_set_threads.argtypes = [ctypes.c_int]
    lib.cnn_oracle_set_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def threads() -> int:
    """OpenMP threads the oracle uses (honours OMP_NUM_THREADS)."""
    return int(_load().cnn_oracle_threads())


def set_threads(n: int) -> int:
    """Use n OpenMP threads from now on (timing only; results do not depend
    on it).  Returns the previous count."""
    return int(_load().cnn_oracle_set_threads(int(n)))


def widen(x: np.ndarray) -> np.ndarray:
    """Exact float64 copy of stored input values.

    float32 / float64 arrays widen directly.  uint16 arrays are read as
    bfloat16 bit patterns: the 16 bits are the top half of an IEEE float32.
    """
    x = np.asarray(x)
    if x.dtype == np.uint16:
        f32 = (x.astype(np.uint32) << np.uint32(16)).view(np.float32)
        return f32.astype(np.float64)
    if x.dtype in (np.float32, np.float64):
        return x.astype(np.float64)
    raise TypeError(f"oracle: unsupported input dtype {x.dtype}")


def _dims(In, Ker, sw, sh):
    if In.ndim != 4 or Ker.ndim != 4:
        raise ValueError("oracle: In and Ker must be 4-d")
    Nb, Nc, Nx, Ny = In.shape
    Nk, Nc2, Nr, Ns = Ker.shape
    if Nc2 != Nc:
        raise ValueError("oracle: channel mismatch")
    if (Nx - Nr) % sw or (Ny - Ns) % sh or Nx < Nr or Ny < Ns:
        raise ValueError("oracle: In extent must be sigma*(N-1)+R (valid convolution)")
    Nw = (Nx - Nr) // sw + 1
    Nh = (Ny - Ns) // sh + 1
    return Nb, Nc, Nk, Nw, Nh, Nr, Ns


def _ptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def conv(In: np.ndarray, Ker: np.ndarray, sw: int = 1, sh: int = 1,
         with_abs: bool = False):
    """Full fp64 forward result Out[b][k][w][h] (and sum |In*Ker| if asked).

    ``In`` is [Nb][Nc][Nx][Ny], ``Ker`` is [Nk][Nc][Nr][Ns]; float32 or
    bfloat16 bits (uint16) or float64.
    """
    In64 = np.ascontiguousarray(widen(In))
    Ker64 = np.ascontiguousarray(widen(Ker))
    Nb, Nc, Nk, Nw, Nh, Nr, Ns = _dims(In64, Ker64, sw, sh)
    out = np.empty((Nb, Nk, Nw, Nh), dtype=np.float64)
    absv = np.empty_like(out) if with_abs else None
    rc = _load().cnn_oracle_fwd(_ptr(In64), _ptr(Ker64), _ptr(out),
                                _ptr(absv) if with_abs else None,
                                Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh)
    if rc != 0:
        raise ValueError(f"oracle: cnn_oracle_fwd returned {rc}")
    return (out, absv) if with_abs else out


def conv_points(In: np.ndarray, Ker: np.ndarray, idx: np.ndarray,
                sw: int = 1, sh: int = 1, with_abs: bool = False):
    """fp64 Out at the (b, k, w, h) rows of ``idx`` (shape [n, 4])."""
    In64 = np.ascontiguousarray(widen(In))
    Ker64 = np.ascontiguousarray(widen(Ker))
    Nb, Nc, Nk, Nw, Nh, Nr, Ns = _dims(In64, Ker64, sw, sh)
    idx = np.ascontiguousarray(np.asarray(idx, dtype=np.int64).reshape(-1, 4))
    n = idx.shape[0]
    out = np.empty(n, dtype=np.float64)
    absv = np.empty(n, dtype=np.float64) if with_abs else None
    rc = _load().cnn_oracle_points(
        _ptr(In64), _ptr(Ker64),
        idx.ctypes.data_as(ctypes.POINTER(ctypes.c_longlong)), n,
        _ptr(out), _ptr(absv) if with_abs else None,
        Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh)
    if rc != 0:
        raise ValueError(f"oracle: cnn_oracle_points returned {rc}")
    return (out, absv) if with_abs else out


def conv_lib(In: np.ndarray, Ker: np.ndarray, sw: int = 1, sh: int = 1,
             with_abs: bool = False):
    """The Sec. 1 CNN equation (valid convolution, strides sw, sh) through
    PyTorch's fp64 CPU convolution, which computes the same cross-correlation
    sum Out[b][k][w][h] = sum_{c,r,s} In[b][c][sw*w+r][sh*h+s] Ker[k][c][r][s]
    (no kernel flip).  The optional second result is sum |In * Ker|, the same
    routine on |In| and |Ker|.  Only the summation order differs from
    ``conv``; the CPU tests hold the two equal output by output."""
    import torch
    In64 = np.ascontiguousarray(widen(In))
    Ker64 = np.ascontiguousarray(widen(Ker))
    _dims(In64, Ker64, sw, sh)
    ti, tk = torch.from_numpy(In64), torch.from_numpy(Ker64)
    with torch.no_grad():
        out = torch.nn.functional.conv2d(ti, tk, stride=(sw, sh)).numpy()
        if not with_abs:
            return out
        absv = torch.nn.functional.conv2d(ti.abs(), tk.abs(), stride=(sw, sh)).numpy()
    return out, absv
