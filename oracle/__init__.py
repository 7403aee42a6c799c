"""kred oracle: fp64 CPU reference for the symbolic-matrix reductions.

TEST INFRASTRUCTURE ONLY.  The tests, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` call it to check and to time the GPU
library; the library itself never imports, links or runs anything here, and
this package shares no code with it.

The arithmetic lives in ``kred_oracle.c`` (plain C, fp64, OpenMP over rows);
this module builds it with gcc on first use, converts fp32 inputs to fp64 and
marshals arguments.  The block-sparse (cluster-wise) reductions of Sec. 3 are
composed here from those routines: each row cluster is reduced over its
gathered columns, and the gradients of the block-sparse Gaussian sum take the
same blocks (a row or column the pattern never pairs gets zero).  What each
routine computes follows Charlier et al.,
"Kernel Operations on the GPU, with Autodiff, without Memory Overflows"
(arXiv:2004.11127): Eq. (1) (Gaussian kernel sum), Eq. (2) with the
reductions of Sec. 2 (sum, log-sum-exp, arg-K-min), and the x-gradient of
Eq. (1) and its vector-Jacobian products (Sec. 2, "Backpropagation").  The C file's header lists the readings
taken where the paper is silent.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kred_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

GAUSS, LAPLACE, SQDIST, SINKHORN = 0, 1, 2, 4
_FORMULAS = {"gauss": GAUSS, "laplace": LAPLACE, "sqdist": SQDIST}

_dp = ctypes.POINTER(ctypes.c_double)
_i64p = ctypes.POINTER(ctypes.c_int64)


def build(force: bool = False) -> str:
    """Compile liboracle.so with gcc (-O2, OpenMP, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-fno-fast-math",
               "-ffp-contract=off", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


NATIVE_FLAGS = ["-O3", "-march=native"]
_native_path = None


def use_native() -> str:
    """Load a copy of the oracle compiled for this host's CPU, for the CPU baseline's timing.

    gcc -O3 -march=native, still with -fno-fast-math and -ffp-contract=off, so
    the arithmetic (and every result) is the portable build's.  It is built in a
    private temporary directory on the machine that runs it (a -march=native
    binary must not travel to another CPU) and replaces the portable build for
    the rest of the process.  Returns the compile command line.
    """
    import tempfile
    global _lib, _native_path
    with _lock:
        d = tempfile.mkdtemp(prefix="kred_oracle_native_")
        path = os.path.join(d, "liboracle_native.so")
        cmd = ["gcc"] + NATIVE_FLAGS + ["-fopenmp", "-fPIC", "-shared", "-fno-fast-math",
                                        "-ffp-contract=off", "-o", path, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        _native_path = path
        _lib = None
    _load()
    return " ".join(cmd[:-4] + ["kred_oracle.c", "-lm"])


def _load():
    global _lib
    with _lock:
        if _lib is None:
            # KRED_ORACLE_LIBRARY may name another build of kred_oracle.c (the
            # sanitizer test's)
            override = os.environ.get("KRED_ORACLE_LIBRARY")
            if _native_path is None and not override:
                build()
            lib = ctypes.CDLL(_native_path or override or _LIB)
            lib.oracle_kernel_sum.argtypes = [ctypes.c_int, ctypes.c_double, ctypes.c_int64,
                                              ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                                              _dp, _dp, _dp, _i64p, ctypes.c_int64, _dp, _dp]
            lib.oracle_gauss_gradx.argtypes = [ctypes.c_double, ctypes.c_int64, ctypes.c_int64,
                                               ctypes.c_int, _dp, _dp, _dp, _i64p,
                                               ctypes.c_int64, _dp, _dp]
            lib.oracle_gauss_vjp.argtypes = [ctypes.c_double, ctypes.c_int64, ctypes.c_int64,
                                             ctypes.c_int, ctypes.c_int, _dp, _dp, _dp, _dp,
                                             _i64p, ctypes.c_int64, _dp, _dp]
            lib.oracle_extreme.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                           ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                           ctypes.c_int, _dp, _dp, _dp, _i64p, ctypes.c_int64,
                                           _dp, _i64p, _dp]
            lib.oracle_kernel_lse.argtypes = [ctypes.c_int, ctypes.c_double, ctypes.c_int64,
                                              ctypes.c_int64, ctypes.c_int, _dp, _dp, _dp, _i64p,
                                              ctypes.c_int64, _dp, _dp]
            lib.oracle_sinkhorn_lse.argtypes = [ctypes.c_double, ctypes.c_int64, ctypes.c_int64,
                                                ctypes.c_int, _dp, _dp, _dp, _i64p,
                                                ctypes.c_int64, _dp, _dp]
            lib.oracle_argkmin.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                           ctypes.c_int, _dp, _dp, _i64p, ctypes.c_int64,
                                           _i64p, _dp]
            lib.oracle_num_threads.restype = ctypes.c_int
            for f in (lib.oracle_kernel_sum, lib.oracle_gauss_gradx, lib.oracle_gauss_vjp,
                      lib.oracle_extreme, lib.oracle_kernel_lse, lib.oracle_sinkhorn_lse,
                      lib.oracle_argkmin):
                f.restype = ctypes.c_int
            _lib = lib
    return _lib


def num_threads() -> int:
    """OpenMP threads the oracle routines run on."""
    return int(_load().oracle_num_threads())


def _f64(a, ncols=None):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.float64))
    if ncols is not None:
        a = a.reshape(-1, ncols)
    return a


def _ptr(a, t=_dp):
    return a.ctypes.data_as(t) if a is not None else None


def _rows(rows, M):
    if rows is None:
        return None, M
    r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    if r.size and (r.min() < 0 or r.max() >= M):
        raise ValueError("row index out of range")
    return r, r.size


def _check(rc):
    if rc != 0:
        raise ValueError("oracle rejected its arguments")


def kernel_sum(formula, x, y, b, sigma=1.0, rows=None):
    """Sum reduction, Eq. (2) with F = kernel(|x_i - y_j|^2) b_j (Eq. (1) for "gauss").

    Returns (a, norm), each (nrows, E) float64; norm = sum_j |F b_j|.
    """
    fcode = _FORMULAS[formula]
    x = _f64(x); y = _f64(y)
    M, D = x.shape
    N = y.shape[0]
    b = np.asarray(b, dtype=np.float64)
    E = b.shape[1] if b.ndim == 2 else 1
    b = _f64(b, E)
    r, nr = _rows(rows, M)
    out = np.empty((nr, E)); norm = np.empty((nr, E))
    _check(_load().oracle_kernel_sum(fcode, float(sigma), M, N, D, E, _ptr(x), _ptr(y),
                                     _ptr(b), _ptr(r, _i64p), nr, _ptr(out), _ptr(norm)))
    return out, norm


def gauss_gradx(x, y, b, sigma, rows=None):
    """Gaussian sum (E = 1) and its x-gradient.

    Returns (out, norm), each (nrows, 1 + D): column 0 is a_i, columns 1..D are
    g_i = sum_j k_ij b_j (y_j - x_i) / sigma^2; norm sums the absolute summands.
    """
    x = _f64(x); y = _f64(y)
    M, D = x.shape
    N = y.shape[0]
    b = _f64(b).reshape(N)
    r, nr = _rows(rows, M)
    out = np.empty((nr, 1 + D)); norm = np.empty((nr, 1 + D))
    _check(_load().oracle_gauss_gradx(float(sigma), M, N, D, _ptr(x), _ptr(y), _ptr(b),
                                      _ptr(r, _i64p), nr, _ptr(out), _ptr(norm)))
    return out, norm


def gauss_vjp(x, y, b, e, sigma, rows=None):
    """Vector-Jacobian product of the Gaussian sum a = K b (E columns) in x.

    For a cotangent e (M x E) of a: g_i = sum_j k_ij <e_i, b_j> (y_j - x_i) / sigma^2,
    the gradient of L = sum_i <e_i, a_i> in x_i.  The y-gradient is
    gauss_vjp(y, x, e, b, sigma); the b-gradient is kernel_sum("gauss", y, x, e).
    Returns (g, norm), each (nrows, D); norm sums the absolute summands.
    """
    x = _f64(x); y = _f64(y)
    M, D = x.shape
    N = y.shape[0]
    b = np.asarray(b, dtype=np.float64)
    E = b.shape[1] if b.ndim == 2 else 1
    b = _f64(b, E); e = _f64(e, E)
    if e.shape[0] != M or b.shape[0] != N:
        raise ValueError("e must be M x E and b N x E")
    r, nr = _rows(rows, M)
    out = np.empty((nr, D)); norm = np.empty((nr, D))
    _check(_load().oracle_gauss_vjp(float(sigma), M, N, D, E, _ptr(x), _ptr(y), _ptr(b),
                                    _ptr(e), _ptr(r, _i64p), nr, _ptr(out), _ptr(norm)))
    return out, norm


def extreme(formula, op, x, y, b=None, param=1.0, rows=None):
    """Min or max reduction (op "min" / "max") with the lowest arg index on ties.

    formula "gauss" / "laplace" / "sqdist": F_ije = kernel(|x_i - y_j|^2) b_je
    ("sqdist" with b None: F_ij = |x_i - y_j|^2); "sinkhorn": F_ij = g_j -
    |x_i - y_j|^2 / eps with b = g.  param: sigma, or eps for "sinkhorn".
    Returns (val, idx int64, scale), each (nrows, E); scale = max_j |F_ije|.
    """
    fcode = SINKHORN if formula == "sinkhorn" else _FORMULAS[formula]
    x = _f64(x); y = _f64(y)
    M, D = x.shape
    N = y.shape[0]
    if b is None:
        E = 1
    else:
        b = np.asarray(b, dtype=np.float64)
        E = b.shape[1] if b.ndim == 2 else 1
        b = _f64(b, E)
    r, nr = _rows(rows, M)
    val = np.empty((nr, E)); idx = np.empty((nr, E), dtype=np.int64); scale = np.empty((nr, E))
    _check(_load().oracle_extreme(fcode, {"min": 0, "max": 1}[op], float(param), M, N, D, E,
                                  _ptr(x), _ptr(y), _ptr(b), _ptr(r, _i64p), nr, _ptr(val),
                                  _ptr(idx, _i64p), _ptr(scale)))
    return val, idx, scale


def sinkhorn_lse(x, y, g, eps, rows=None):
    """Log-sum-exp reduction a_i = log sum_j exp(g_j - |x_i - y_j|^2 / eps).

    Returns (a, m): a (nrows,) and the row maxima m_i = max_j s_ij.
    """
    x = _f64(x); y = _f64(y)
    M, D = x.shape
    N = y.shape[0]
    g = _f64(g).reshape(N)
    r, nr = _rows(rows, M)
    out = np.empty(nr); mx = np.empty(nr)
    _check(_load().oracle_sinkhorn_lse(float(eps), M, N, D, _ptr(x), _ptr(y), _ptr(g),
                                       _ptr(r, _i64p), nr, _ptr(out), _ptr(mx)))
    return out, mx


def kernel_lse(formula, x, y, g, sigma, rows=None):
    """Log-domain kernel sum a_i = log sum_j k_ij exp(g_j) for "gauss" or "laplace".

    Returns (a, m): a (nrows,) and the row maxima m_i = max_j (g_j + log k_ij).
    """
    fcode = _FORMULAS[formula]
    x = _f64(x); y = _f64(y)
    M, D = x.shape
    N = y.shape[0]
    g = _f64(g).reshape(N)
    r, nr = _rows(rows, M)
    out = np.empty(nr); mx = np.empty(nr)
    _check(_load().oracle_kernel_lse(fcode, float(sigma), M, N, D, _ptr(x), _ptr(y), _ptr(g),
                                     _ptr(r, _i64p), nr, _ptr(out), _ptr(mx)))
    return out, mx


def argkmin(x, y, K, rows=None):
    """Arg-K-min: indices of the K smallest |x_i - y_j|^2, ascending by (distance, index).

    Returns (idx int64 (nrows, K), dist float64 (nrows, K)).
    """
    x = _f64(x); y = _f64(y)
    M, D = x.shape
    N = y.shape[0]
    if not (1 <= K <= min(N, 1024)):
        raise ValueError("need 1 <= K <= min(N, 1024)")
    r, nr = _rows(rows, M)
    idx = np.empty((nr, K), dtype=np.int64); dist = np.empty((nr, K))
    _check(_load().oracle_argkmin(M, N, D, int(K), _ptr(x), _ptr(y), _ptr(r, _i64p), nr,
                                  _ptr(idx, _i64p), _ptr(dist)))
    return idx, dist


def _cluster_columns(col_ptr, col_ranges, I, N):
    """Column indices of row cluster I: its ranges, clamped to [0, N), in list order."""
    cols = []
    for q in range(int(col_ptr[I]), int(col_ptr[I + 1])):
        js = min(max(int(col_ranges[q][0]), 0), N)
        je = min(max(int(col_ranges[q][1]), js), N)
        cols.extend(range(js, je))
    return np.asarray(cols, dtype=np.int64)


def ranges_reduce(kind, x, y, b, row_ranges, col_ptr, col_ranges, **kw):
    """Block-sparse (cluster-wise) reduction.

    Row cluster I is rows [row_ranges[I][0], row_ranges[I][1]); its rows reduce
    over the columns of its ranges col_ranges[col_ptr[I] : col_ptr[I + 1]] only
    (the paper's cluster-wise block-sparsity, Sec. 3).  Each cluster is handed
    to the dense routine above on its gathered columns; rows outside every
    cluster get the empty reduction.  kind:
      "sum" (formula=, sigma=), "gradx" (sigma=), "lse" (eps=; or formula= and
      sigma= for the log-domain kernel sums), "argkmin" / "kmin" (K=),
      "min" / "max" (formula=, param=).
    Returns (out, aux): out as the library writes it; aux the normaliser (sums,
    gradient), the row maximum (log-sum-exp) or the index array (min / max).
    """
    x = np.asarray(x); y = np.asarray(y)
    M, D = x.shape
    N = y.shape[0]
    R = len(row_ranges)
    formula = kw.get("formula")
    if kind == "sum":
        E = b.shape[1]
        out = np.zeros((M, E)); aux = np.zeros((M, E))
    elif kind == "gradx":
        out = np.zeros((M, 1 + D)); aux = np.zeros((M, 1 + D))
    elif kind == "lse":
        out = np.full(M, -np.inf); aux = np.full(M, -np.inf)
    elif kind in ("argkmin", "kmin"):
        K = kw["K"]
        out = np.full((M, K), -1 if kind == "argkmin" else np.inf)
        aux = None
    else:
        E = 1 if b is None or formula == "sinkhorn" else b.shape[1]
        out = np.full((M, E), np.inf if kind == "min" else -np.inf)
        aux = np.full((M, E), -1, dtype=np.int64)
    for I in range(R):
        r0 = min(max(int(row_ranges[I][0]), 0), M)
        r1 = min(max(int(row_ranges[I][1]), r0), M)
        if r1 <= r0:
            continue
        cols = _cluster_columns(col_ptr, col_ranges, I, N)
        xs = x[r0:r1]
        if cols.size == 0:
            continue
        ys = y[cols]
        bs = None if b is None else np.asarray(b)[cols]
        if kind == "sum":
            o, n = kernel_sum(formula, xs, ys, bs, sigma=kw.get("sigma", 1.0))
            out[r0:r1] = o; aux[r0:r1] = n
        elif kind == "gradx":
            o, n = gauss_gradx(xs, ys, bs, kw["sigma"])
            out[r0:r1] = o; aux[r0:r1] = n
        elif kind == "lse":
            if formula in ("gauss", "laplace"):
                o, m = kernel_lse(formula, xs, ys, bs, kw["sigma"])
            else:
                o, m = sinkhorn_lse(xs, ys, bs, kw["eps"])
            out[r0:r1] = o; aux[r0:r1] = m
        elif kind in ("argkmin", "kmin"):
            K = min(kw["K"], cols.size)
            idx, dist = argkmin(xs, ys, K)
            if kind == "argkmin":
                out[r0:r1, :K] = cols[idx]
            else:
                out[r0:r1, :K] = dist
        else:
            v, i, _ = extreme(formula, kind, xs, ys, bs, param=kw.get("param", 1.0))
            out[r0:r1] = v; aux[r0:r1] = cols[i]
    return out, aux


def ranges_backward(x, y, b, e, sigma, row_ranges, col_ptr, col_ranges):
    """Gradients of L = sum_i <e_i, a_i> for the block-sparse Gaussian sum.

    a_i = sum_{j in S(i)} k_ij b_j with S(i) the column ranges of row i's
    cluster (Sec. 3's cluster-wise block-sparsity); the derivative of such a
    reduction is again one of the same form (Sec. 2, "Backpropagation"), taken
    over the kept pairs only.  Built from the row-cluster pattern alone: each
    cluster's gathered block goes through the dense routines, its y- and
    b-gradients scattered back onto its columns.  Returns
    (gx, nx, gy, ny, gb, nb): the gradients and their normalisers (sums of
    absolute summands); rows and columns outside the pattern get zeros.
    """
    x = np.asarray(x, dtype=np.float64); y = np.asarray(y, dtype=np.float64)
    M, D = x.shape
    N = y.shape[0]
    b = np.asarray(b, dtype=np.float64).reshape(N, -1)
    E = b.shape[1]
    e = np.asarray(e, dtype=np.float64).reshape(M, E)
    gx = np.zeros((M, D)); nx = np.zeros((M, D))
    gy = np.zeros((N, D)); ny = np.zeros((N, D))
    gb = np.zeros((N, E)); nb = np.zeros((N, E))
    for I in range(len(row_ranges)):
        r0 = min(max(int(row_ranges[I][0]), 0), M)
        r1 = min(max(int(row_ranges[I][1]), r0), M)
        cols = _cluster_columns(col_ptr, col_ranges, I, N)
        if r1 <= r0 or cols.size == 0:
            continue
        xs, es, ys, bs = x[r0:r1], e[r0:r1], y[cols], b[cols]
        g, n = gauss_vjp(xs, ys, bs, es, sigma)
        gx[r0:r1] += g; nx[r0:r1] += n
        g, n = gauss_vjp(ys, xs, es, bs, sigma)
        np.add.at(gy, cols, g); np.add.at(ny, cols, n)
        g, n = kernel_sum("gauss", ys, xs, es, sigma=sigma)
        np.add.at(gb, cols, g); np.add.at(nb, cols, n)
    return gx, nx, gy, ny, gb, nb
