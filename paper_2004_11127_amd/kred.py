"""Python binding for libkred (ctypes): argument marshalling only.

Every step of a reduction runs in the HIP kernels of libkred.so; this module
turns torch tensors into device pointers and a HIP stream handle and calls the
C ABI of include/kred.h.  torch provides device memory and streams only.
There is no CPU fallback: without the built library, or with tensors that are
not on a GPU, calls raise.
"""
from __future__ import annotations

import ctypes
import os
import re

PKG = os.path.dirname(os.path.abspath(__file__))
# KRED_LIBRARY may name another build of the same library (the sanitizer test's)
LIB_PATH = os.environ.get("KRED_LIBRARY") or os.path.join(PKG, "libkred.so")
HEADER = os.path.join(os.path.dirname(PKG), "include", "kred.h")

FORMULAS = {"gauss": 0, "laplace": 1, "sqdist": 2, "gauss_gradx": 3, "sinkhorn": 4}
REDUCTIONS = {"sum": 0, "lse": 1, "argkmin": 2, "min": 3, "max": 4, "argmin": 5, "argmax": 6,
              "kmin": 7}
INDEX_REDUCTIONS = (2, 5, 6)     # int32 outputs
STATUS = {0: "KRED_OK", 1: "KRED_ERR_INVALID_ARG", 2: "KRED_ERR_UNSUPPORTED", 3: "KRED_ERR_NOMEM",
          4: "KRED_ERR_HIP", 5: "KRED_ERR_NO_DEVICE", 6: "KRED_ERR_SCRATCH"}
NOALLOC_SCRATCH_BYTES = 32 << 20
FLAG_PROFILE = 1
FLAG_DIRECT = 2
FLAG_FAST = 4
MAX_D, MAX_E, MAX_K, MAX_COL_BLOCKS = 256, 64, 64, 256


class KredError(RuntimeError):
    def __init__(self, status, what=""):
        self.status = status
        super().__init__("%s%s (%s)" % (what + ": " if what else "", STATUS.get(status, status),
                                        strerror(status) if _lib is not None else ""))


class Params(ctypes.Structure):
    _fields_ = [("sigma", ctypes.c_float), ("eps", ctypes.c_float), ("K", ctypes.c_int32),
                ("col_blocks", ctypes.c_int32), ("flags", ctypes.c_uint32)]


_lib = None


def load():
    """Load libkred.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise FileNotFoundError("libkred.so is not built; run `python -m paper_2004_11127_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        pp = ctypes.POINTER(Params)
        lib.kred_create.argtypes = [ctypes.POINTER(vp), ctypes.c_int]
        lib.kred_destroy.argtypes = [vp]
        lib.kred_run.argtypes = [vp, ctypes.c_int, ctypes.c_int, pp, i64, i64, i32, i32,
                                 vp, vp, vp, vp, vp]
        lib.kred_run_noalloc.argtypes = lib.kred_run.argtypes
        lib.kred_validate.argtypes = [ctypes.c_int, ctypes.c_int, pp, i64, i64, i32, i32,
                                      vp, vp, vp, vp]
        lib.kred_scratch_bytes.argtypes = [ctypes.c_int, ctypes.c_int, pp, i64, i64, i32, i32]
        lib.kred_scratch_bytes.restype = i64
        lib.kred_profile_collect.argtypes = [vp, ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_double),
                                             ctypes.POINTER(ctypes.c_char_p)]
        lib.kred_gauss_backward.argtypes = [vp, pp, i64, i64, i32, i32, vp, vp, vp, vp,
                                            vp, vp, vp, vp]
        lib.kred_validate_backward.argtypes = [pp, i64, i64, i32, i32, vp, vp, vp, vp, vp, vp, vp]
        lib.kred_run_ranges.argtypes = [vp, ctypes.c_int, ctypes.c_int, pp, i64, i64, i32, i32,
                                        vp, vp, vp, vp, i32, vp, vp, vp, vp]
        lib.kred_validate_ranges.argtypes = [ctypes.c_int, ctypes.c_int, pp, i64, i64, i32, i32,
                                             vp, vp, vp, vp, i32, vp, vp, vp]
        lib.kred_gauss_backward_ranges.argtypes = [vp, pp, i64, i64, i32, i32, vp, vp, vp, vp,
                                                   vp, vp, vp, i32, vp, vp, vp, i32, vp, vp, vp,
                                                   vp]
        lib.kred_validate_backward_ranges.argtypes = [pp, i64, i64, i32, i32, vp, vp, vp, vp, vp,
                                                      vp, vp, i32, vp, vp, vp, i32, vp, vp, vp]
        lib.kred_cluster_pattern.argtypes = [vp, i64, i64, i32, vp, vp, ctypes.c_double,
                                             ctypes.c_double, vp, vp, vp, vp, vp, i64, vp, vp]
        lib.kred_cluster_pattern.restype = ctypes.c_int
        lib.kred_gather_rows.argtypes = [vp, i64, i32, vp, vp, vp, i32, vp]
        lib.kred_gather_rows.restype = ctypes.c_int
        lib.kred_strerror.argtypes = [ctypes.c_int]
        lib.kred_strerror.restype = ctypes.c_char_p
        lib.kred_version.restype = i32
        for f in (lib.kred_create, lib.kred_destroy, lib.kred_run, lib.kred_run_noalloc,
                  lib.kred_validate,
                  lib.kred_gauss_backward, lib.kred_validate_backward, lib.kred_run_ranges,
                  lib.kred_validate_ranges, lib.kred_gauss_backward_ranges,
                  lib.kred_validate_backward_ranges, lib.kred_profile_collect):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def header_symbols():
    """Names of the functions include/kred.h declares."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(kred_[a-z_]+)\s*\(",
                                 text, flags=re.M)))


def strerror(status):
    return load().kred_strerror(int(status)).decode()


def version():
    return load().kred_version()


def make_params(sigma=1.0, eps=1.0, K=0, col_blocks=0, flags=0):
    return Params(float(sigma), float(eps), int(K), int(col_blocks), int(flags))


def _codes(formula, reduction):
    f = FORMULAS[formula] if isinstance(formula, str) else int(formula)
    r = REDUCTIONS[reduction] if isinstance(reduction, str) else int(reduction)
    return f, r


def validate(formula, reduction, M, N, D, E, x=16, y=16, b=16, out=16, **params):
    """Host-only argument check (no GPU needed).

    Pointers are plain integers here and are checked only for null and alignment.
    """
    f, r = _codes(formula, reduction)
    p = make_params(**params)
    return load().kred_validate(f, r, ctypes.byref(p), int(M), int(N), int(D), int(E),
                                x, y, b, out)


def validate_backward(M, N, D, E, x=16, y=16, b=16, e=16, gx=16, gy=16, gb=16, **params):
    """Host-only argument check of the Gaussian backward (pointers as plain integers)."""
    p = make_params(**params)
    return load().kred_validate_backward(ctypes.byref(p), int(M), int(N), int(D), int(E),
                                         x, y, b, e, gx, gy, gb)


def validate_backward_ranges(M, N, D, E, nr, nc, x=16, y=16, b=16, e=16, gx=16, gy=16, gb=16,
                             rr=16, cp=16, cr=16, cc=16, rp=16, rt=16, **params):
    """Host-only argument check of the block-sparse backward (pointers as plain integers)."""
    p = make_params(**params)
    return load().kred_validate_backward_ranges(ctypes.byref(p), int(M), int(N), int(D), int(E),
                                                x, y, b, e, gx, gy, gb, int(nr), rr, cp, cr,
                                                int(nc), cc, rp, rt)


def validate_ranges(formula, reduction, M, N, D, E, nr, x=16, y=16, b=16, out=16, rr=16, cp=16,
                    cr=16, **params):
    """Host-only argument check of a block-sparse call (pointers as plain integers)."""
    f, r = _codes(formula, reduction)
    p = make_params(**params)
    return load().kred_validate_ranges(f, r, ctypes.byref(p), int(M), int(N), int(D), int(E),
                                       x, y, b, out, int(nr), rr, cp, cr)


def scratch_bytes(formula, reduction, M, N, D, E, **params):
    f, r = _codes(formula, reduction)
    p = make_params(**params)
    return load().kred_scratch_bytes(f, r, ctypes.byref(p), int(M), int(N), int(D), int(E))


def output_shape(formula, reduction, M, D, E, K=0):
    """Shape of the output; E = 0 stands for a call without b."""
    f, r = _codes(formula, reduction)
    if r in (REDUCTIONS["argkmin"], REDUCTIONS["kmin"]):
        return (M, K)
    if r in (REDUCTIONS["min"], REDUCTIONS["max"], REDUCTIONS["argmin"], REDUCTIONS["argmax"]):
        return (M, 1 if (E == 0 or f == FORMULAS["sinkhorn"]) else E)
    if f == FORMULAS["gauss_gradx"]:
        return (M, 1 + D)
    if r == REDUCTIONS["lse"]:
        return (M, 1)
    return (M, E)


class Context:
    """A kred context on one GPU (owns the library's scratch memory)."""

    def __init__(self, device=0):
        import torch
        if not torch.cuda.is_available():
            raise RuntimeError("kred needs a GPU: torch.cuda.is_available() is False")
        self.device = int(device)
        h = ctypes.c_void_p()
        st = load().kred_create(ctypes.byref(h), self.device)
        if st != 0:
            raise KredError(st, "kred_create")
        self._h = h

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            load().kred_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    @staticmethod
    def _dev_ptr(t, name, dtype):
        import torch
        if t is None:
            return None
        if not isinstance(t, torch.Tensor) or not t.is_cuda:
            raise TypeError("%s must be a GPU torch tensor" % name)
        if t.dtype != dtype or not t.is_contiguous():
            raise TypeError("%s must be a contiguous %s tensor" % (name, dtype))
        return t.data_ptr() if t.numel() else None

    def _idx_ptr(self, t, name):
        """Device pointer of an int32 index array; an empty one (a pattern with no
        ranges) gets a small zeroed buffer of the context's device, never read, so
        that the library sees a valid pointer."""
        import torch
        ptr = self._dev_ptr(t, name, torch.int32)
        if ptr is None and t is not None:
            if getattr(self, "_empty_idx", None) is None:
                self._empty_idx = torch.zeros(4, dtype=torch.int32, device=t.device)
            ptr = self._empty_idx.data_ptr()
        return ptr

    def run_ranges(self, formula, reduction, x, y, b, row_ranges, col_ptr, col_ranges, out=None,
                   sigma=1.0, eps=1.0, K=0, col_blocks=0, flags=0, stream=None):
        """Block-sparse reduction (kred_run_ranges): row cluster I = rows
        row_ranges[I, 0] .. row_ranges[I, 1] - 1 reduces over the column ranges
        col_ranges[col_ptr[I] : col_ptr[I + 1]] only.  The index arrays are int32
        GPU tensors (nr x 2, nr + 1, nnz x 2); col_blocks splits each cluster's
        columns into that many chunks (0 = automatic); otherwise as run()."""
        return self.run(formula, reduction, x, y, b, out=out, sigma=sigma, eps=eps, K=K,
                        col_blocks=col_blocks, flags=flags, stream=stream,
                        _ranges=(row_ranges, col_ptr, col_ranges))

    def run_noalloc(self, formula, reduction, x, y, b=None, out=None, sigma=1.0, eps=1.0, K=0,
                    col_blocks=0, flags=0, stream=None):
        """As run, through kred_run_noalloc: the library's fixed per-GPU scratch, no
        device allocation (pass `out` to allocate nothing here either)."""
        return self.run(formula, reduction, x, y, b, out=out, sigma=sigma, eps=eps, K=K,
                        col_blocks=col_blocks, flags=flags, stream=stream, _noalloc=True)

    def run(self, formula, reduction, x, y, b=None, out=None, sigma=1.0, eps=1.0, K=0,
            col_blocks=0, flags=0, stream=None, _ranges=None, _noalloc=False):
        """Evaluate the reduction; returns `out` (allocated when None).

        x: (M, D) float32, y: (N, D) float32, b: (N, E) float32 or None (arg-K-min,
        K-min, and the squared distance's min / max reductions), all contiguous on
        the context's GPU.  Index outputs (arg-K-min, arg-min, arg-max) are int32.
        The call is asynchronous on `stream` (a torch.cuda.Stream; default the
        current stream).
        """
        import torch
        f, r = _codes(formula, reduction)
        M, D = x.shape
        N = y.shape[0]
        if y.dim() != 2 or y.shape[1] != D:
            raise ValueError("y must be (N, D) with the same D as x")
        E = 0 if b is None else (b.shape[1] if b.dim() == 2 else 1)
        if b is not None and b.shape[0] != N:
            raise ValueError("b must have N rows")
        shape = output_shape(f, r, M, D, E, K)
        odt = torch.int32 if r in INDEX_REDUCTIONS else torch.float32
        if out is None:
            out = torch.empty(shape, dtype=odt, device=x.device)
        elif tuple(out.shape) != shape:
            raise ValueError("out must have shape %s" % (shape,))
        p = make_params(sigma, eps, K, col_blocks, flags)
        s = (stream if stream is not None else torch.cuda.current_stream(x.device)).cuda_stream
        bptr = self._dev_ptr(b, "b", torch.float32)
        if b is not None and bptr is None:
            # an empty b (N = 0) is never read, but its presence sets the output width
            bptr = 16
        args = (self._h, f, r, ctypes.byref(p), M, N, D, E, self._dev_ptr(x, "x", torch.float32),
                self._dev_ptr(y, "y", torch.float32), bptr, self._dev_ptr(out, "out", odt))
        if _ranges is None:
            st = (load().kred_run_noalloc if _noalloc else load().kred_run)(*args, s)
        else:
            rr, cp, cr = _ranges
            nr = rr.shape[0]
            if tuple(cp.shape) != (nr + 1,) or rr.dim() != 2 or rr.shape[1] != 2:
                raise ValueError("row_ranges must be (nr, 2) and col_ptr (nr + 1,)")
            st = load().kred_run_ranges(*args, nr, self._idx_ptr(rr, "row_ranges"),
                                        self._idx_ptr(cp, "col_ptr"),
                                        self._idx_ptr(cr, "col_ranges"), s)
        if st != 0:
            raise KredError(st, "kred_run(%s, %s, M=%d, N=%d, D=%d, E=%d)" % (formula, reduction,
                                                                             M, N, D, E))
        return out

    def cluster_pattern(self, x, y, cell, cutoff, col_cap=None, stream=None):
        """Block-sparse truncation pattern built on the GPU (kred_cluster_pattern).

        x (M, D), y (N, D): contiguous float32 on the context's GPU.  Returns a
        dict of int32 GPU tensors order_x (M,), order_y (N,), row_ranges (M, 2),
        col_ptr (M + 1,), col_ranges (nnz, 2) and the int64 GPU tensor counts
        (clusters of x, column ranges, pairs, overflow).  With col_cap None a
        first call with no room for column ranges sizes them (one read of the
        counts), then the second fills them; otherwise col_ranges has col_cap
        rows and nothing is read back (check counts[3] for overflow).
        """
        import torch
        M, D = x.shape
        N = y.shape[0]
        if y.dim() != 2 or y.shape[1] != D:
            raise ValueError("y must be (N, D) with the same D as x")
        s = (stream if stream is not None else torch.cuda.current_stream(x.device)).cuda_stream
        dev = x.device
        i32 = dict(dtype=torch.int32, device=dev)
        t = dict(order_x=torch.empty(M, **i32), order_y=torch.empty(N, **i32),
                 row_ranges=torch.empty((M, 2), **i32), col_ptr=torch.empty(M + 1, **i32),
                 counts=torch.empty(4, dtype=torch.int64, device=dev))

        def call(cap, cr):
            st = load().kred_cluster_pattern(
                self._h, M, N, D, self._dev_ptr(x, "x", torch.float32),
                self._dev_ptr(y, "y", torch.float32), float(cell), float(cutoff),
                t["order_x"].data_ptr(), t["order_y"].data_ptr(), t["row_ranges"].data_ptr(),
                t["col_ptr"].data_ptr(), cr.data_ptr() if cap > 0 else None, cap,
                t["counts"].data_ptr(), s)
            if st != 0:
                raise KredError(st, "kred_cluster_pattern(M=%d, N=%d, D=%d)" % (M, N, D))

        if col_cap is None:
            call(0, None)
            col_cap = int(t["counts"][1].item())
        t["col_ranges"] = torch.empty((max(col_cap, 1), 2), **i32)
        call(col_cap, t["col_ranges"])
        t["col_ranges"] = t["col_ranges"][:col_cap]
        return t

    def gather_rows(self, src, index, inverse=False, out=None, stream=None):
        """Row permutation on the GPU (kred_gather_rows): out[i] = src[index[i]],
        or out[index[i]] = src[i] with inverse.  src (n, w) float32, index (n,) int32."""
        import torch
        n = src.shape[0]
        w = 1 if src.dim() == 1 else src.shape[1]
        if out is None:
            out = torch.empty_like(src)
        s = (stream if stream is not None else torch.cuda.current_stream(src.device)).cuda_stream
        st = load().kred_gather_rows(self._h, n, w, self._dev_ptr(src, "src", torch.float32),
                                     self._dev_ptr(index, "index", torch.int32),
                                     self._dev_ptr(out, "out", torch.float32), 1 if inverse else 0, s)
        if st != 0:
            raise KredError(st, "kred_gather_rows(n=%d, width=%d)" % (n, w))
        return out

    def gauss_backward_ranges(self, x, y, b, e, pattern, transposed, sigma=1.0, gx=True,
                              gy=True, gb=True, col_blocks=0, flags=0, stream=None):
        """Gradients of the block-sparse Gaussian sum (kred_gauss_backward_ranges).

        pattern = (row_ranges, col_ptr, col_ranges) as for run_ranges, serving gx;
        transposed = (col_clusters, row_ptr, row_ranges_t), the same block set seen
        from the columns (clusters.transpose_pattern builds it), serving gy and gb.
        Index arrays are int32 GPU tensors; otherwise as gauss_backward.
        """
        return self.gauss_backward(x, y, b, e, sigma=sigma, gx=gx, gy=gy, gb=gb,
                                   col_blocks=col_blocks, flags=flags, stream=stream,
                                   _ranges=(pattern, transposed))

    def gauss_backward(self, x, y, b, e, sigma=1.0, gx=True, gy=True, gb=True, col_blocks=0,
                       flags=0, stream=None, _ranges=None):
        """Gradients of L = sum_i <e_i, a_i> for the Gaussian sum a = K b.

        x (M, D), y (N, D), b (N, E), e (M, E): contiguous float32 on the context's
        GPU.  gx, gy, gb: True (allocate), a preallocated tensor, or False/None
        (not computed).  Returns the tuple (gx, gy, gb), None where not computed.
        """
        import torch
        M, D = x.shape
        N = y.shape[0]
        if y.dim() != 2 or y.shape[1] != D:
            raise ValueError("y must be (N, D) with the same D as x")
        b2 = b if b.dim() == 2 else b.reshape(-1, 1)
        e2 = e if e.dim() == 2 else e.reshape(-1, 1)
        E = b2.shape[1]
        if b2.shape[0] != N or tuple(e2.shape) != (M, E):
            raise ValueError("b must be (N, E) and e (M, E)")

        def want(v, shape):
            if v is True:
                return torch.empty(shape, dtype=torch.float32, device=x.device)
            if v is None or v is False:
                return None
            if tuple(v.shape) != shape:
                raise ValueError("gradient output must have shape %s" % (shape,))
            return v

        ox, oy, ob = want(gx, (M, D)), want(gy, (N, D)), want(gb, (N, E))
        p = make_params(sigma, 1.0, 0, col_blocks, flags)
        s = (stream if stream is not None else torch.cuda.current_stream(x.device)).cuda_stream
        f32 = torch.float32
        args = (self._h, ctypes.byref(p), M, N, D, E,
                self._dev_ptr(x, "x", f32), self._dev_ptr(y, "y", f32),
                self._dev_ptr(b2, "b", f32), self._dev_ptr(e2, "e", f32),
                self._dev_ptr(ox, "gx", f32), self._dev_ptr(oy, "gy", f32),
                self._dev_ptr(ob, "gb", f32))
        if _ranges is None:
            st = load().kred_gauss_backward(*args, s)
        else:
            pat = []
            for (a0, a1, a2), name in zip(_ranges, ("pattern", "transposed")):
                n = a0.shape[0]
                if a0.dim() != 2 or a0.shape[1] != 2 or tuple(a1.shape) != (n + 1,):
                    raise ValueError("%s: clusters must be (n, 2) and the pointer (n + 1,)" % name)
                pat += [n, self._idx_ptr(a0, name), self._idx_ptr(a1, name),
                        self._idx_ptr(a2, name)]
            st = load().kred_gauss_backward_ranges(*args, *pat, s)
        if st != 0:
            raise KredError(st, "kred_gauss_backward(M=%d, N=%d, D=%d, E=%d)" % (M, N, D, E))
        return ox, oy, ob

    def profile_collect(self):
        """(count, total_ms, kernel) of main kernels timed since the last collect."""
        n = ctypes.c_int32()
        ms = ctypes.c_double()
        name = ctypes.c_char_p()
        st = load().kred_profile_collect(self._h, ctypes.byref(n), ctypes.byref(ms), ctypes.byref(name))
        if st != 0:
            raise KredError(st, "kred_profile_collect")
        return n.value, ms.value, name.value.decode() if name.value else ""
