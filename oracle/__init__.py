"""fp64 CPU oracle of the Delta Attention prefill (arXiv 2505.11254).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no
code with the GPU library and never imports it.

The arithmetic lives in ``delta_oracle.c`` (plain fp64 loops, OpenMP over
rows).  This module only builds that file with gcc and marshals numpy arrays.

Inputs are token-major arrays ``q [T, Hq, d]``, ``k, v [T, Hkv, d]`` holding
either fp64 values or IEEE bfloat16 bit patterns (``uint16``); the latter are
widened to fp64 exactly inside the C code.  ``cu`` lists sequence starts
(``B + 1`` entries, host int64).  See ``delta_oracle.c`` for the definitions
and the readings of the paper it takes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "delta_oracle.c")
_LIB = os.path.join(_HERE, "libdelta_oracle.so")

MODE_DENSE = 0
MODE_SPARSE = 1

# correction variants of step 5 (see dao_delta_attention_variant)
CORR_DELTA, CORR_RECOMPUTE, CORR_INTERP, CORR_EMA, CORR_ABG = 0, 1, 2, 3, 4

_lib = None


def build(force: bool = True, src: str = _SRC, dst: str = _LIB) -> str:
    """Compile ``delta_oracle.c`` (or a copy of it) into a shared library with gcc."""
    if force or not os.path.exists(dst):
        tmp = dst + ".tmp"
        cmd = ["gcc", "-O3", "-march=x86-64-v3", "-fopenmp", "-fPIC", "-shared",
               "-Wall", "-Wextra", src, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, dst)
    return dst


def _bind(path):
    lib = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
    lib.dao_attention.argtypes = [vp, vp, vp, i32, vp, i32, i32, i32, i32, i32, i32, i32,
                                  vp, i64, vp, vp, vp, i32]
    lib.dao_attention_weights.argtypes = [vp, vp, vp, i32, vp, i32, i32, i32, i32, i32, i32,
                                          i32, i32, i32, i64, vp, vp]
    lib.dao_delta_attention.argtypes = [vp, vp, vp, i32, vp, i32, i32, i32, i32, i32, i32,
                                        i32, vp, vp, vp, i32]
    lib.dao_delta_attention_rows.argtypes = [vp, vp, vp, i32, vp, i32, i32, i32, i32, i32,
                                             i32, i32, vp, i64, vp, vp, i32]
    lib.dao_delta_attention_variant.argtypes = [vp, vp, vp, i32, vp, i32, i32, i32, i32, i32,
                                                i32, i32, i32, ctypes.c_double, ctypes.c_double,
                                                ctypes.c_double, vp, i32]
    lib.dao_block_attention.argtypes = [vp, vp, vp, i32, vp, i32, i32, i32, i32, vp, vp, i32,
                                        i32, vp, i64, vp, i32]
    lib.dao_block_delta_attention.argtypes = [vp, vp, vp, i32, vp, i32, i32, i32, i32, vp, vp,
                                              i32, i32, i32, vp, vp, vp, i32]
    lib.dao_block_delta_attention_rows.argtypes = [vp, vp, vp, i32, vp, i32, i32, i32, i32, vp,
                                                   vp, i32, i32, i32, vp, i64, vp, vp, i32]
    lib.dao_block_attention_weights.argtypes = [vp, vp, vp, i32, vp, i32, i32, i32, i32, vp, vp,
                                                i32, i32, i32, i32, i64, vp, vp]
    for f in (lib.dao_attention, lib.dao_attention_weights, lib.dao_delta_attention,
              lib.dao_delta_attention_rows, lib.dao_delta_attention_variant,
              lib.dao_block_attention, lib.dao_block_delta_attention,
              lib.dao_block_delta_attention_rows, lib.dao_block_attention_weights):
        f.restype = ctypes.c_int
    lib.dao_max_threads.restype = ctypes.c_int
    lib.dao_max_threads.argtypes = []
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        _lib = _bind(_LIB)
    return _lib


def max_threads() -> int:
    """OpenMP threads the oracle uses by default."""
    return int(_load().dao_max_threads())


def _as_input(x):
    """Return (contiguous ndarray, is_bf16) for a numpy array or torch CPU tensor."""
    if type(x).__module__.startswith("torch"):
        import torch
        x = x.detach().cpu().contiguous()
        if x.dtype == torch.bfloat16:
            return x.view(torch.int16).numpy().view(np.uint16), True
        return x.to(torch.float64).numpy(), False
    x = np.ascontiguousarray(x)
    if x.dtype == np.uint16:
        return x, True
    return np.ascontiguousarray(x, dtype=np.float64), False


class _Problem:
    def __init__(self, q, k, v, cu):
        self.q, bq = _as_input(q)
        self.k, bk = _as_input(k)
        self.v, bv = _as_input(v)
        if not (bq == bk == bv):
            raise ValueError("q, k, v must all be bf16 bit patterns or all be fp64")
        self.bf16 = int(bq)
        if self.q.ndim != 3 or self.k.ndim != 3 or self.v.ndim != 3:
            raise ValueError("q, k, v must be [T, H, d]")
        self.T, self.Hq, self.d = self.q.shape
        self.Hkv = self.k.shape[1]
        if self.k.shape != (self.T, self.Hkv, self.d) or self.v.shape != self.k.shape:
            raise ValueError("k and v must be [T, Hkv, d] with q's T and d")
        if cu is None:
            cu = [0, self.T]
        self.cu = np.ascontiguousarray(np.asarray(cu, dtype=np.int64))
        self.B = len(self.cu) - 1
        if self.cu[0] != 0 or self.cu[-1] != self.T:
            raise ValueError("cu must start at 0 and end at T")

    def ptrs(self):
        return (self.q.ctypes.data, self.k.ctypes.data, self.v.ctypes.data, self.bf16,
                self.cu.ctypes.data, self.B, self.Hq, self.Hkv, self.d)


def _check(rc, name):
    if rc != 0:
        raise RuntimeError(f"oracle {name} failed with code {rc}")


def _rows_array(rows):
    r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64).reshape(-1, 3))
    return r


class Oracle:
    """The oracle's entry points bound to one build of ``delta_oracle.c``."""

    def __init__(self, libpath: str | None = None):
        self._lib = _bind(libpath) if libpath else _load()

    def attention(self, q, k, v, cu=None, *, mode=MODE_DENSE, window=1, n_sink=0, rows=None,
                  nthreads=0, return_stats=False):
        """Dense causal (``MODE_DENSE``) or sink+window (``MODE_SPARSE``) attention.

        Returns ``[T, Hq, d]`` (or ``[n_rows, d]`` when ``rows`` lists (b, h, i)
        triples), plus the per-row score max and normaliser when ``return_stats``.
        """
        P = _Problem(q, k, v, cu)
        if rows is None:
            out = np.zeros((P.T, P.Hq, P.d))
            m = np.zeros((P.T, P.Hq))
            z = np.zeros((P.T, P.Hq))
            rp, nr = None, 0
        else:
            r = _rows_array(rows)
            out = np.zeros((len(r), P.d))
            m = np.zeros(len(r))
            z = np.zeros(len(r))
            rp, nr = r.ctypes.data, len(r)
        rc = self._lib.dao_attention(*P.ptrs(), window, n_sink, mode, rp, nr, out.ctypes.data,
                                     m.ctypes.data, z.ctypes.data, nthreads)
        _check(rc, "attention")
        return (out, m, z) if return_stats else out

    def attention_weights(self, q, k, v, cu=None, *, mode, window=1, n_sink=0, b=0, h=0, i=0):
        """Softmax weights the oracle gives row (b, h, i) over keys 0..i, and its output."""
        P = _Problem(q, k, v, cu)
        w = np.zeros(i + 1)
        o = np.zeros(P.d)
        rc = self._lib.dao_attention_weights(*P.ptrs(), window, n_sink, mode, b, h, i,
                                             w.ctypes.data, o.ctypes.data)
        _check(rc, "attention_weights")
        return w, o

    def delta_attention(self, q, k, v, cu=None, *, window, n_sink, gamma, nthreads=0,
                        return_parts=False):
        """Algorithm 1 over whole sequences: ``[T, Hq, d]`` fp64.

        With ``return_parts`` also returns the sparse output A*V and the
        correction added to each row (zero on dense tail rows).
        """
        P = _Problem(q, k, v, cu)
        out = np.zeros((P.T, P.Hq, P.d))
        sp = np.zeros((P.T, P.Hq, P.d)) if return_parts else None
        dl = np.zeros((P.T, P.Hq, P.d)) if return_parts else None
        rc = self._lib.dao_delta_attention(*P.ptrs(), window, n_sink, gamma, out.ctypes.data,
                                           sp.ctypes.data if sp is not None else None,
                                           dl.ctypes.data if dl is not None else None,
                                           nthreads)
        _check(rc, "delta_attention")
        return (out, sp, dl) if return_parts else out

    def delta_attention_rows(self, q, k, v, cu=None, *, window, n_sink, gamma, rows,
                             nthreads=0, return_delta=False):
        """Algorithm 1's value at selected rows: ``rows`` is an (n, 3) list of (b, h, i)."""
        P = _Problem(q, k, v, cu)
        r = _rows_array(rows)
        out = np.zeros((len(r), P.d))
        dl = np.zeros((len(r), P.d)) if return_delta else None
        rc = self._lib.dao_delta_attention_rows(*P.ptrs(), window, n_sink, gamma,
                                                r.ctypes.data, len(r), out.ctypes.data,
                                                dl.ctypes.data if dl is not None else None,
                                                nthreads)
        _check(rc, "delta_attention_rows")
        return (out, dl) if return_delta else out


class _Blocks:
    """Key-block lists in CSR form: ``ptr`` [B, Hkv, nqb + 1] offsets into ``idx``
    (key tile indices, tiles of 64 keys, local to each sequence), query blocks of
    ``block_q`` rows."""

    def __init__(self, P, ptr, idx, block_q):
        self.ptr = np.ascontiguousarray(np.asarray(ptr, dtype=np.int64))
        self.idx = np.ascontiguousarray(np.asarray(idx, dtype=np.int64).reshape(-1))
        if self.ptr.ndim != 3 or self.ptr.shape[:2] != (P.B, P.Hkv):
            raise ValueError("block ptr must be [B, Hkv, nqb + 1]")
        self.nqb = self.ptr.shape[2] - 1
        self.block_q = int(block_q)
        if self.idx.size == 0:
            self.idx = np.zeros(1, dtype=np.int64)

    def args(self):
        return self.ptr.ctypes.data, self.idx.ctypes.data, self.nqb, self.block_q


def _block_attention(self, q, k, v, cu=None, *, blk_ptr, blk_idx, block_q, rows=None,
                     nthreads=0):
    """Sparse attention whose key sets come from key-block lists (see
    ``delta_oracle.c``): ``[T, Hq, d]``, or ``[n_rows, d]`` for (b, h, i) rows."""
    P = _Problem(q, k, v, cu)
    Bl = _Blocks(P, blk_ptr, blk_idx, block_q)
    if rows is None:
        out = np.zeros((P.T, P.Hq, P.d))
        rp, nr = None, 0
    else:
        r = _rows_array(rows)
        out = np.zeros((len(r), P.d))
        rp, nr = r.ctypes.data, len(r)
    rc = self._lib.dao_block_attention(*P.ptrs(), *Bl.args(), rp, nr, out.ctypes.data, nthreads)
    _check(rc, "block_attention")
    return out


def _block_delta_attention(self, q, k, v, cu=None, *, blk_ptr, blk_idx, block_q, gamma,
                           nthreads=0, return_parts=False):
    """Algorithm 1 with f* from key-block lists: ``[T, Hq, d]`` fp64 (plus the
    sparse output and the per-row correction with ``return_parts``)."""
    P = _Problem(q, k, v, cu)
    Bl = _Blocks(P, blk_ptr, blk_idx, block_q)
    out = np.zeros((P.T, P.Hq, P.d))
    sp = np.zeros((P.T, P.Hq, P.d)) if return_parts else None
    dl = np.zeros((P.T, P.Hq, P.d)) if return_parts else None
    rc = self._lib.dao_block_delta_attention(*P.ptrs(), *Bl.args(), gamma, out.ctypes.data,
                                             sp.ctypes.data if sp is not None else None,
                                             dl.ctypes.data if dl is not None else None,
                                             nthreads)
    _check(rc, "block_delta_attention")
    return (out, sp, dl) if return_parts else out


def _block_delta_attention_rows(self, q, k, v, cu=None, *, blk_ptr, blk_idx, block_q, gamma,
                                rows, nthreads=0):
    """Algorithm 1 with f* from key-block lists, at selected (b, h, i) rows."""
    P = _Problem(q, k, v, cu)
    Bl = _Blocks(P, blk_ptr, blk_idx, block_q)
    r = _rows_array(rows)
    out = np.zeros((len(r), P.d))
    rc = self._lib.dao_block_delta_attention_rows(*P.ptrs(), *Bl.args(), gamma, r.ctypes.data,
                                                  len(r), out.ctypes.data, None, nthreads)
    _check(rc, "block_delta_attention_rows")
    return out


def _block_attention_weights(self, q, k, v, cu=None, *, blk_ptr, blk_idx, block_q, b=0, h=0,
                             i=0):
    """Softmax weights of row (b, h, i) under key-block lists, and its output."""
    P = _Problem(q, k, v, cu)
    Bl = _Blocks(P, blk_ptr, blk_idx, block_q)
    w = np.zeros(i + 1)
    o = np.zeros(P.d)
    rc = self._lib.dao_block_attention_weights(*P.ptrs(), *Bl.args(), b, h, i, w.ctypes.data,
                                               o.ctypes.data)
    _check(rc, "block_attention_weights")
    return w, o


Oracle.block_attention = _block_attention
Oracle.block_delta_attention = _block_delta_attention
Oracle.block_delta_attention_rows = _block_delta_attention_rows
Oracle.block_attention_weights = _block_attention_weights


def block_attention(*args, **kw):
    return Oracle().block_attention(*args, **kw)


def block_delta_attention(*args, **kw):
    return Oracle().block_delta_attention(*args, **kw)


def block_delta_attention_rows(*args, **kw):
    return Oracle().block_delta_attention_rows(*args, **kw)


def block_attention_weights(*args, **kw):
    return Oracle().block_attention_weights(*args, **kw)


def _variant(self, q, k, v, cu=None, *, window, n_sink, gamma, mode, params=(0.0, 0.0, 0.0),
             nthreads=0):
    """Algorithm 1 with the correction of step 5 chosen by ``mode`` (CORR_*)."""
    P = _Problem(q, k, v, cu)
    out = np.zeros((P.T, P.Hq, P.d))
    p = list(params) + [0.0] * (3 - len(params))
    rc = self._lib.dao_delta_attention_variant(*P.ptrs(), window, n_sink, gamma, mode,
                                               float(p[0]), float(p[1]), float(p[2]),
                                               out.ctypes.data, nthreads)
    _check(rc, "delta_attention_variant")
    return out


Oracle.delta_attention_variant = _variant


def delta_attention_variant(*args, **kw):
    return Oracle().delta_attention_variant(*args, **kw)


delta_attention_variant.__doc__ = _variant.__doc__


def attention(*args, **kw):
    return Oracle().attention(*args, **kw)


def attention_weights(*args, **kw):
    return Oracle().attention_weights(*args, **kw)


def delta_attention(*args, **kw):
    return Oracle().delta_attention(*args, **kw)


def delta_attention_rows(*args, **kw):
    return Oracle().delta_attention_rows(*args, **kw)


for _f, _m in ((attention, Oracle.attention), (attention_weights, Oracle.attention_weights),
               (delta_attention, Oracle.delta_attention),
               (delta_attention_rows, Oracle.delta_attention_rows)):
    _f.__doc__ = _m.__doc__
