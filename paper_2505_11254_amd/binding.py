"""ctypes binding of ``libdelta_attn.so`` (C ABI in ``include/delta_attn.h``).

Argument marshalling only: every step of the attention path runs in the HIP
kernels of the library.  torch supplies device memory and the stream.  There
is no fallback: a missing library or a non-gfx950 device raises.

Tensors are token-major bf16 on the GPU: q [T, Hq, d], k/v [T, Hkv, d].
A fixed-length batch passes ``B`` (T = B * N); a ragged batch passes
``cu_seqlens`` (int32, B + 1 entries, on the GPU) and ``max_seqlen``.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdelta_attn.so")

STATUS = {0: "DA_OK", 1: "DA_ERR_NULL", 2: "DA_ERR_SHAPE", 3: "DA_ERR_PARAM",
          4: "DA_ERR_UNSUPPORTED", 5: "DA_ERR_ALIGN", 6: "DA_ERR_WORKSPACE", 7: "DA_ERR_HIP"}

# C entry points and their argument types: p = pointer, i = int, z = size_t, u = unsigned,
# f = float
SIGNATURES = {
    "delta_attn_prefill": "ppppiiiiiiiipzp",
    "delta_attn_prefill_varlen": "pppppiiiiiiiipzp",
    "delta_attn_prefill_steps": "pppppiiiiiiiipzpu",
    "delta_attn_prefill_correction": "pppppiiiiiiiiifffpzp",
    "sparse_attn_prefill": "ppppiiiiiiip",
    "sparse_attn_prefill_varlen": "pppppiiiiiiip",
    "dense_causal_attn_prefill": "ppppiiiiip",
    "dense_causal_attn_prefill_varlen": "pppppiiiiip",
    "blocksparse_attn_prefill": "pppppiiiiiippp",
    "delta_attn_prefill_blocksparse": "pppppiiiiiippipzpu",
    "da_check_inputs": "piiiipplpp",
    "delta_attn_prefill_noalloc": "pppppiiiiiiiip",
}


class Plan(ctypes.Structure):
    """da_plan of include/delta_attn.h: how the library tiles a problem."""
    _fields_ = [(n, ctypes.c_int) for n in ("fused", "sparse_heads", "rows_heads", "key_chunks",
                                            "chunk_keys", "key_tile", "rows_per_wave",
                                            "waves_per_block", "sparse_slab_rows")]

    def as_dict(self):
        return {n: int(getattr(self, n)) for n, _ in self._fields_}


class DeltaAttnError(RuntimeError):
    def __init__(self, fn, status, hip_error=0):
        self.status = status
        self.hip_error = hip_error
        msg = f"{fn} returned {STATUS.get(status, status)}"
        if status == 7:
            msg += f" (hipError_t {hip_error})"
        super().__init__(msg)


_lib = None


# DA_ABI_VERSION of include/delta_attn.h that this binding's structures follow.
ABI_VERSION = 2


def load_library(path: str = LIB_PATH, check_abi: bool = True):
    """Load the HIP library (raises if it has not been built, or, with check_abi,
    if it was built against another ABI version than this binding's)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() "
                           "(hipcc for gfx950); there is no fallback implementation")
    lib = ctypes.CDLL(path)
    codes = {"p": ctypes.c_void_p, "i": ctypes.c_int, "z": ctypes.c_size_t,
             "u": ctypes.c_uint, "f": ctypes.c_float, "l": ctypes.c_int64}
    for name, sig in SIGNATURES.items():
        f = getattr(lib, name)
        f.argtypes = [codes[c] for c in sig]
        f.restype = ctypes.c_int
    lib.da_workspace_bytes.argtypes = [ctypes.c_int] * 6
    lib.da_workspace_bytes.restype = ctypes.c_size_t
    lib.da_workspace_bytes_correction.argtypes = [ctypes.c_int] * 7
    lib.da_workspace_bytes_correction.restype = ctypes.c_size_t
    lib.da_fused_supported.argtypes = [ctypes.c_int] * 3
    lib.da_fused_supported.restype = ctypes.c_int
    lib.da_fused_supported_blocksparse.argtypes = [ctypes.c_int] * 4
    lib.da_fused_supported_blocksparse.restype = ctypes.c_int
    lib.da_status_string.argtypes = [ctypes.c_int]
    lib.da_status_string.restype = ctypes.c_char_p
    lib.da_last_hip_error.argtypes = []
    lib.da_last_hip_error.restype = ctypes.c_int
    lib.da_abi_version.argtypes = []
    lib.da_abi_version.restype = ctypes.c_int
    lib.da_launch_plan.argtypes = [ctypes.c_int] * 7 + [ctypes.POINTER(Plan)]
    lib.da_launch_plan.restype = ctypes.c_int
    if check_abi and lib.da_abi_version() != ABI_VERSION:
        raise RuntimeError(f"{path} has ABI version {lib.da_abi_version()}, this binding needs "
                           f"{ABI_VERSION}: rebuild it with __graft_entry__.build()")
    _lib = lib
    return lib


def _call(name, *args):
    lib = load_library()
    rc = getattr(lib, name)(*args)
    if rc != 0:
        raise DeltaAttnError(name, rc, lib.da_last_hip_error())


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream(device, stream):
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return ctypes.c_void_p(s.cuda_stream)


def _on_device(name, t, dev, dtype):
    """t must be a contiguous tensor of `dtype` on the GPU `dev` (the kernels
    dereference its pointer on that device)."""
    if not getattr(t, "is_cuda", False) or t.device != dev:
        raise ValueError(f"{name} must be on {dev} (got {t.device})")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} (got {t.dtype})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _span(t):
    n = t.numel() * t.element_size()
    return t.data_ptr(), t.data_ptr() + n


def _check(q, k, v, out=None, cu_seqlens=None, workspace=None, block_ptr=None,
           block_idx=None):
    """Everything the C ABI takes on trust about the tensors behind its
    pointers: device, dtype, layout, matching shapes and no aliasing of the
    output with an input.  Raises ValueError before anything is launched."""
    dev = q.device
    for name, t in (("q", q), ("k", k), ("v", v)):
        _on_device(name, t, dev, torch.bfloat16)
        if t.dim() != 3:
            raise ValueError(f"{name} must be [T, H, d]")
    if tuple(k.shape) != tuple(v.shape):
        raise ValueError(f"k and v must have the same shape (got {tuple(k.shape)} and "
                         f"{tuple(v.shape)})")
    if k.shape[0] != q.shape[0] or k.shape[2] != q.shape[2]:
        raise ValueError("k and v must be [T, Hkv, d] with the T and d of q")
    if out is not None:
        _on_device("out", out, dev, torch.bfloat16)
        if tuple(out.shape) != tuple(q.shape):
            raise ValueError(f"out must have the shape of q {tuple(q.shape)}")
        o0, o1 = _span(out)
        for name, t in (("q", q), ("k", k), ("v", v)):
            t0, t1 = _span(t)
            if o0 < t1 and t0 < o1:
                raise ValueError(f"out must not overlap {name}")
    if cu_seqlens is not None:
        _on_device("cu_seqlens", cu_seqlens, dev, torch.int32)
        if cu_seqlens.dim() != 1 or cu_seqlens.numel() < 2:
            raise ValueError("cu_seqlens must be 1-D with B + 1 >= 2 entries")
    if workspace is not None:
        _on_device("workspace", workspace, dev, None)
    for name, t in (("block_ptr", block_ptr), ("block_idx", block_idx)):
        if t is not None:
            _on_device(name, t, dev, torch.int32)


def _shapes(q, k, v, B, cu_seqlens, max_seqlen):
    _check(q, k, v, cu_seqlens=cu_seqlens)
    T, Hq, d = q.shape
    Hkv = k.shape[1]
    if cu_seqlens is None:
        B = 1 if B is None else int(B)
        if B < 1 or T % B != 0:
            raise ValueError("T must be a multiple of B for a fixed-length batch")
        return B, T // B, Hq, Hkv, d
    if max_seqlen is None:
        raise ValueError("max_seqlen is required with cu_seqlens")
    return cu_seqlens.numel() - 1, int(max_seqlen), Hq, Hkv, d


def workspace_bytes(B, max_seqlen, Hq, Hkv, d, gamma) -> int:
    return int(load_library().da_workspace_bytes(B, max_seqlen, Hq, Hkv, d, gamma))


def launch_plan(B, max_seqlen, Hq, Hkv, d, gamma, block_q=0) -> dict:
    """The library's tiling of a problem (da_launch_plan; host only)."""
    p = Plan()
    lib = load_library()
    rc = lib.da_launch_plan(B, max_seqlen, Hq, Hkv, d, gamma, block_q, ctypes.byref(p))
    if rc != 0:
        raise DeltaAttnError("da_launch_plan", rc)
    return p.as_dict()


def fused_supported(Hq, Hkv, gamma) -> bool:
    """Whether delta_attn_prefill takes the fused schedule for these sizes."""
    return bool(load_library().da_fused_supported(Hq, Hkv, gamma))


def delta_attn_prefill(q, k, v, *, window, n_sink, gamma, B=None, cu_seqlens=None,
                       max_seqlen=None, out=None, workspace=None, stream=None):
    """Delta Attention prefill (Algorithm 1); returns ``out`` [T, Hq, d] bf16."""
    B_, N, Hq, Hkv, d = _shapes(q, k, v, B, cu_seqlens, max_seqlen)
    if out is None:
        out = torch.empty_like(q)
    nbytes = workspace_bytes(B_, N, Hq, Hkv, d, gamma)
    if workspace is None:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=q.device)
    _check(q, k, v, out, cu_seqlens, workspace)
    wsz = workspace.numel() * workspace.element_size()
    st = _stream(q.device, stream)
    if cu_seqlens is None:
        _call("delta_attn_prefill", _ptr(q), _ptr(k), _ptr(v), _ptr(out), B_, Hq, Hkv, N, d,
              window, n_sink, gamma, _ptr(workspace), wsz, st)
    else:
        _call("delta_attn_prefill_varlen", _ptr(q), _ptr(k), _ptr(v), _ptr(out),
              _ptr(cu_seqlens), B_, N, Hq, Hkv, d, window, n_sink, gamma, _ptr(workspace),
              wsz, st)
    return out


def delta_attn_prefill_noalloc(q, k, v, *, window, n_sink, gamma, B=None, cu_seqlens=None,
                               max_seqlen=None, out=None, stream=None):
    """Delta Attention prefill whose workspace is the library's static device
    array (delta_attn_prefill_noalloc): the call allocates nothing on the
    device; pass ``out`` to allocate nothing here either."""
    B_, N, Hq, Hkv, d = _shapes(q, k, v, B, cu_seqlens, max_seqlen)
    if out is None:
        out = torch.empty_like(q)
    _check(q, k, v, out, cu_seqlens)
    _call("delta_attn_prefill_noalloc", _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(cu_seqlens),
          B_, N, Hq, Hkv, d, window, n_sink, gamma, _stream(q.device, stream))
    return out


STEP_SPARSE, STEP_DENSE_ROWS, STEP_CORRECT, STEP_ALL, STEP_FUSED = 1, 2, 4, 7, 8
CORR_DELTA, CORR_RECOMPUTE, CORR_INTERP, CORR_EMA, CORR_ABG = 0, 1, 2, 3, 4


def delta_attn_prefill_correction(q, k, v, *, window, n_sink, gamma, mode,
                                  params=(0.0, 0.0, 0.0), B=None, cu_seqlens=None,
                                  max_seqlen=None, out=None, workspace=None, stream=None):
    """Algorithm 1 with the step-5 correction chosen by ``mode`` (CORR_*)."""
    B_, N, Hq, Hkv, d = _shapes(q, k, v, B, cu_seqlens, max_seqlen)
    if out is None:
        out = torch.empty_like(q)
    nbytes = int(load_library().da_workspace_bytes_correction(B_, N, Hq, Hkv, d, gamma, mode))
    if workspace is None:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=q.device)
    _check(q, k, v, out, cu_seqlens, workspace)
    wsz = workspace.numel() * workspace.element_size()
    p = list(params) + [0.0] * (3 - len(params))
    _call("delta_attn_prefill_correction", _ptr(q), _ptr(k), _ptr(v), _ptr(out),
          _ptr(cu_seqlens), B_, N, Hq, Hkv, d, window, n_sink, gamma, mode, float(p[0]),
          float(p[1]), float(p[2]), _ptr(workspace), wsz, _stream(q.device, stream))
    return out


def delta_attn_prefill_steps(q, k, v, out, workspace, steps, *, window, n_sink, gamma, B=None,
                             cu_seqlens=None, max_seqlen=None, stream=None):
    """Run the given steps of Algorithm 1 (bit mask of STEP_*) on existing buffers."""
    B_, N, Hq, Hkv, d = _shapes(q, k, v, B, cu_seqlens, max_seqlen)
    _check(q, k, v, out, cu_seqlens, workspace)
    wsz = workspace.numel() * workspace.element_size()
    _call("delta_attn_prefill_steps", _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(cu_seqlens),
          B_, N, Hq, Hkv, d, window, n_sink, gamma, _ptr(workspace), wsz,
          _stream(q.device, stream), steps)
    return out


def sparse_attn_prefill(q, k, v, *, window, n_sink, B=None, cu_seqlens=None, max_seqlen=None,
                        out=None, stream=None):
    """Sink + sliding-window attention for every row (the f* of the paper)."""
    B_, N, Hq, Hkv, d = _shapes(q, k, v, B, cu_seqlens, max_seqlen)
    if out is None:
        out = torch.empty_like(q)
    _check(q, k, v, out, cu_seqlens)
    st = _stream(q.device, stream)
    if cu_seqlens is None:
        _call("sparse_attn_prefill", _ptr(q), _ptr(k), _ptr(v), _ptr(out), B_, Hq, Hkv, N, d,
              window, n_sink, st)
    else:
        _call("sparse_attn_prefill_varlen", _ptr(q), _ptr(k), _ptr(v), _ptr(out),
              _ptr(cu_seqlens), B_, N, Hq, Hkv, d, window, n_sink, st)
    return out


def dense_causal_attn_prefill(q, k, v, *, B=None, cu_seqlens=None, max_seqlen=None, out=None,
                              stream=None):
    """Dense causal attention for every row (the quadratic baseline f)."""
    B_, N, Hq, Hkv, d = _shapes(q, k, v, B, cu_seqlens, max_seqlen)
    if out is None:
        out = torch.empty_like(q)
    _check(q, k, v, out, cu_seqlens)
    st = _stream(q.device, stream)
    if cu_seqlens is None:
        _call("dense_causal_attn_prefill", _ptr(q), _ptr(k), _ptr(v), _ptr(out), B_, Hq, Hkv,
              N, d, st)
    else:
        _call("dense_causal_attn_prefill_varlen", _ptr(q), _ptr(k), _ptr(v), _ptr(out),
              _ptr(cu_seqlens), B_, N, Hq, Hkv, d, st)
    return out


def fused_supported_blocksparse(Hq, Hkv, gamma, block_q) -> bool:
    """Whether the key-block-list path takes the fused schedule for these sizes."""
    return bool(load_library().da_fused_supported_blocksparse(Hq, Hkv, gamma, block_q))


def _blocks(block_ptr, block_idx, B, Hkv, N, block_q):
    """Pointers of the key-block lists after checking their device, dtype and
    that block_ptr holds [B, Hkv, ceil(N / block_q) + 1] offsets."""
    if block_q not in (64, 128, 256):
        raise ValueError("block_q must be 64, 128 or 256")
    nqb = -(-N // block_q)
    if block_ptr.numel() != B * Hkv * (nqb + 1):
        raise ValueError(f"block_ptr must hold B * Hkv * (ceil(N / block_q) + 1) = "
                         f"{B * Hkv * (nqb + 1)} offsets (got {block_ptr.numel()})")
    return _ptr(block_ptr), _ptr(block_idx)


def blocksparse_attn_prefill(q, k, v, *, block_q, block_ptr, block_idx, B=None,
                             cu_seqlens=None, max_seqlen=None, out=None, stream=None):
    """Sparse attention whose key sets come from key-block lists, for every row."""
    B_, N, Hq, Hkv, d = _shapes(q, k, v, B, cu_seqlens, max_seqlen)
    if out is None:
        out = torch.empty_like(q)
    _check(q, k, v, out, cu_seqlens, block_ptr=block_ptr, block_idx=block_idx)
    _call("blocksparse_attn_prefill", _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(cu_seqlens),
          B_, N, Hq, Hkv, d, block_q, *_blocks(block_ptr, block_idx, B_, Hkv, N, block_q),
          _stream(q.device, stream))
    return out


def delta_attn_prefill_blocksparse(q, k, v, *, block_q, block_ptr, block_idx, gamma, B=None,
                                   cu_seqlens=None, max_seqlen=None, out=None, workspace=None,
                                   stream=None, steps=0):
    """Delta Attention with f* from key-block lists; ``steps`` 0 runs the whole path."""
    B_, N, Hq, Hkv, d = _shapes(q, k, v, B, cu_seqlens, max_seqlen)
    if out is None:
        out = torch.empty_like(q)
    nbytes = workspace_bytes(B_, N, Hq, Hkv, d, gamma)
    if workspace is None:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=q.device)
    _check(q, k, v, out, cu_seqlens, workspace, block_ptr, block_idx)
    wsz = workspace.numel() * workspace.element_size()
    _call("delta_attn_prefill_blocksparse", _ptr(q), _ptr(k), _ptr(v), _ptr(out),
          _ptr(cu_seqlens), B_, N, Hq, Hkv, d, block_q,
          *_blocks(block_ptr, block_idx, B_, Hkv, N, block_q), gamma,
          _ptr(workspace), wsz, _stream(q.device, stream), steps)
    return out


def check_inputs(*, max_seqlen, B=None, cu_seqlens=None, Hkv=None, block_q=None,
                 block_ptr=None, block_idx=None, stream=None):
    """Count violations of the rules cu_seqlens and key-block lists must follow
    (see da_check_inputs); synchronises the stream.  Returns the count."""
    import torch as _t
    dev = (cu_seqlens if cu_seqlens is not None else block_ptr).device
    if B is None:
        B = cu_seqlens.numel() - 1
    result = _t.zeros(1, dtype=_t.int32, device=dev)
    nnz = block_idx.numel() if block_idx is not None else 0
    lib = load_library()
    rc = lib.da_check_inputs(_ptr(cu_seqlens), B, max_seqlen, Hkv or 0, block_q or 0,
                             _ptr(block_ptr), _ptr(block_idx), nnz, _ptr(result),
                             _stream(dev, stream))
    if rc not in (0, 3):
        raise DeltaAttnError("da_check_inputs", rc, lib.da_last_hip_error())
    return int(result.item())

