"""ctypes binding of libhybattn (include/hybrid_attn.h), same names as the C ABI.

Argument marshalling only: shapes come from the torch tensors, pointers from
``data_ptr()``, the stream from torch's current stream, and every nonzero
status raises :class:`HybError` with the library's message.  All arithmetic
runs in the library's HIP kernels; there is no fallback path -- if the
library has not been built, loading it raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libhybattn.so")

HYB_F32, HYB_BF16 = 0, 1
HYB_OUT_F32 = 1
HYB_STEP_SPLIT, HYB_STEP_WHOLE, HYB_STEP_HALVES = 2, 4, 8
_STEP_KERNEL = {None: 0, "auto": 0, "split": HYB_STEP_SPLIT, "whole": HYB_STEP_WHOLE,
                "halves": HYB_STEP_HALVES}
OP_STEP, OP_COMMIT, OP_PREFILL, OP_SOFTMAX_PREFIX, OP_BACKWARD, OP_BACKWARD_FULL = 0, 1, 2, 3, 4, 5
STATUS = {0: "HYB_OK", 1: "HYB_ENULL", 2: "HYB_EINVAL", 3: "HYB_EALIGN",
          4: "HYB_EDTYPE", 5: "HYB_EUNSUPPORTED", 6: "HYB_EWORKSPACE",
          7: "HYB_ELAUNCH"}
EXPORTS = ("hybrid_attn_step", "hybrid_attn_step_commit", "hybrid_state_commit",
           "hybrid_state_prefill", "hybrid_state_prefill_noalloc", "softmax_prefix_step",
           "softmax_prefix_step_paged",
           "hybrid_attn_backward", "hybrid_attn_backward_full", "hybrid_workspace_bytes",
           "hybrid_last_error")
NOALLOC_SCRATCH_BYTES = 64 << 20


class HybError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


class Dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "batch", "n_q_heads", "n_kv_heads", "head_dim", "block", "feat_dim",
        "dtype", "n_slots", "flags")]


_lib = None


def load():
    """Load libhybattn.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build it with "
            "`python -m paper_2608_06628_amd.build` (no fallback exists)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    P = ctypes.POINTER(Dims)
    lib.hybrid_attn_step.argtypes = [P] + [vp] * 11
    lib.hybrid_attn_step_commit.argtypes = [P] + [vp] * 11
    lib.hybrid_state_commit.argtypes = [P] + [vp] * 8
    lib.hybrid_state_prefill.argtypes = [P, i32] + [vp] * 10 + [sz, vp]
    lib.hybrid_state_prefill_noalloc.argtypes = [P, i32] + [vp] * 10
    lib.softmax_prefix_step.argtypes = [P] + [vp] * 6 + [i32, vp, vp, sz, vp]
    lib.softmax_prefix_step_paged.argtypes = [P] + [vp] * 5 + [i32, i32, vp, i32, vp, vp, vp,
                                                                sz, vp]
    lib.hybrid_attn_backward.argtypes = [P, i32] + [vp] * 11 + [sz, vp]
    lib.hybrid_attn_backward_full.argtypes = [P, i32] + [vp] * 14 + [sz, vp]
    lib.hybrid_workspace_bytes.argtypes = [P, i32, i32]
    lib.hybrid_workspace_bytes.restype = sz
    lib.hybrid_last_error.argtypes = []
    lib.hybrid_last_error.restype = ctypes.c_char_p
    for n in ("hybrid_attn_step", "hybrid_attn_step_commit", "hybrid_state_commit", "hybrid_state_prefill",
              "hybrid_attn_backward", "hybrid_attn_backward_full",
              "hybrid_state_prefill_noalloc", "softmax_prefix_step", "softmax_prefix_step_paged"):
        getattr(lib, n).restype = ctypes.c_int
    _lib = lib
    return lib


def last_error() -> str:
    return load().hybrid_last_error().decode()


def _check(rc: int):
    if rc != 0:
        raise HybError(rc, last_error())


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return HYB_BF16
    if t.dtype == torch.float32:
        return HYB_F32
    raise TypeError(f"unsupported activation dtype {t.dtype}")


def _ptr(t, name, dtype=None):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def make_dims(B, Hq, Hkv, d, L, f, dtype, n_slots, flags=0) -> Dims:
    return Dims(B, Hq, Hkv, d, L, f, dtype, n_slots, flags)


def _out_flags(out, act, out_f32):
    """Output dtype: fp32 when asked (or when out is an fp32 tensor)."""
    if out is not None:
        out_f32 = out.dtype == torch.float32
    odt = torch.float32 if out_f32 else act
    return (HYB_OUT_F32 if out_f32 and act != torch.float32 else 0), odt


def hybrid_attn_step(q, k, v, W, alpha, S, z, slots=None, out=None, out_f32=False,
                     stream=None, block_len=None, kernel=None):
    """q [B][L][Hq][d], k/v [B][L][Hkv][d], W [Hq][F][d], alpha [Hq] f32,
    S [n_slots][Hq][d][f] f32 (S_h transposed), z [n_slots][Hq][f] f32 -> out [B][L][Hq][d]
    in q's dtype (fp32 with out_f32).  block_len [B] int32 (device): active rows
    per request; rows past it of out are left as they were.  kernel: None or
    "auto" (the library picks), "split", "whole" or "halves" (HYB_STEP_SPLIT /
    HYB_STEP_WHOLE / HYB_STEP_HALVES)."""
    lib = load()
    B, L, Hq, d = q.shape
    act = q.dtype
    flags, odt = _out_flags(out, act, out_f32)
    flags |= _STEP_KERNEL[kernel]
    dims = make_dims(B, Hq, k.shape[2], d, L, z.shape[2], _dt(q), S.shape[0], flags)
    if out is None:
        out = torch.empty(q.shape, dtype=odt, device=q.device)
    _check(lib.hybrid_attn_step(
        ctypes.byref(dims), _ptr(q, "q"), _ptr(k, "k", act), _ptr(v, "v", act),
        _ptr(W, "W", act), _ptr(alpha, "alpha", torch.float32),
        _ptr(S, "S", torch.float32), _ptr(z, "z", torch.float32),
        _ptr(slots, "slots", torch.int32), _ptr(block_len, "block_len", torch.int32),
        _ptr(out, "out", odt), _stream(stream)))
    return out


def hybrid_attn_step_commit(q, k, v, W, alpha, S, z, slots=None, out=None, out_f32=False,
                            stream=None, block_len=None):
    """The step of hybrid_attn_step on the state as it is, then the commit of
    k/v into S, z in place, in one launch; returns out."""
    lib = load()
    B, L, Hq, d = q.shape
    act = q.dtype
    flags, odt = _out_flags(out, act, out_f32)
    dims = make_dims(B, Hq, k.shape[2], d, L, z.shape[2], _dt(q), S.shape[0], flags)
    if out is None:
        out = torch.empty(q.shape, dtype=odt, device=q.device)
    _check(lib.hybrid_attn_step_commit(
        ctypes.byref(dims), _ptr(q, "q"), _ptr(k, "k", act), _ptr(v, "v", act),
        _ptr(W, "W", act), _ptr(alpha, "alpha", torch.float32),
        _ptr(S, "S", torch.float32), _ptr(z, "z", torch.float32),
        _ptr(slots, "slots", torch.int32), _ptr(block_len, "block_len", torch.int32),
        _ptr(out, "out", odt), _stream(stream)))
    return out


def hybrid_state_commit(k, v, W, S, z, slots=None, stream=None, block_len=None):
    """Folds the block k/v [B][L][Hkv][d] into S, z in place."""
    lib = load()
    B, L, Hkv, d = k.shape
    dims = make_dims(B, W.shape[0], Hkv, d, L, z.shape[2], _dt(k), S.shape[0])
    act = k.dtype
    _check(lib.hybrid_state_commit(
        ctypes.byref(dims), _ptr(k, "k"), _ptr(v, "v", act), _ptr(W, "W", act),
        _ptr(S, "S", torch.float32), _ptr(z, "z", torch.float32),
        _ptr(slots, "slots", torch.int32), _ptr(block_len, "block_len", torch.int32),
        _stream(stream)))


def workspace_bytes(dims: Dims, op: int, extent: int = 0) -> int:
    return int(load().hybrid_workspace_bytes(ctypes.byref(dims), op, extent))


def hybrid_state_prefill(q, k, v, W, alpha, S, z, block, slots=None, out=None,
                         want_out=True, out_f32=False, ws=None, stream=None):
    """Block-causal prefill of k/v [B][T][Hkv][d] (and q [B][T][Hq][d] when
    outputs are wanted); updates S, z in place and returns out (or None)."""
    lib = load()
    B, T, Hkv, d = k.shape
    Hq = W.shape[0]
    act = k.dtype
    flags, odt = _out_flags(out, act, out_f32)
    dims = make_dims(B, Hq, Hkv, d, block, z.shape[2], _dt(k), S.shape[0], flags)
    if want_out and out is None:
        out = torch.empty((B, T, Hq, d), dtype=odt, device=k.device)
    if not want_out:
        out = None
    need = workspace_bytes(dims, OP_PREFILL, T)
    if need and ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=k.device)
    _check(lib.hybrid_state_prefill(
        ctypes.byref(dims), T, _ptr(q, "q", act) if want_out else None,
        _ptr(k, "k"), _ptr(v, "v", act), _ptr(W, "W", act),
        _ptr(alpha, "alpha", torch.float32) if want_out else None,
        _ptr(S, "S", torch.float32), _ptr(z, "z", torch.float32),
        _ptr(slots, "slots", torch.int32), _ptr(out, "out", odt) if want_out else None,
        _ptr(ws, "ws") if ws is not None else None,
        ws.numel() * ws.element_size() if ws is not None else 0, _stream(stream)))
    return out


def hybrid_state_prefill_noalloc(q, k, v, W, alpha, S, z, block, slots=None, out=None,
                                 want_out=True, out_f32=False, stream=None):
    """hybrid_state_prefill with the library-held scratch buffer as its
    workspace: the call allocates no device memory (out is allocated here
    only when the caller passes none)."""
    lib = load()
    B, T, Hkv, d = k.shape
    Hq = W.shape[0]
    act = k.dtype
    flags, odt = _out_flags(out, act, out_f32)
    dims = make_dims(B, Hq, Hkv, d, block, z.shape[2], _dt(k), S.shape[0], flags)
    if want_out and out is None:
        out = torch.empty((B, T, Hq, d), dtype=odt, device=k.device)
    if not want_out:
        out = None
    _check(lib.hybrid_state_prefill_noalloc(
        ctypes.byref(dims), T, _ptr(q, "q", act) if want_out else None,
        _ptr(k, "k"), _ptr(v, "v", act), _ptr(W, "W", act),
        _ptr(alpha, "alpha", torch.float32) if want_out else None,
        _ptr(S, "S", torch.float32), _ptr(z, "z", torch.float32),
        _ptr(slots, "slots", torch.int32), _ptr(out, "out", odt) if want_out else None,
        _stream(stream)))
    return out


def softmax_prefix_step(q, k, v, k_cache, v_cache, prefix_len, out=None, ws=None,
                        out_f32=False, stream=None):
    """Exact softmax of q [B][L][Hq][d] over k_cache/v_cache [B][Pmax][Hkv][d]
    (first prefix_len[b] rows, int32 on the device) plus the block k/v."""
    lib = load()
    B, L, Hq, d = q.shape
    Hkv = k.shape[2]
    Pmax = k_cache.shape[1]
    act = q.dtype
    flags, odt = _out_flags(out, act, out_f32)
    dims = make_dims(B, Hq, Hkv, d, L, 64, _dt(q), 1, flags)
    if out is None:
        out = torch.empty(q.shape, dtype=odt, device=q.device)
    need = workspace_bytes(dims, OP_SOFTMAX_PREFIX, Pmax)
    if need and ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=q.device)
    _check(lib.softmax_prefix_step(
        ctypes.byref(dims), _ptr(q, "q"), _ptr(k, "k", act), _ptr(v, "v", act),
        _ptr(k_cache, "k_cache", act), _ptr(v_cache, "v_cache", act),
        _ptr(prefix_len, "prefix_len", torch.int32), Pmax, _ptr(out, "out", odt),
        _ptr(ws, "ws") if ws is not None else None,
        ws.numel() * ws.element_size() if ws is not None else 0, _stream(stream)))
    return out


def softmax_prefix_step_paged(q, k, v, k_pages, v_pages, page_table, prefix_len, out=None,
                              ws=None, out_f32=False, stream=None):
    """softmax_prefix_step over a paged cache: k_pages/v_pages
    [n_pages][page_size][Hkv][d], page_table [B][max_pages] int32 and
    prefix_len [B] int32 on the device."""
    lib = load()
    B, L, Hq, d = q.shape
    Hkv = k.shape[2]
    n_pages, page_size = k_pages.shape[0], k_pages.shape[1]
    max_pages = page_table.shape[1]
    act = q.dtype
    flags, odt = _out_flags(out, act, out_f32)
    dims = make_dims(B, Hq, Hkv, d, L, 64, _dt(q), 1, flags)
    if out is None:
        out = torch.empty(q.shape, dtype=odt, device=q.device)
    need = workspace_bytes(dims, OP_SOFTMAX_PREFIX, max_pages * page_size)
    if need and ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=q.device)
    _check(lib.softmax_prefix_step_paged(
        ctypes.byref(dims), _ptr(q, "q"), _ptr(k, "k", act), _ptr(v, "v", act),
        _ptr(k_pages, "k_pages", act), _ptr(v_pages, "v_pages", act), n_pages, page_size,
        _ptr(page_table, "page_table", torch.int32), max_pages,
        _ptr(prefix_len, "prefix_len", torch.int32), _ptr(out, "out", odt),
        _ptr(ws, "ws") if ws is not None else None,
        ws.numel() * ws.element_size() if ws is not None else 0, _stream(stream)))
    return out


def hybrid_attn_backward(q, k, v, W, alpha, block, dout=None, target=None, dW=None,
                         dalpha=None, loss=None, ws=None, stream=None):
    """Gradient of the block-causal hybrid layer over q [B][T][Hq][d],
    k/v [B][T][Hkv][d] (empty starting state, blocks of `block` tokens) with
    respect to W [Hq][F][d] and alpha [Hq].  Give dout (upstream gradient) or
    target (the teacher's output; squared-error loss).  Returns
    (dW fp32 [Hq][F][d], dalpha fp32 [Hq], loss fp32 [Hq] or None)."""
    lib = load()
    B, T, Hq, d = q.shape
    Hkv = k.shape[2]
    F = W.shape[1]
    act = q.dtype
    dims = make_dims(B, Hq, Hkv, d, block, 2 * F, _dt(q), 1, 0)
    dev = q.device
    if dW is None:
        dW = torch.empty((Hq, F, d), dtype=torch.float32, device=dev)
    if dalpha is None:
        dalpha = torch.empty(Hq, dtype=torch.float32, device=dev)
    if target is not None and loss is None:
        loss = torch.empty(Hq, dtype=torch.float32, device=dev)
    need = workspace_bytes(dims, OP_BACKWARD, T)
    if ws is None and need:
        ws = torch.empty(need, dtype=torch.uint8, device=dev)
    _check(lib.hybrid_attn_backward(
        ctypes.byref(dims), T, _ptr(q, "q"), _ptr(k, "k", act), _ptr(v, "v", act),
        _ptr(W, "W", act), _ptr(alpha, "alpha", torch.float32),
        _ptr(dout, "dout", act), _ptr(target, "target", act),
        _ptr(dW, "dW", torch.float32), _ptr(dalpha, "dalpha", torch.float32),
        _ptr(loss, "loss", torch.float32),
        _ptr(ws, "ws") if ws is not None else None,
        ws.numel() * ws.element_size() if ws is not None else 0, _stream(stream)))
    return dW, dalpha, loss


def hybrid_attn_backward_full(q, k, v, W, alpha, block, dout=None, target=None, ws=None,
                              stream=None):
    """hybrid_attn_backward plus the gradients with respect to the inputs.
    Returns (dq fp32 [B][T][Hq][d], dk, dv fp32 [B][T][Hkv][d], dW, dalpha,
    loss or None)."""
    lib = load()
    B, T, Hq, d = q.shape
    Hkv = k.shape[2]
    F = W.shape[1]
    act = q.dtype
    dims = make_dims(B, Hq, Hkv, d, block, 2 * F, _dt(q), 1, 0)
    dev = q.device
    f32 = torch.float32
    dq = torch.empty((B, T, Hq, d), dtype=f32, device=dev)
    dk = torch.empty((B, T, Hkv, d), dtype=f32, device=dev)
    dv = torch.empty((B, T, Hkv, d), dtype=f32, device=dev)
    dW = torch.empty((Hq, F, d), dtype=f32, device=dev)
    dalpha = torch.empty(Hq, dtype=f32, device=dev)
    loss = torch.empty(Hq, dtype=f32, device=dev) if target is not None else None
    need = workspace_bytes(dims, OP_BACKWARD_FULL, T)
    if ws is None and need:
        ws = torch.empty(need, dtype=torch.uint8, device=dev)
    _check(lib.hybrid_attn_backward_full(
        ctypes.byref(dims), T, _ptr(q, "q"), _ptr(k, "k", act), _ptr(v, "v", act),
        _ptr(W, "W", act), _ptr(alpha, "alpha", f32),
        _ptr(dout, "dout", act), _ptr(target, "target", act),
        _ptr(dq, "dq", f32), _ptr(dk, "dk", f32), _ptr(dv, "dv", f32),
        _ptr(dW, "dW", f32), _ptr(dalpha, "dalpha", f32), _ptr(loss, "loss", f32),
        _ptr(ws, "ws") if ws is not None else None,
        ws.numel() * ws.element_size() if ws is not None else 0, _stream(stream)))
    return dq, dk, dv, dW, dalpha, loss
