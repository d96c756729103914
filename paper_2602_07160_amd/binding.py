"""Python binding of libfem.so (argument marshalling only).

Each function has the name of the C entry point it calls (``include/fem.h``)
and takes torch tensors for the device buffers: torch provides device memory
and the stream, every step of the read runs in the library's HIP kernels.
There is no fallback: if libfem.so is missing or a call fails, an exception
is raised.
"""

from __future__ import annotations

import ctypes
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfem.so")

FEM_DTYPE = {torch.float32: 0, torch.bfloat16: 1}

EXPORTS = ("fem_softmax_fwd", "fem_softmax_fwd_ex", "fem_softmax_fwd_train", "fem_softmax_bwd",
           "fem_softmax_bwd_workspace_bytes", "fem_softmax_gated_fwd", "fem_softmax_decode",
           "fem_softmax_decode_workspace_bytes", "fem_softmax_decode_noalloc", "fem_linear_fwd", "fem_linear_workspace_bytes",
           "fem_gla_fwd", "fem_gla_workspace_bytes", "fem_status_str")

FEM_FLAG_ENCODER = 1
FEM_FLAG_OUT_BF16 = 2

_lib = None


class FemError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


def load() -> ctypes.CDLL:
    """Load libfem.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run `python -m paper_2602_07160_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        vp, i, f, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t
        lib.fem_softmax_fwd.argtypes = [vp, vp, vp, f, f, i, i, i, i, i, vp]
        lib.fem_softmax_fwd.restype = i
        lib.fem_softmax_fwd_ex.argtypes = [vp, vp, vp, f, vp, i, i, i, i, i, i, i, vp]
        lib.fem_softmax_fwd_ex.restype = i
        lib.fem_softmax_decode.argtypes = [vp, vp, vp, vp, f, f, i, i, i, i, i, i, vp, sz, vp]
        lib.fem_softmax_decode.restype = i
        lib.fem_softmax_decode_workspace_bytes.argtypes = [i, i, i, i, i]
        lib.fem_softmax_decode_workspace_bytes.restype = sz
        lib.fem_softmax_decode_noalloc.argtypes = [vp, vp, vp, vp, f, f, i, i, i, i, i, i, vp]
        lib.fem_softmax_decode_noalloc.restype = i
        lib.fem_softmax_gated_fwd.argtypes = [vp, vp, vp, f, f, f, f, i, i, i, i, i, vp]
        lib.fem_softmax_gated_fwd.restype = i
        lib.fem_linear_fwd.argtypes = [vp, vp, vp, f, f, i, i, i, i, i, i, i, vp, sz, vp]
        lib.fem_linear_fwd.restype = i
        lib.fem_linear_workspace_bytes.argtypes = [i, i, i, i, i, i]
        lib.fem_linear_workspace_bytes.restype = sz
        lib.fem_gla_fwd.argtypes = [vp, vp, vp, f, f, f, i, i, i, i, i, i, i, vp, sz, vp]
        lib.fem_gla_fwd.restype = i
        lib.fem_gla_workspace_bytes.argtypes = [i, i, i, i, i, i]
        lib.fem_gla_workspace_bytes.restype = sz
        lib.fem_softmax_fwd_train.argtypes = [vp, vp, vp, f, f, f, i, i, i, i, i, vp]
        lib.fem_softmax_fwd_train.restype = i
        lib.fem_softmax_bwd.argtypes = [vp, vp, vp, f, f, f, f, f, f, f, f, i, i, i, i, i, vp, sz,
                                        vp]
        lib.fem_softmax_bwd.restype = i
        lib.fem_softmax_bwd_workspace_bytes.argtypes = [i, i, i, i]
        lib.fem_softmax_bwd_workspace_bytes.restype = sz
        lib.fem_status_str.argtypes = [i]
        lib.fem_status_str.restype = ctypes.c_char_p
        _lib = lib
    return _lib


def fem_status_str(status: int) -> str:
    return load().fem_status_str(int(status)).decode()


def _check(rc: int):
    if rc != 0:
        raise FemError(rc, fem_status_str(rc))


def _dev_tensor(x: torch.Tensor, name: str, dtype=None) -> torch.Tensor:
    if not isinstance(x, torch.Tensor) or not x.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not x.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and x.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {x.dtype}")
    return x


def _workspace(nbytes: int, device, ws, stream):
    """(tensor, pointer, size) of the workspace for a call that needs
    ``nbytes``: the caller's uint8 GPU tensor ``ws`` if given, else a new one
    from torch's allocator (its blocks are 512-byte aligned), allocated on the
    stream the call runs on so that torch does not hand the memory out again
    before the call's kernels have run.  (None, None, 0) when nothing is
    needed."""
    if ws is not None:
        _dev_tensor(ws, "ws", torch.uint8)
        return ws, ws.data_ptr(), ws.numel()
    if nbytes == 0:
        return None, None, 0
    s = torch.cuda.current_stream(device) if stream is None else stream
    if not isinstance(s, torch.cuda.Stream):
        s = torch.cuda.ExternalStream(int(s), device=device)
    with torch.cuda.stream(s):
        t = torch.empty(nbytes, device=device, dtype=torch.uint8)
    return t, t.data_ptr(), nbytes


def _stream_handle(device, stream) -> int:
    s = torch.cuda.current_stream(device) if stream is None else stream
    return s.cuda_stream if isinstance(s, torch.cuda.Stream) else int(s)


def fem_softmax_fwd(q, k, v, beta, out=None, stream=None) -> torch.Tensor:
    """Causal softmax-prior FEM read.  q, k, v: [B, H, T, d] bf16 or fp32;
    beta: [H, d] fp32.  Returns out [B, H, T, d] fp32 (enqueued on ``stream``,
    default torch's current stream)."""
    lib = load()
    if q.dtype not in FEM_DTYPE:
        raise ValueError(f"unsupported dtype {q.dtype}")
    for name, x in (("q", q), ("k", k), ("v", v)):
        _dev_tensor(x, name, q.dtype)
        if x.dim() != 4 or x.shape != q.shape:
            raise ValueError(f"{name} must be [B, H, T, d] like q")
    B, H, T, d = q.shape
    _dev_tensor(beta, "beta", torch.float32)
    if tuple(beta.shape) != (H, d):
        raise ValueError("beta must be [H, d]")
    if out is None:
        out = torch.empty((B, H, T, d), device=q.device, dtype=torch.float32)
    _dev_tensor(out, "out", torch.float32)
    if tuple(out.shape) != (B, H, T, d):
        raise ValueError("out must be [B, H, T, d]")
    with torch.cuda.device(q.device):
        rc = lib.fem_softmax_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), beta.data_ptr(),
                                 out.data_ptr(), B, H, T, d, FEM_DTYPE[q.dtype],
                                 _stream_handle(q.device, stream))
    _check(rc)
    return out


def fem_softmax_fwd_ex(q, k, v, beta, out=None, causal: bool = True, out_dtype=torch.float32,
                       stream=None) -> torch.Tensor:
    """Variants of the softmax-prior read: causal or encoder (all keys),
    d_v = d_qk or d_qk / 2, fp32 or bf16 output.  q, k: [B, H, T, d_qk] bf16;
    v: [B, H, T, d_v] bf16; beta: [H, d_v] fp32.  Returns [B, H, T, d_v]."""
    lib = load()
    for name, x in (("q", q), ("k", k), ("v", v)):
        _dev_tensor(x, name, torch.bfloat16)
        if x.dim() != 4:
            raise ValueError(f"{name} must be [B, H, T, width]")
    if k.shape != q.shape or v.shape[:3] != q.shape[:3]:
        raise ValueError("q, k must be [B, H, T, d_qk] and v [B, H, T, d_v]")
    B, H, T, dqk = q.shape
    dv = v.shape[3]
    _dev_tensor(beta, "beta", torch.float32)
    if tuple(beta.shape) != (H, dv):
        raise ValueError("beta must be [H, d_v]")
    if out_dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("out_dtype must be float32 or bfloat16")
    if out is None:
        out = torch.empty((B, H, T, dv), device=q.device, dtype=out_dtype)
    _dev_tensor(out, "out", out_dtype)
    if tuple(out.shape) != (B, H, T, dv):
        raise ValueError("out must be [B, H, T, d_v]")
    flags = (0 if causal else FEM_FLAG_ENCODER) | \
        (FEM_FLAG_OUT_BF16 if out_dtype == torch.bfloat16 else 0)
    with torch.cuda.device(q.device):
        rc = lib.fem_softmax_fwd_ex(q.data_ptr(), k.data_ptr(), v.data_ptr(), beta.data_ptr(),
                                    out.data_ptr(), B, H, T, dqk, dv, flags, FEM_DTYPE[q.dtype],
                                    _stream_handle(q.device, stream))
    _check(rc)
    return out


def _decode_args(q, k_cache, v_cache, beta, lens, out):
    _dev_tensor(q, "q", torch.bfloat16)
    _dev_tensor(k_cache, "k_cache", torch.bfloat16)
    _dev_tensor(v_cache, "v_cache", torch.bfloat16)
    if q.dim() != 3 or k_cache.dim() != 4 or v_cache.dim() != 4:
        raise ValueError("q must be [B, H, d_qk], caches [B, H, L, width]")
    B, H, dqk = q.shape
    L = k_cache.shape[2]
    if tuple(k_cache.shape) != (B, H, L, dqk) or v_cache.shape[:3] != k_cache.shape[:3]:
        raise ValueError("k_cache must be [B, H, L, d_qk] and v_cache [B, H, L, d_v]")
    dv = v_cache.shape[3]
    _dev_tensor(beta, "beta", torch.float32)
    if tuple(beta.shape) != (H, dv):
        raise ValueError("beta must be [H, d_v]")
    if lens is not None:
        _dev_tensor(lens, "lens", torch.int32)
        if tuple(lens.shape) != (B,):
            raise ValueError("lens must be [B]")
    if out is None:
        out = torch.empty((B, H, dv), device=q.device, dtype=torch.float32)
    _dev_tensor(out, "out", torch.float32)
    if tuple(out.shape) != (B, H, dv):
        raise ValueError("out must be [B, H, d_v]")
    return B, H, L, dqk, dv, out


def fem_softmax_decode_noalloc(q, k_cache, v_cache, beta, lens=None, out=None,
                               stream=None) -> torch.Tensor:
    """fem_softmax_decode without a workspace: the library keeps the partial
    results in a fixed 8 MiB array per device (for callers that cannot
    allocate; overlapping calls on one device race).  Same arguments and
    result as fem_softmax_decode."""
    lib = load()
    B, H, L, dqk, dv, out = _decode_args(q, k_cache, v_cache, beta, lens, out)
    with torch.cuda.device(q.device):
        rc = lib.fem_softmax_decode_noalloc(q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
                                            None if lens is None else lens.data_ptr(),
                                            beta.data_ptr(), out.data_ptr(), B, H, L, dqk, dv,
                                            FEM_DTYPE[q.dtype], _stream_handle(q.device, stream))
    _check(rc)
    return out


def fem_softmax_decode(q, k_cache, v_cache, beta, lens=None, out=None, ws=None,
                       stream=None) -> torch.Tensor:
    """One decoding step: q [B, H, d_qk] reads the first lens[b] rows of the
    caches k_cache [B, H, L, d_qk], v_cache [B, H, L, d_v] (bf16).  lens: [B]
    int32 GPU tensor or None (all L).  ws: optional uint8 GPU workspace of at
    least fem_softmax_decode_workspace_bytes(...) bytes.  Returns [B, H, d_v]
    fp32."""
    lib = load()
    B, H, L, dqk, dv, out = _decode_args(q, k_cache, v_cache, beta, lens, out)
    need = lib.fem_softmax_decode_workspace_bytes(B, H, L, dqk, dv)
    with torch.cuda.device(q.device):
        wst, wsp, wsn = _workspace(need, q.device, ws, stream)
        rc = lib.fem_softmax_decode(q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
                                    None if lens is None else lens.data_ptr(), beta.data_ptr(),
                                    out.data_ptr(), B, H, L, dqk, dv, FEM_DTYPE[q.dtype],
                                    wsp, wsn, _stream_handle(q.device, stream))
    _check(rc)
    return out


def fem_softmax_gated_fwd(q, k, v, beta_max, lam, gate=None, out=None, stream=None) -> torch.Tensor:
    """Two-level gated read g * ((1 - lam) * mu + lam * F(beta_max)) with the
    causal softmax prior.  q, k, v: [B, H, T, d] bf16; beta_max: [H, d] fp32;
    lam, gate: [B, H, T, d] fp32 (gate None means g = 1).  Returns
    [B, H, T, d] fp32."""
    lib = load()
    for name, x in (("q", q), ("k", k), ("v", v)):
        _dev_tensor(x, name, torch.bfloat16)
        if x.dim() != 4 or x.shape != q.shape:
            raise ValueError(f"{name} must be [B, H, T, d] like q")
    B, H, T, d = q.shape
    _dev_tensor(beta_max, "beta_max", torch.float32)
    if tuple(beta_max.shape) != (H, d):
        raise ValueError("beta_max must be [H, d]")
    for name, x in (("lam", lam), ("gate", gate)):
        if x is None and name == "gate":
            continue
        _dev_tensor(x, name, torch.float32)
        if tuple(x.shape) != (B, H, T, d):
            raise ValueError(f"{name} must be [B, H, T, d]")
    if out is None:
        out = torch.empty((B, H, T, d), device=q.device, dtype=torch.float32)
    _dev_tensor(out, "out", torch.float32)
    if tuple(out.shape) != (B, H, T, d):
        raise ValueError("out must be [B, H, T, d]")
    with torch.cuda.device(q.device):
        rc = lib.fem_softmax_gated_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                       beta_max.data_ptr(), lam.data_ptr(),
                                       None if gate is None else gate.data_ptr(),
                                       out.data_ptr(), B, H, T, d, FEM_DTYPE[q.dtype],
                                       _stream_handle(q.device, stream))
    _check(rc)
    return out


def fem_linear_fwd(q, k, v, beta, out=None, chunk: int = 64, ws=None,
                   stream=None) -> torch.Tensor:
    """Causal linear-prior (phi = elu + 1) FEM read.  q, k: [B, H, T, d_k];
    v: [B, H, T, d_v] bf16; beta: [H, d_v] fp32; ws: optional uint8 GPU
    workspace of at least fem_linear_workspace_bytes(...) bytes.  Returns
    [B, H, T, d_v] fp32."""
    lib = load()
    if q.dtype not in FEM_DTYPE:
        raise ValueError(f"unsupported dtype {q.dtype}")
    _dev_tensor(q, "q", q.dtype)
    _dev_tensor(k, "k", q.dtype)
    _dev_tensor(v, "v", q.dtype)
    if q.dim() != 4 or k.shape != q.shape or v.dim() != 4 or v.shape[:3] != q.shape[:3]:
        raise ValueError("q, k must be [B, H, T, d_k] and v [B, H, T, d_v]")
    B, H, T, dk = q.shape
    dv = v.shape[3]
    _dev_tensor(beta, "beta", torch.float32)
    if tuple(beta.shape) != (H, dv):
        raise ValueError("beta must be [H, d_v]")
    if out is None:
        out = torch.empty((B, H, T, dv), device=q.device, dtype=torch.float32)
    _dev_tensor(out, "out", torch.float32)
    if tuple(out.shape) != (B, H, T, dv):
        raise ValueError("out must be [B, H, T, d_v]")
    need = lib.fem_linear_workspace_bytes(B, H, T, dk, dv, int(chunk))
    with torch.cuda.device(q.device):
        wst, wsp, wsn = _workspace(need, q.device, ws, stream)
        rc = lib.fem_linear_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), beta.data_ptr(),
                                out.data_ptr(), B, H, T, dk, dv, int(chunk),
                                FEM_DTYPE[q.dtype], wsp, wsn, _stream_handle(q.device, stream))
    _check(rc)
    return out


def fem_gla_fwd(q, k, v, g, beta, out=None, chunk: int = 64, ws=None,
                stream=None) -> torch.Tensor:
    """Causal GLA-prior FEM read.  q, k: [B, H, T, d_k] bf16; v: [B, H, T, d_v]
    bf16; g: [B, H, T, d_k] fp32 log-decays; beta: [H, d_v] fp32.  Returns
    [B, H, T, d_v] fp32."""
    lib = load()
    _dev_tensor(q, "q", torch.bfloat16)
    _dev_tensor(k, "k", torch.bfloat16)
    _dev_tensor(v, "v", torch.bfloat16)
    _dev_tensor(g, "g", torch.float32)
    if q.dim() != 4 or k.shape != q.shape or g.shape != q.shape or v.dim() != 4 or \
            v.shape[:3] != q.shape[:3]:
        raise ValueError("q, k, g must be [B, H, T, d_k] and v [B, H, T, d_v]")
    B, H, T, dk = q.shape
    dv = v.shape[3]
    _dev_tensor(beta, "beta", torch.float32)
    if tuple(beta.shape) != (H, dv):
        raise ValueError("beta must be [H, d_v]")
    if out is None:
        out = torch.empty((B, H, T, dv), device=q.device, dtype=torch.float32)
    _dev_tensor(out, "out", torch.float32)
    if tuple(out.shape) != (B, H, T, dv):
        raise ValueError("out must be [B, H, T, d_v]")
    need = lib.fem_gla_workspace_bytes(B, H, T, dk, dv, int(chunk))
    with torch.cuda.device(q.device):
        wst, wsp, wsn = _workspace(need, q.device, ws, stream)
        rc = lib.fem_gla_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), g.data_ptr(),
                             beta.data_ptr(), out.data_ptr(), B, H, T, dk, dv, int(chunk),
                             FEM_DTYPE[q.dtype], wsp, wsn, _stream_handle(q.device, stream))
    _check(rc)
    return out


def fem_softmax_fwd_train(q, k, v, beta, out=None, lse=None, stream=None):
    """fem_softmax_fwd (bf16) that also returns the prior's log-normaliser
    lse [B, H, T] fp32.  Returns (out, lse)."""
    lib = load()
    for name, x in (("q", q), ("k", k), ("v", v)):
        _dev_tensor(x, name, torch.bfloat16)
        if x.dim() != 4 or x.shape != q.shape:
            raise ValueError(f"{name} must be [B, H, T, d] like q")
    B, H, T, d = q.shape
    _dev_tensor(beta, "beta", torch.float32)
    if tuple(beta.shape) != (H, d):
        raise ValueError("beta must be [H, d]")
    out = torch.empty((B, H, T, d), device=q.device, dtype=torch.float32) if out is None else out
    lse = torch.empty((B, H, T), device=q.device, dtype=torch.float32) if lse is None else lse
    _dev_tensor(out, "out", torch.float32)
    _dev_tensor(lse, "lse", torch.float32)
    if tuple(out.shape) != (B, H, T, d) or tuple(lse.shape) != (B, H, T):
        raise ValueError("out must be [B, H, T, d] and lse [B, H, T]")
    with torch.cuda.device(q.device):
        rc = lib.fem_softmax_fwd_train(q.data_ptr(), k.data_ptr(), v.data_ptr(), beta.data_ptr(),
                                       out.data_ptr(), lse.data_ptr(), B, H, T, d,
                                       FEM_DTYPE[q.dtype], _stream_handle(q.device, stream))
    _check(rc)
    return out, lse


def fem_softmax_bwd(q, k, v, beta, out, lse, dout, ws=None, stream=None):
    """Gradients of sum(dout * out) w.r.t. q, k, v (fp32, shaped like them) and
    beta ([H, d], summed over batch and time).  ws: optional uint8 GPU
    workspace of at least fem_softmax_bwd_workspace_bytes(...) bytes.  Returns
    (dq, dk, dv, dbeta)."""
    lib = load()
    for name, x in (("q", q), ("k", k), ("v", v)):
        _dev_tensor(x, name, torch.bfloat16)
        if x.dim() != 4 or x.shape != q.shape:
            raise ValueError(f"{name} must be [B, H, T, d] like q")
    B, H, T, d = q.shape
    _dev_tensor(beta, "beta", torch.float32)
    for name, x, shp in (("out", out, (B, H, T, d)), ("lse", lse, (B, H, T)),
                         ("dout", dout, (B, H, T, d))):
        _dev_tensor(x, name, torch.float32)
        if tuple(x.shape) != shp:
            raise ValueError(f"{name} must be {list(shp)}")
    if tuple(beta.shape) != (H, d):
        raise ValueError("beta must be [H, d]")
    dq = torch.empty((B, H, T, d), device=q.device, dtype=torch.float32)
    dk = torch.empty_like(dq)
    dv = torch.empty_like(dq)
    db = torch.empty((H, d), device=q.device, dtype=torch.float32)
    need = lib.fem_softmax_bwd_workspace_bytes(B, H, T, d)
    with torch.cuda.device(q.device):
        wst, wsp, wsn = _workspace(need, q.device, ws, stream)
        rc = lib.fem_softmax_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), beta.data_ptr(),
                                 out.data_ptr(), lse.data_ptr(), dout.data_ptr(), dq.data_ptr(),
                                 dk.data_ptr(), dv.data_ptr(), db.data_ptr(), B, H, T, d,
                                 FEM_DTYPE[q.dtype], wsp, wsn, _stream_handle(q.device, stream))
    _check(rc)
    return dq, dk, dv, db


def workspace_bytes(entry: str, *sizes) -> int:
    """Exact workspace size (bytes) of the entry point ``entry`` ("linear",
    "gla", "decode" or "bwd") for the given size arguments, as in fem.h."""
    lib = load()
    fn = {"linear": lib.fem_linear_workspace_bytes, "gla": lib.fem_gla_workspace_bytes,
          "decode": lib.fem_softmax_decode_workspace_bytes,
          "bwd": lib.fem_softmax_bwd_workspace_bytes}[entry]
    return int(fn(*[int(x) for x in sizes]))
