"""Fused attention forward+backward for AMD Instinct MI355X (gfx950).

A thin ctypes binding over the C ABI of ``libattn_mi355x.so`` (declared in
``include/attn_mi355x.h``). The binding only marshals arguments: every step of
the computation runs in the library's HIP kernels. PyTorch provides device
memory and the current stream.

    O, L = attn_fwd(q, k, v, scale, causal)
    O, L, dQ, dK, dV = attn_fwd_bwd(q, k, v, do, scale, causal)
    O, L, P = attn_mat_fwd(q, k, v, scale, causal)          # naive path: P stored
    dQ, dK, dV = attn_mat_bwd(q, k, v, O, do, P, scale, causal)

Tensors are contiguous [B, H, n, d] on one GPU, all bfloat16 or all float32;
L is float32 [B, H, n] (natural-log log-sum-exp of the scaled, masked scores).
There is no fallback: if the library is missing or the device is not a GPU,
the call raises.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Tuple

import torch  # loads the process's HIP runtime before the library

__all__ = ["attn_fwd", "attn_fwd_bwd", "attn_fwd_bwd_timed", "attn_fwd_bwd_noalloc", "attn_noalloc_max_rows",
           "attn_bwd", "attn_workspace_bytes", "attn_strerror",
           "attn_mat_bytes", "attn_mat_lda", "attn_mat_fwd", "attn_mat_bwd", "attn_mat_fwd_bwd",
           "attn_fwd_bwd_atomic", "attn_workspace_bytes_atomic", "attn_decode", "attn_decode_workspace_bytes",
           "AttnError", "lib", "LIB_PATH", "ATTN_BF16", "ATTN_F32"]

# ATTN_MI355X_LIB may name another build of the same library (A/B comparison
# of compiler settings); by default the in-tree build is loaded.
LIB_PATH = os.environ.get("ATTN_MI355X_LIB") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "libattn_mi355x.so")
ATTN_BF16 = 0
ATTN_F32 = 1

_lib = None


class AttnError(RuntimeError):
    def __init__(self, code: int, where: str):
        super().__init__(f"{where} failed with code {code}: {attn_strerror(code)}")
        self.code = code


def lib() -> ctypes.CDLL:
    """Load libattn_mi355x.so (once) and declare the C signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2609_33916_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i, f, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    L.attn_workspace_bytes.argtypes = [i, i, i, i]
    L.attn_workspace_bytes.restype = sz
    L.attn_fwd.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, f, i, i, vp]
    L.attn_fwd.restype = i
    L.attn_fwd_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz,
                               i, i, i, i, f, i, i, vp]
    L.attn_fwd_bwd.restype = i
    L.attn_fwd_bwd_timed.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz,
                                     i, i, i, i, f, i, i, vp, ctypes.POINTER(vp)]
    L.attn_fwd_bwd_timed.restype = i
    L.attn_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, i, i, i, i, f, i, i, vp]
    L.attn_bwd.restype = i
    L.attn_noalloc_max_rows.argtypes = []
    L.attn_noalloc_max_rows.restype = sz
    L.attn_fwd_bwd_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, f, i, i, vp]
    L.attn_fwd_bwd_noalloc.restype = i
    L.attn_decode_workspace_bytes.argtypes = [i, i, i, i, i, i]
    L.attn_decode_workspace_bytes.restype = sz
    L.attn_decode.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, i, i, i, i, i, i, f, i, vp]
    L.attn_decode.restype = i
    L.attn_workspace_bytes_atomic.argtypes = [i, i, i, i]
    L.attn_workspace_bytes_atomic.restype = sz
    L.attn_fwd_bwd_atomic.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz,
                                      i, i, i, i, f, i, i, vp]
    L.attn_fwd_bwd_atomic.restype = i
    L.attn_mat_bytes.argtypes = [i, i, i, i]
    L.attn_mat_bytes.restype = sz
    L.attn_mat_fwd.argtypes = [vp, vp, vp, vp, vp, vp, sz, i, i, i, i, f, i, i, vp]
    L.attn_mat_fwd.restype = i
    L.attn_mat_bwd.argtypes = [vp, vp, vp, vp, vp, vp, sz, vp, vp, vp, vp, sz, i, i, i, i, f, i, i, vp]
    L.attn_mat_bwd.restype = i
    L.attn_mat_fwd_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, sz, vp, vp, vp, vp, sz,
                                   i, i, i, i, f, i, i, vp]
    L.attn_mat_fwd_bwd.restype = i
    L.attn_strerror.argtypes = [i]
    L.attn_strerror.restype = ctypes.c_char_p
    _lib = L
    return L


def attn_strerror(code: int) -> str:
    return lib().attn_strerror(int(code)).decode()


def attn_workspace_bytes(B: int, H: int, n: int, d: int) -> int:
    return int(lib().attn_workspace_bytes(B, H, n, d))


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return ATTN_BF16
    if t.dtype == torch.float32:
        return ATTN_F32
    raise TypeError(f"unsupported dtype {t.dtype} (bfloat16 or float32)")


def _check(name: str, t: torch.Tensor, ref: torch.Tensor) -> None:
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != ref.dtype or tuple(t.shape) != tuple(ref.shape) or t.device != ref.device:
        raise ValueError(f"{name} must match q in dtype, shape and device")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _check_out(name: str, t, shape, dtype: torch.dtype, ref: torch.Tensor) -> None:
    """An output the kernels write: a contiguous GPU tensor of exactly `shape`
    and `dtype` on q's device. The C ABI receives only its address, so a
    wrong size or a host tensor would be written out of bounds."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch.Tensor")
    if not t.is_cuda or t.device != ref.device:
        raise ValueError(f"{name} must be a GPU tensor on q's device")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _check_workspace(ws, nbytes: int, ref: torch.Tensor):
    """A caller-supplied workspace: contiguous, on q's GPU, at least `nbytes`.
    Returns (pointer, size in bytes)."""
    if not isinstance(ws, torch.Tensor):
        raise ValueError("workspace must be a torch.Tensor")
    if not ws.is_cuda or ws.device != ref.device:
        raise ValueError("workspace must be a GPU tensor on q's device")
    if not ws.is_contiguous():
        raise ValueError("workspace must be contiguous")
    size = ws.numel() * ws.element_size()
    if size < nbytes:
        raise ValueError(f"workspace holds {size} bytes, {nbytes} needed")
    return ws.data_ptr(), size


def _outputs(q: torch.Tensor, out, names):
    """Preallocated outputs checked against q (each `names` entry is 'x' for a
    tensor shaped like q, 'L' for the float32 [B, H, n] row vector), or new
    ones."""
    B, H, n, _ = q.shape
    if out is None:
        return tuple(torch.empty_like(q) if nm != "L" else
                     torch.empty((B, H, n), dtype=torch.float32, device=q.device) for nm in names)
    out = tuple(out)
    if len(out) != len(names):
        raise ValueError(f"out must hold {len(names)} tensors")
    for nm, t in zip(names, out):
        if nm == "L":
            _check_out("L", t, (B, H, n), torch.float32, q)
        else:
            _check_out(nm, t, q.shape, q.dtype, q)
    return out


def _stream(dev: torch.device) -> int:
    return torch.cuda.current_stream(dev).cuda_stream


def _scale(scale: Optional[float], d: int) -> float:
    return 1.0 / math.sqrt(d) if scale is None else float(scale)


def attn_fwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, scale: Optional[float] = None,
             causal: bool = False, out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None):
    """Forward pass: returns (O, L). ``scale`` defaults to 1/sqrt(d)."""
    if q.dim() != 4:
        raise ValueError("q must be [B, H, n, d]")
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check(name, t, q)
    B, H, n, d = q.shape
    O, L = _outputs(q, out, ("O", "L"))
    rc = lib().attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), O.data_ptr(), L.data_ptr(),
                        B, H, n, d, _scale(scale, d), int(bool(causal)), _dtype_code(q),
                        _stream(q.device))
    if rc != 0:
        raise AttnError(rc, "attn_fwd")
    return O, L


def attn_fwd_bwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, do: torch.Tensor,
                 scale: Optional[float] = None, causal: bool = False,
                 out: Optional[Tuple[torch.Tensor, ...]] = None,
                 workspace: Optional[torch.Tensor] = None):
    """Fused forward+backward: returns (O, L, dQ, dK, dV).

    ``out`` may supply preallocated (O, L, dQ, dK, dV) and ``workspace`` a
    uint8 GPU tensor of at least attn_workspace_bytes(B, H, n, d) bytes."""
    return _fwd_bwd(q, k, v, do, scale, causal, out, workspace, None)


def attn_noalloc_max_rows() -> int:
    """Largest B * H * n that attn_fwd_bwd_noalloc accepts."""
    return int(lib().attn_noalloc_max_rows())


def attn_fwd_bwd_noalloc(q, k, v, do, out, scale: Optional[float] = None, causal: bool = False):
    """attn_fwd_bwd without a workspace: the library's fixed per-GPU scratch
    holds the D and log-sum-exp rows, so the call allocates nothing. The
    outputs (O, L, dQ, dK, dV) must be preallocated and passed as ``out``.
    Calls that may overlap on one GPU race on the shared scratch."""
    if q.dim() != 4:
        raise ValueError("q must be [B, H, n, d]")
    for name, t in (("q", q), ("k", k), ("v", v), ("do", do)):
        _check(name, t, q)
    if out is None:
        raise ValueError("out (O, L, dQ, dK, dV) is required: this entry point allocates nothing")
    B, H, n, d = q.shape
    O, L, dQ, dK, dV = _outputs(q, out, ("O", "L", "dQ", "dK", "dV"))
    rc = lib().attn_fwd_bwd_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), do.data_ptr(),
                                    O.data_ptr(), L.data_ptr(), dQ.data_ptr(), dK.data_ptr(), dV.data_ptr(),
                                    B, H, n, d, _scale(scale, d), int(bool(causal)), _dtype_code(q),
                                    _stream(q.device))
    if rc != 0:
        raise AttnError(rc, "attn_fwd_bwd_noalloc")
    return O, L, dQ, dK, dV


def attn_bwd(q, k, v, o, lse, do, scale: Optional[float] = None, causal: bool = False,
             out=None, workspace=None):
    """Backward only from the forward's O and L: returns (dQ, dK, dV)."""
    if q.dim() != 4:
        raise ValueError("q must be [B, H, n, d]")
    for name, t in (("q", q), ("k", k), ("v", v), ("o", o), ("do", do)):
        _check(name, t, q)
    B, H, n, d = q.shape
    if lse.dtype != torch.float32 or tuple(lse.shape) != (B, H, n) or not lse.is_contiguous() \
            or lse.device != q.device:
        raise ValueError("lse must be contiguous float32 [B, H, n] on q's device")
    dQ, dK, dV = _outputs(q, out, ("dQ", "dK", "dV"))
    wsb = attn_workspace_bytes(B, H, n, d)
    if workspace is None:
        workspace = torch.empty(max(wsb, 1), dtype=torch.uint8, device=q.device)
    ws_ptr, ws_len = _check_workspace(workspace, wsb, q)
    rc = lib().attn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(),
                        do.data_ptr(), dQ.data_ptr(), dK.data_ptr(), dV.data_ptr(),
                        ws_ptr, ws_len,
                        B, H, n, d, _scale(scale, d), int(bool(causal)), _dtype_code(q),
                        _stream(q.device))
    if rc != 0:
        raise AttnError(rc, "attn_bwd")
    return dQ, dK, dV


def attn_fwd_bwd_timed(q, k, v, do, events, scale: Optional[float] = None, causal: bool = False,
                       out=None, workspace=None):
    """attn_fwd_bwd that records 4 caller-created hipEvent_t handles (ints)
    around its three kernels on the current stream."""
    if len(events) != 4:
        raise ValueError("events must hold 4 hipEvent_t handles")
    return _fwd_bwd(q, k, v, do, scale, causal, out, workspace, events)


def _fwd_bwd(q, k, v, do, scale, causal, out, workspace, events):
    if q.dim() != 4:
        raise ValueError("q must be [B, H, n, d]")
    for name, t in (("q", q), ("k", k), ("v", v), ("do", do)):
        _check(name, t, q)
    B, H, n, d = q.shape
    O, L, dQ, dK, dV = _outputs(q, out, ("O", "L", "dQ", "dK", "dV"))
    wsb = attn_workspace_bytes(B, H, n, d)
    if workspace is None:
        workspace = torch.empty(max(wsb, 1), dtype=torch.uint8, device=q.device)
    ws_ptr, ws_len = _check_workspace(workspace, wsb, q)
    args = (q.data_ptr(), k.data_ptr(), v.data_ptr(), do.data_ptr(),
            O.data_ptr(), L.data_ptr(), dQ.data_ptr(), dK.data_ptr(), dV.data_ptr(),
            ws_ptr, ws_len,
            B, H, n, d, _scale(scale, d), int(bool(causal)), _dtype_code(q), _stream(q.device))
    if events is None:
        rc = lib().attn_fwd_bwd(*args)
        where = "attn_fwd_bwd"
    else:
        arr = (ctypes.c_void_p * 4)(*events)
        rc = lib().attn_fwd_bwd_timed(*args, arr)
        where = "attn_fwd_bwd_timed"
    if rc != 0:
        raise AttnError(rc, where)
    return O, L, dQ, dK, dV


# ---------------------------------------------------------------- naive path --
def attn_mat_lda(n: int) -> int:
    """Row stride (elements) of the stored attention matrix: n rounded up to 128."""
    return (n + 127) // 128 * 128


def attn_mat_bytes(B: int, H: int, n: int, dtype: torch.dtype) -> int:
    code = ATTN_BF16 if dtype == torch.bfloat16 else ATTN_F32
    return int(lib().attn_mat_bytes(B, H, n, code))


def _mat_buffer(q: torch.Tensor, P: Optional[torch.Tensor]) -> torch.Tensor:
    B, H, n, _ = q.shape
    if P is None:
        return torch.empty((B, H, n, attn_mat_lda(n)), dtype=q.dtype, device=q.device)
    _check_out("P", P, (B, H, n, attn_mat_lda(n)), q.dtype, q)
    return P


def attn_mat_fwd(q, k, v, scale: Optional[float] = None, causal: bool = False, out=None, P=None):
    """Naive forward: returns (O, L, P); P is [B, H, n, attn_mat_lda(n)] with
    P[..., i, j] the attention probability of key j < n for query i."""
    if q.dim() != 4:
        raise ValueError("q must be [B, H, n, d]")
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check(name, t, q)
    B, H, n, d = q.shape
    O, L = _outputs(q, out, ("O", "L"))
    P = _mat_buffer(q, P)
    rc = lib().attn_mat_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), O.data_ptr(), L.data_ptr(),
                            P.data_ptr(), P.numel() * P.element_size(),
                            B, H, n, d, _scale(scale, d), int(bool(causal)), _dtype_code(q),
                            _stream(q.device))
    if rc != 0:
        raise AttnError(rc, "attn_mat_fwd")
    return O, L, P


def attn_mat_bwd(q, k, v, o, do, P, scale: Optional[float] = None, causal: bool = False,
                 out=None, workspace=None):
    """Naive backward from the stored P: returns (dQ, dK, dV)."""
    if q.dim() != 4:
        raise ValueError("q must be [B, H, n, d]")
    for name, t in (("q", q), ("k", k), ("v", v), ("o", o), ("do", do)):
        _check(name, t, q)
    B, H, n, d = q.shape
    if P is None:
        raise ValueError("P (the forward's stored attention matrix) is required")
    P = _mat_buffer(q, P)
    dQ, dK, dV = _outputs(q, out, ("dQ", "dK", "dV"))
    wsb = attn_workspace_bytes(B, H, n, d)
    if workspace is None:
        workspace = torch.empty(max(wsb, 1), dtype=torch.uint8, device=q.device)
    ws_ptr, ws_len = _check_workspace(workspace, wsb, q)
    rc = lib().attn_mat_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), do.data_ptr(),
                            P.data_ptr(), P.numel() * P.element_size(),
                            dQ.data_ptr(), dK.data_ptr(), dV.data_ptr(),
                            ws_ptr, ws_len,
                            B, H, n, d, _scale(scale, d), int(bool(causal)), _dtype_code(q),
                            _stream(q.device))
    if rc != 0:
        raise AttnError(rc, "attn_mat_bwd")
    return dQ, dK, dV


def attn_mat_fwd_bwd(q, k, v, do, scale: Optional[float] = None, causal: bool = False,
                     out=None, P=None, workspace=None):
    """Naive forward+backward: returns (O, L, dQ, dK, dV, P)."""
    if q.dim() != 4:
        raise ValueError("q must be [B, H, n, d]")
    for name, t in (("q", q), ("k", k), ("v", v), ("do", do)):
        _check(name, t, q)
    B, H, n, d = q.shape
    O, L, dQ, dK, dV = _outputs(q, out, ("O", "L", "dQ", "dK", "dV"))
    P = _mat_buffer(q, P)
    wsb = attn_workspace_bytes(B, H, n, d)
    if workspace is None:
        workspace = torch.empty(max(wsb, 1), dtype=torch.uint8, device=q.device)
    ws_ptr, ws_len = _check_workspace(workspace, wsb, q)
    rc = lib().attn_mat_fwd_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), do.data_ptr(),
                                O.data_ptr(), L.data_ptr(), P.data_ptr(), P.numel() * P.element_size(),
                                dQ.data_ptr(), dK.data_ptr(), dV.data_ptr(),
                                ws_ptr, ws_len,
                                B, H, n, d, _scale(scale, d), int(bool(causal)), _dtype_code(q),
                                _stream(q.device))
    if rc != 0:
        raise AttnError(rc, "attn_mat_fwd_bwd")
    return O, L, dQ, dK, dV, P


# ------------------------------------------------------------ atomic dQ --
def attn_workspace_bytes_atomic(B: int, H: int, n: int, d: int) -> int:
    return int(lib().attn_workspace_bytes_atomic(B, H, n, d))


def attn_fwd_bwd_atomic(q, k, v, do, scale: Optional[float] = None, causal: bool = False,
                        out=None, workspace=None):
    """Forward+backward with dQ accumulated by atomic adds in the dK/dV
    kernel (bfloat16 only): returns (O, L, dQ, dK, dV)."""
    if q.dim() != 4:
        raise ValueError("q must be [B, H, n, d]")
    for name, t in (("q", q), ("k", k), ("v", v), ("do", do)):
        _check(name, t, q)
    B, H, n, d = q.shape
    O, L, dQ, dK, dV = _outputs(q, out, ("O", "L", "dQ", "dK", "dV"))
    wsb = attn_workspace_bytes_atomic(B, H, n, d)
    if workspace is None:
        workspace = torch.empty(max(wsb, 16), dtype=torch.uint8, device=q.device)
    ws_ptr, ws_len = _check_workspace(workspace, wsb, q)
    rc = lib().attn_fwd_bwd_atomic(q.data_ptr(), k.data_ptr(), v.data_ptr(), do.data_ptr(),
                                   O.data_ptr(), L.data_ptr(), dQ.data_ptr(), dK.data_ptr(), dV.data_ptr(),
                                   ws_ptr, ws_len,
                                   B, H, n, d, _scale(scale, d), int(bool(causal)), _dtype_code(q),
                                   _stream(q.device))
    if rc != 0:
        raise AttnError(rc, "attn_fwd_bwd_atomic")
    return O, L, dQ, dK, dV


# --------------------------------------------------------------- decode --
def attn_decode_workspace_bytes(B: int, Hq: int, Hkv: int, n: int, d: int, append: bool = True) -> int:
    return int(lib().attn_decode_workspace_bytes(B, Hq, Hkv, n, d, int(bool(append))))


def attn_decode(q, k_cache, v_cache, k_new=None, v_new=None, cache_lens=None, n: Optional[int] = None,
                scale: Optional[float] = None, out=None, workspace=None):
    """One decode step: appends k_new/v_new ([B, Hkv, d]) at row cache_lens[b]
    of the caches ([B, Hkv, n_cap, d], updated in place) and attends q
    ([B, Hq, d]) to the first cache_lens[b] + 1 rows. cache_lens is an int32
    GPU tensor [B] or None (every sequence holds n tokens). Returns (O, L)."""
    if q.dim() != 3 or k_cache.dim() != 4:
        raise ValueError("q must be [B, Hq, d] and the caches [B, Hkv, n_cap, d]")
    B, Hq, d = q.shape
    Hkv, n_cap = k_cache.shape[1], k_cache.shape[2]
    for name, t in (("k_cache", k_cache), ("v_cache", v_cache)):
        if not t.is_cuda or t.device != q.device or t.dtype != q.dtype or tuple(t.shape) != (B, Hkv, n_cap, d) \
                or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous GPU tensor [B, Hkv, n_cap, d] of q's dtype")
    if not q.is_cuda or not q.is_contiguous():
        raise ValueError("q must be a contiguous GPU tensor")
    append = k_new is not None
    if append:
        for name, t in (("k_new", k_new), ("v_new", v_new)):
            if t is None or not t.is_cuda or t.device != q.device or t.dtype != q.dtype \
                    or tuple(t.shape) != (B, Hkv, d) or not t.is_contiguous():
                raise ValueError(f"{name} must be a contiguous GPU tensor [B, Hkv, d] of q's dtype")
    if cache_lens is not None:
        if not cache_lens.is_cuda or cache_lens.device != q.device or cache_lens.dtype != torch.int32 \
                or tuple(cache_lens.shape) != (B,) or not cache_lens.is_contiguous():
            raise ValueError("cache_lens must be an int32 GPU tensor [B]")
    if n is None:
        if cache_lens is None:
            raise ValueError("n is required without cache_lens")
        n = int(cache_lens.max().item())
    if out is None:
        O = torch.empty_like(q)
        L = torch.empty((B, Hq), dtype=torch.float32, device=q.device)
    else:
        if len(out) != 2:
            raise ValueError("out must hold (O, L)")
        O, L = out
        _check_out("O", O, (B, Hq, d), q.dtype, q)
        if L is not None:
            _check_out("L", L, (B, Hq), torch.float32, q)
    wsb = attn_decode_workspace_bytes(B, Hq, Hkv, n, d, append)
    if workspace is None and wsb > 0:
        workspace = torch.empty(wsb, dtype=torch.uint8, device=q.device)
    if workspace is not None:
        ws_ptr, ws_len = _check_workspace(workspace, wsb, q)
    else:
        ws_ptr, ws_len = None, 0
    rc = lib().attn_decode(q.data_ptr(), k_new.data_ptr() if append else None,
                           v_new.data_ptr() if append else None, k_cache.data_ptr(), v_cache.data_ptr(),
                           cache_lens.data_ptr() if cache_lens is not None else None,
                           O.data_ptr(), L.data_ptr() if L is not None else None, ws_ptr, ws_len,
                           B, Hq, Hkv, n, n_cap, d, _scale(scale, d), _dtype_code(q), _stream(q.device))
    if rc != 0:
        raise AttnError(rc, "attn_decode")
    return O, L
