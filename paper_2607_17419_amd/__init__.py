"""libkata: causal KATA-M1 attention (rank-one PSD feature map) on MI355X.

Thin Python binding over the C ABI in include/kata.h.  It only marshals torch
device tensors (pointers, sizes, the current HIP stream) into the library;
every step of the computation runs in the library's HIP kernels.  There is no
fallback: if libkata.so is missing or fails to load, every call raises.

    import paper_2607_17419_amd as kata
    out = kata.fwd_chunked(q, k, v, C=64)           # q, k: [B,H,T,d]; v: [B,H,T,dv]
    S, z = kata.prefill_state(k, v)                 # packed state after T tokens
    o = kata.decode_step(S, z, q1, k1, v1)          # one token per head, in place
"""
from __future__ import annotations

import ctypes
import os

__all__ = [
    "KataError", "lib", "fwd_chunked", "fwd_chunked_timed", "fwd_chunked_alloc", "workspace_bytes",
    "default_span", "prefill_state", "decode_step", "packed_dim", "LIB_PATH",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkata.so")

KATA_OK, KATA_ERR_INVALID_ARG, KATA_ERR_UNSUPPORTED, KATA_ERR_HIP = 0, 1, 2, 3
KATA_F32, KATA_BF16 = 0, 1

# every symbol include/kata.h declares
EXPORTED = (
    "kata_fwd_chunked", "kata_fwd_chunked_ws", "kata_fwd_chunked_timed", "kata_fwd_workspace_bytes",
    "kata_fwd_chunked_train_ws", "kata_bwd_chunked_ex",
    "kata_fwd_default_span", "kata_fwd_quadratic", "kata_fwd_quadratic_ws",
    "kata_fwd_quadratic_workspace_bytes", "kata_prefill_state", "kata_decode_step",
    "kata_mg_fwd_chunked", "kata_mg_fwd_chunked_ws", "kata_mg_fwd_chunked_timed",
    "kata_mg_fwd_workspace_bytes", "kata_mg_fwd_quadratic_ws",
    "kata_mg_fwd_quadratic_workspace_bytes", "kata_mg_prefill_state", "kata_mg_decode_step",
    "kata_lin_dim", "kata_lin_fwd_chunked", "kata_lin_fwd_chunked_ws",
    "kata_lin_fwd_chunked_timed", "kata_lin_fwd_workspace_bytes", "kata_lin_default_span",
    "kata_bwd_chunked", "kata_bwd_chunked_ws", "kata_bwd_chunked_timed",
    "kata_bwd_workspace_bytes", "kata_bwd_fused_scan",
    "kata_fwd_chunked_noalloc", "kata_noalloc_scratch_bytes",
    "kata_status_string", "kata_abi_version",
)

# kata_lin_feature_t
LIN_IDENTITY, LIN_RELU, LIN_ELU, LIN_LORENTZ, LIN_LORENTZ_S = 0, 1, 2, 3, 4


class KataError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {_status_name(status)} ({status})")


_lib = None


def lib():
    """The loaded libkata (ctypes.CDLL); raises if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libkata.so not found at {LIB_PATH}; run "
                          "`python -m paper_2607_17419_amd.build` first")
    L = ctypes.CDLL(LIB_PATH)
    vp, i, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    L.kata_fwd_chunked.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, i, vp]
    L.kata_fwd_chunked.restype = i
    L.kata_fwd_chunked_noalloc.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, i, vp]
    L.kata_fwd_chunked_noalloc.restype = i
    L.kata_noalloc_scratch_bytes.argtypes = []
    L.kata_noalloc_scratch_bytes.restype = sz
    L.kata_fwd_chunked_ws.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, i, i, vp, sz, vp]
    L.kata_fwd_chunked_ws.restype = i
    L.kata_fwd_chunked_timed.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, i, i, vp, sz, vp, vp]
    L.kata_fwd_chunked_timed.restype = i
    L.kata_fwd_chunked_train_ws.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, i, i, vp, sz, vp]
    L.kata_fwd_chunked_train_ws.restype = i
    L.kata_fwd_workspace_bytes.argtypes = [i, i, i, i, i, i, i, i]
    L.kata_fwd_workspace_bytes.restype = sz
    L.kata_fwd_default_span.argtypes = [i, i, i, i, i, i, i]
    L.kata_fwd_default_span.restype = i
    L.kata_prefill_state.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, vp]
    L.kata_prefill_state.restype = i
    L.kata_decode_step.argtypes = [vp, vp, vp, vp, vp, vp, i, i, i, i, i, vp]
    L.kata_decode_step.restype = i
    L.kata_fwd_quadratic.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, vp]
    L.kata_fwd_quadratic.restype = i
    L.kata_fwd_quadratic_ws.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, vp, sz, vp]
    L.kata_fwd_quadratic_ws.restype = i
    L.kata_fwd_quadratic_workspace_bytes.argtypes = [i, i, i, i, i, i]
    L.kata_fwd_quadratic_workspace_bytes.restype = sz
    L.kata_mg_fwd_chunked.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, i, i, vp]
    L.kata_mg_fwd_chunked.restype = i
    L.kata_mg_fwd_chunked_ws.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, i, i, i, vp, sz, vp]
    L.kata_mg_fwd_chunked_ws.restype = i
    L.kata_mg_fwd_chunked_timed.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, i, i, i, vp, sz,
                                            vp, vp]
    L.kata_mg_fwd_chunked_timed.restype = i
    L.kata_mg_fwd_workspace_bytes.argtypes = [i, i, i, i, i, i, i, i, i]
    L.kata_mg_fwd_workspace_bytes.restype = sz
    L.kata_mg_fwd_quadratic_ws.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, i, vp, sz, vp]
    L.kata_mg_fwd_quadratic_ws.restype = i
    L.kata_mg_fwd_quadratic_workspace_bytes.argtypes = [i, i, i, i, i, i, i]
    L.kata_mg_fwd_quadratic_workspace_bytes.restype = sz
    L.kata_mg_prefill_state.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, i, vp]
    L.kata_mg_prefill_state.restype = i
    L.kata_mg_decode_step.argtypes = [vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, vp]
    L.kata_mg_decode_step.restype = i
    f = ctypes.c_float
    L.kata_lin_dim.argtypes = [i, i]
    L.kata_lin_dim.restype = i
    L.kata_lin_fwd_chunked.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, i, f, i, i, vp]
    L.kata_lin_fwd_chunked.restype = i
    L.kata_lin_fwd_chunked_ws.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, i, f, i, i, i, vp,
                                          sz, vp]
    L.kata_lin_fwd_chunked_ws.restype = i
    L.kata_lin_fwd_chunked_timed.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, i, f, i, i, i, vp,
                                             sz, vp, vp]
    L.kata_lin_fwd_chunked_timed.restype = i
    L.kata_lin_fwd_workspace_bytes.argtypes = [i, i, i, i, i, i, i, i, i]
    L.kata_lin_fwd_workspace_bytes.restype = sz
    L.kata_lin_default_span.argtypes = [i, i, i, i, i, i, i, i]
    L.kata_lin_default_span.restype = i
    L.kata_bwd_chunked.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, i, i, vp]
    L.kata_bwd_chunked.restype = i
    L.kata_bwd_chunked_ws.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, i, i,
                                      vp, sz, vp]
    L.kata_bwd_chunked_ws.restype = i
    L.kata_bwd_chunked_timed.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, i, i,
                                         vp, sz, vp, vp]
    L.kata_bwd_chunked_timed.restype = i
    L.kata_bwd_chunked_ex.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, i, i,
                                      vp, sz, vp, vp]
    L.kata_bwd_chunked_ex.restype = i
    L.kata_bwd_workspace_bytes.argtypes = [i, i, i, i, i, i, i, i]
    L.kata_bwd_workspace_bytes.restype = sz
    L.kata_bwd_fused_scan.argtypes = [i, i, i, i, i, i, i, i]
    L.kata_bwd_fused_scan.restype = i
    L.kata_status_string.argtypes = [i]
    L.kata_status_string.restype = ctypes.c_char_p
    L.kata_abi_version.argtypes = []
    L.kata_abi_version.restype = i
    _lib = L
    return L


def _status_name(s: int) -> str:
    try:
        return lib().kata_status_string(s).decode()
    except Exception:  # library not loadable: still report the number
        return f"status {s}"


def _check(status: int, what: str):
    if status != KATA_OK:
        raise KataError(status, what)


def packed_dim(d: int) -> int:
    return d * (d + 1) // 2


def _dtype_code(t):
    import torch
    if t.dtype == torch.float32:
        return KATA_F32
    if t.dtype == torch.bfloat16:
        return KATA_BF16
    raise TypeError(f"q/k/v must be float32 or bfloat16, got {t.dtype}")


def _dev(t, name):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream, device):
    import torch
    s = torch.cuda.current_stream(device) if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _qkv_shapes(q, k, v):
    if q.dim() != 4 or k.shape != q.shape or v.dim() != 4 or v.shape[:3] != q.shape[:3]:
        raise ValueError(f"expected q,k [B,H,T,d] and v [B,H,T,dv]; got {tuple(q.shape)}, "
                         f"{tuple(k.shape)}, {tuple(v.shape)}")
    if not (q.dtype == k.dtype == v.dtype):
        raise TypeError("q, k and v must share one dtype")
    B, H, T, d = q.shape
    return B, H, T, d, v.shape[3]


def workspace_bytes(B, H, T, d, dv, C, dtype_code, span_chunks=0) -> int:
    return int(lib().kata_fwd_workspace_bytes(B, H, T, d, dv, C, dtype_code, span_chunks))


def default_span(B, H, T, d, dv, C, dtype_code) -> int:
    return int(lib().kata_fwd_default_span(B, H, T, d, dv, C, dtype_code))


def fwd_chunked(q, k, v, C: int, span_chunks: int = 0, out=None, workspace=None, stream=None):
    """Causal KATA-M1 forward via kata_fwd_chunked_ws; returns out [B,H,T,dv] fp32.

    The workspace is a torch uint8 device tensor (allocated here if not given).
    """
    import torch
    B, H, T, d, dv = _qkv_shapes(q, k, v)
    code = _dtype_code(q)
    if out is None:
        out = torch.empty((B, H, T, dv), dtype=torch.float32, device=q.device)
    nbytes = workspace_bytes(B, H, T, d, dv, C, code, span_chunks)
    if nbytes == 0:
        # let the library report why
        _check(lib().kata_fwd_chunked_ws(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"),
                                         _dev(out, "out"), B, H, T, d, dv, C, code,
                                         span_chunks, ctypes.c_void_p(0), 0,
                                         _stream(stream, q.device)), "kata_fwd_chunked_ws")
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=q.device)
    _check(lib().kata_fwd_chunked_ws(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(out, "out"),
                                     B, H, T, d, dv, C, code, span_chunks,
                                     _dev(workspace, "workspace"), workspace.numel(),
                                     _stream(stream, q.device)), "kata_fwd_chunked_ws")
    return out


def fwd_chunked_timed(q, k, v, C: int, events, span_chunks: int = 0, out=None, workspace=None,
                      stream=None):
    """fwd_chunked that also records 4 caller-created HIP events (a ctypes array
    of 4 void pointers) around the three stages on the launch stream."""
    import torch
    B, H, T, d, dv = _qkv_shapes(q, k, v)
    code = _dtype_code(q)
    if out is None:
        out = torch.empty((B, H, T, dv), dtype=torch.float32, device=q.device)
    nbytes = workspace_bytes(B, H, T, d, dv, C, code, span_chunks)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=q.device)
    _check(lib().kata_fwd_chunked_timed(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"),
                                        _dev(out, "out"), B, H, T, d, dv, C, code, span_chunks,
                                        _dev(workspace, "workspace"), workspace.numel(),
                                        events, _stream(stream, q.device)),
           "kata_fwd_chunked_timed")
    return out


def fwd_chunked_train(q, k, v, C: int, span_chunks: int = 0, out=None, den=None, workspace=None,
                      stream=None):
    """Forward via kata_fwd_chunked_train_ws, which also writes the row
    denominators D_t for the backward; returns (out [B,H,T,dv], den [B,H,T])
    fp32."""
    import torch
    B, H, T, d, dv = _qkv_shapes(q, k, v)
    code = _dtype_code(q)
    if out is None:
        out = torch.empty((B, H, T, dv), dtype=torch.float32, device=q.device)
    if den is None:
        den = torch.empty((B, H, T), dtype=torch.float32, device=q.device)
    nbytes = workspace_bytes(B, H, T, d, dv, C, code, span_chunks)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=q.device)
    _check(lib().kata_fwd_chunked_train_ws(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"),
                                           _dev(out, "out"), _dev(den, "den"), B, H, T, d, dv, C,
                                           code, span_chunks, _dev(workspace, "workspace"),
                                           workspace.numel(), _stream(stream, q.device)),
           "kata_fwd_chunked_train_ws")
    return out, den


def fwd_chunked_alloc(q, k, v, C: int, out=None, stream=None):
    """Causal forward via kata_fwd_chunked (library allocates its workspace
    stream-ordered); returns out [B,H,T,dv] fp32."""
    import torch
    B, H, T, d, dv = _qkv_shapes(q, k, v)
    code = _dtype_code(q)
    if out is None:
        out = torch.empty((B, H, T, dv), dtype=torch.float32, device=q.device)
    _check(lib().kata_fwd_chunked(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(out, "out"),
                                  B, H, T, d, dv, C, code, _stream(stream, q.device)),
           "kata_fwd_chunked")
    return out


def noalloc_scratch_bytes() -> int:
    return int(lib().kata_noalloc_scratch_bytes())


def fwd_chunked_noalloc(q, k, v, C: int, out=None, stream=None):
    """Causal forward via kata_fwd_chunked_noalloc (workspace in the library's
    per-device scratch array, nothing allocated by the library); returns out
    [B,H,T,dv] fp32 (allocated here by torch if not given)."""
    import torch
    B, H, T, d, dv = _qkv_shapes(q, k, v)
    code = _dtype_code(q)
    if out is None:
        out = torch.empty((B, H, T, dv), dtype=torch.float32, device=q.device)
    _check(lib().kata_fwd_chunked_noalloc(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"),
                                          _dev(out, "out"), B, H, T, d, dv, C, code,
                                          _stream(stream, q.device)),
           "kata_fwd_chunked_noalloc")
    return out


def quadratic_workspace_bytes(B, H, T, d, dv, dtype_code) -> int:
    return int(lib().kata_fwd_quadratic_workspace_bytes(B, H, T, d, dv, dtype_code))


def fwd_quadratic(q, k, v, out=None, workspace=None, stream=None):
    """Causal KATA-M1 forward in the quadratic form via kata_fwd_quadratic_ws;
    returns out [B,H,T,dv] fp32.  The workspace (a torch uint8 device tensor)
    is allocated here if not given."""
    import torch
    B, H, T, d, dv = _qkv_shapes(q, k, v)
    code = _dtype_code(q)
    if out is None:
        out = torch.empty((B, H, T, dv), dtype=torch.float32, device=q.device)
    nbytes = quadratic_workspace_bytes(B, H, T, d, dv, code)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=q.device)
    _check(lib().kata_fwd_quadratic_ws(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"),
                                       _dev(out, "out"), B, H, T, d, dv, code,
                                       _dev(workspace, "workspace"), workspace.numel(),
                                       _stream(stream, q.device)), "kata_fwd_quadratic_ws")
    return out


def fwd_quadratic_alloc(q, k, v, out=None, stream=None):
    """Quadratic forward via kata_fwd_quadratic (library allocates its
    workspace stream-ordered); returns out [B,H,T,dv] fp32."""
    import torch
    B, H, T, d, dv = _qkv_shapes(q, k, v)
    code = _dtype_code(q)
    if out is None:
        out = torch.empty((B, H, T, dv), dtype=torch.float32, device=q.device)
    _check(lib().kata_fwd_quadratic(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(out, "out"),
                                    B, H, T, d, dv, code, _stream(stream, q.device)),
           "kata_fwd_quadratic")
    return out


def prefill_state(k, v, S=None, z=None, stream=None):
    """Packed state after all T tokens: S [B,H,n,dv], z [B,H,n] (fp32)."""
    import torch
    if k.dim() != 4 or v.dim() != 4 or v.shape[:3] != k.shape[:3] or k.dtype != v.dtype:
        raise ValueError("expected k [B,H,T,d] and v [B,H,T,dv] of one dtype")
    B, H, T, d = k.shape
    dv = v.shape[3]
    n = packed_dim(d)
    if S is None:
        S = torch.empty((B, H, n, dv), dtype=torch.float32, device=k.device)
    if z is None:
        z = torch.empty((B, H, n), dtype=torch.float32, device=k.device)
    _check(lib().kata_prefill_state(_dev(k, "k"), _dev(v, "v"), _dev(S, "S"), _dev(z, "z"),
                                    B, H, T, d, dv, _dtype_code(k), _stream(stream, k.device)),
           "kata_prefill_state")
    return S, z


def decode_step(S, z, q, k, v, out=None, stream=None):
    """One decode step (S, z updated in place); q, k [B,H,d], v [B,H,dv] -> out [B,H,dv]."""
    import torch
    if q.dim() != 3 or k.shape != q.shape or v.dim() != 3 or v.shape[:2] != q.shape[:2]:
        raise ValueError("expected q, k [B,H,d] and v [B,H,dv]")
    if not (q.dtype == k.dtype == v.dtype):
        raise TypeError("q, k and v must share one dtype")
    B, H, d = q.shape
    dv = v.shape[2]
    if out is None:
        out = torch.empty((B, H, dv), dtype=torch.float32, device=q.device)
    _check(lib().kata_decode_step(_dev(S, "S"), _dev(z, "z"), _dev(q, "q"), _dev(k, "k"),
                                  _dev(v, "v"), _dev(out, "out"), B, H, d, dv, _dtype_code(q),
                                  _stream(stream, q.device)), "kata_decode_step")
    return out


# ---- KATA-Mg (g feature blocks of d/g coordinates; g = 1 is KATA-M1) ------------

def packed_dim_mg(d: int, g: int) -> int:
    m = d // g
    return g * (m * (m + 1) // 2)


def mg_workspace_bytes(B, H, T, d, dv, C, g, dtype_code, span_chunks=0) -> int:
    return int(lib().kata_mg_fwd_workspace_bytes(B, H, T, d, dv, C, g, dtype_code, span_chunks))


def mg_fwd_chunked(q, k, v, C: int, g: int, span_chunks: int = 0, out=None, workspace=None,
                   stream=None):
    """Causal KATA-Mg forward via kata_mg_fwd_chunked_ws; returns out [B,H,T,dv] fp32."""
    import torch
    B, H, T, d, dv = _qkv_shapes(q, k, v)
    code = _dtype_code(q)
    if out is None:
        out = torch.empty((B, H, T, dv), dtype=torch.float32, device=q.device)
    nbytes = mg_workspace_bytes(B, H, T, d, dv, C, g, code, span_chunks)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=q.device)
    _check(lib().kata_mg_fwd_chunked_ws(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"),
                                        _dev(out, "out"), B, H, T, d, dv, C, g, code, span_chunks,
                                        _dev(workspace, "workspace"), workspace.numel(),
                                        _stream(stream, q.device)), "kata_mg_fwd_chunked_ws")
    return out


def mg_fwd_chunked_timed(q, k, v, C: int, g: int, events, span_chunks: int = 0, out=None,
                         workspace=None, stream=None):
    """mg_fwd_chunked that also records 4 caller-created HIP events around the
    three stages on the launch stream."""
    import torch
    B, H, T, d, dv = _qkv_shapes(q, k, v)
    code = _dtype_code(q)
    if out is None:
        out = torch.empty((B, H, T, dv), dtype=torch.float32, device=q.device)
    nbytes = mg_workspace_bytes(B, H, T, d, dv, C, g, code, span_chunks)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=q.device)
    _check(lib().kata_mg_fwd_chunked_timed(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"),
                                           _dev(out, "out"), B, H, T, d, dv, C, g, code,
                                           span_chunks, _dev(workspace, "workspace"),
                                           workspace.numel(), events, _stream(stream, q.device)),
           "kata_mg_fwd_chunked_timed")
    return out


def mg_fwd_chunked_alloc(q, k, v, C: int, g: int, out=None, stream=None):
    """KATA-Mg forward via kata_mg_fwd_chunked (stream-ordered library workspace)."""
    import torch
    B, H, T, d, dv = _qkv_shapes(q, k, v)
    code = _dtype_code(q)
    if out is None:
        out = torch.empty((B, H, T, dv), dtype=torch.float32, device=q.device)
    _check(lib().kata_mg_fwd_chunked(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(out, "out"),
                                     B, H, T, d, dv, C, g, code, _stream(stream, q.device)),
           "kata_mg_fwd_chunked")
    return out


def mg_fwd_quadratic(q, k, v, g: int, out=None, workspace=None, stream=None):
    """KATA-Mg forward in the quadratic form via kata_mg_fwd_quadratic_ws."""
    import torch
    B, H, T, d, dv = _qkv_shapes(q, k, v)
    code = _dtype_code(q)
    if out is None:
        out = torch.empty((B, H, T, dv), dtype=torch.float32, device=q.device)
    nbytes = int(lib().kata_mg_fwd_quadratic_workspace_bytes(B, H, T, d, dv, g, code))
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=q.device)
    _check(lib().kata_mg_fwd_quadratic_ws(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"),
                                          _dev(out, "out"), B, H, T, d, dv, g, code,
                                          _dev(workspace, "workspace"), workspace.numel(),
                                          _stream(stream, q.device)), "kata_mg_fwd_quadratic_ws")
    return out


def mg_prefill_state(k, v, g: int, S=None, z=None, stream=None):
    """KATA-Mg packed state after all T tokens: S [B,H,n_g,dv], z [B,H,n_g] (fp32)."""
    import torch
    if k.dim() != 4 or v.dim() != 4 or v.shape[:3] != k.shape[:3] or k.dtype != v.dtype:
        raise ValueError("expected k [B,H,T,d] and v [B,H,T,dv] of one dtype")
    B, H, T, d = k.shape
    dv = v.shape[3]
    n = packed_dim_mg(d, g)
    if S is None:
        S = torch.empty((B, H, n, dv), dtype=torch.float32, device=k.device)
    if z is None:
        z = torch.empty((B, H, n), dtype=torch.float32, device=k.device)
    _check(lib().kata_mg_prefill_state(_dev(k, "k"), _dev(v, "v"), _dev(S, "S"), _dev(z, "z"),
                                       B, H, T, d, dv, g, _dtype_code(k),
                                       _stream(stream, k.device)), "kata_mg_prefill_state")
    return S, z


def mg_decode_step(S, z, q, k, v, g: int, out=None, stream=None):
    """One KATA-Mg decode step (S, z updated in place) -> out [B,H,dv]."""
    import torch
    if q.dim() != 3 or k.shape != q.shape or v.dim() != 3 or v.shape[:2] != q.shape[:2]:
        raise ValueError("expected q, k [B,H,d] and v [B,H,dv]")
    if not (q.dtype == k.dtype == v.dtype):
        raise TypeError("q, k and v must share one dtype")
    B, H, d = q.shape
    dv = v.shape[2]
    if out is None:
        out = torch.empty((B, H, dv), dtype=torch.float32, device=q.device)
    _check(lib().kata_mg_decode_step(_dev(S, "S"), _dev(z, "z"), _dev(q, "q"), _dev(k, "k"),
                                     _dev(v, "v"), _dev(out, "out"), B, H, d, dv, g,
                                     _dtype_code(q), _stream(stream, q.device)),
           "kata_mg_decode_step")
    return out


# ---- linear features --------------------------------------------------------

def lin_dim(d: int, feature: int) -> int:
    return int(lib().kata_lin_dim(d, feature))


def lin_workspace_bytes(B, H, T, d, dv, C, feature, dtype_code, span_chunks=0) -> int:
    return int(lib().kata_lin_fwd_workspace_bytes(B, H, T, d, dv, C, feature, dtype_code,
                                                  span_chunks))


def lin_default_span(B, H, T, d, dv, C, feature, dtype_code) -> int:
    return int(lib().kata_lin_default_span(B, H, T, d, dv, C, feature, dtype_code))


def lin_fwd_chunked(q, k, v, C: int, feature: int, eps: float = 0.0, normalize: bool = True,
                    span_chunks: int = 0, out=None, workspace=None, stream=None, events=None):
    """Causal linear attention with a linear feature map via kata_lin_fwd_chunked_ws
    (or kata_lin_fwd_chunked_timed when `events`, a ctypes array of 4 HIP events,
    is given); returns out [B,H,T,dv] fp32."""
    import torch
    B, H, T, d, dv = _qkv_shapes(q, k, v)
    code = _dtype_code(q)
    if out is None:
        out = torch.empty((B, H, T, dv), dtype=torch.float32, device=q.device)
    nbytes = lin_workspace_bytes(B, H, T, d, dv, C, feature, code, span_chunks)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=q.device)
    args = (_dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(out, "out"), B, H, T, d, dv, C,
            feature, float(eps), int(normalize), code, span_chunks, _dev(workspace, "workspace"),
            workspace.numel())
    if events is None:
        _check(lib().kata_lin_fwd_chunked_ws(*args, _stream(stream, q.device)),
               "kata_lin_fwd_chunked_ws")
    else:
        _check(lib().kata_lin_fwd_chunked_timed(*args, events, _stream(stream, q.device)),
               "kata_lin_fwd_chunked_timed")
    return out


def lin_fwd_chunked_alloc(q, k, v, C: int, feature: int, eps: float = 0.0,
                          normalize: bool = True, out=None, stream=None):
    """The same forward via kata_lin_fwd_chunked (stream-ordered library workspace)."""
    import torch
    B, H, T, d, dv = _qkv_shapes(q, k, v)
    code = _dtype_code(q)
    if out is None:
        out = torch.empty((B, H, T, dv), dtype=torch.float32, device=q.device)
    _check(lib().kata_lin_fwd_chunked(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(out, "out"),
                                      B, H, T, d, dv, C, feature, float(eps), int(normalize),
                                      code, _stream(stream, q.device)), "kata_lin_fwd_chunked")
    return out


# ---- backward -----------------------------------------------------------------

def bwd_workspace_bytes(B, H, T, d, dv, C, g, dtype_code) -> int:
    return int(lib().kata_bwd_workspace_bytes(B, H, T, d, dv, C, g, dtype_code))


def bwd_fused_scan(B, H, T, d, dv, C, g, dtype_code) -> int:
    """1 when the backward's state launches also scan (kata_bwd_fused_scan)."""
    return int(lib().kata_bwd_fused_scan(B, H, T, d, dv, C, g, dtype_code))


def bwd_chunked(q, k, v, out, dout, C: int, g: int = 1, workspace=None, stream=None,
                events=None, grads=None, den=None):
    """Gradients (dq, dk, dv) of the causal KATA-Mg forward (g = 1: M1) via
    kata_bwd_chunked_ws (or kata_bwd_chunked_timed when `events`, a ctypes
    array of 7 HIP events, is given; or kata_bwd_chunked_ex when `den`, the
    denominators from fwd_chunked_train, is given); fp32 tensors shaped like
    q, k, v."""
    import torch
    B, H, T, d, dv = _qkv_shapes(q, k, v)
    code = _dtype_code(q)
    for name, t in (("out", out), ("dout", dout)):
        if t.dtype != torch.float32 or tuple(t.shape) != (B, H, T, dv):
            raise ValueError(f"{name} must be fp32 [B,H,T,dv]")
    if grads is None:
        grads = (torch.empty((B, H, T, d), dtype=torch.float32, device=q.device),
                 torch.empty((B, H, T, d), dtype=torch.float32, device=q.device),
                 torch.empty((B, H, T, dv), dtype=torch.float32, device=q.device))
    dq, dk, dvv = grads
    nbytes = bwd_workspace_bytes(B, H, T, d, dv, C, g, code)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=q.device)
    args = (_dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(out, "out"), _dev(dout, "dout"),
            _dev(dq, "dq"), _dev(dk, "dk"), _dev(dvv, "dv"), B, H, T, d, dv, C, g, code,
            _dev(workspace, "workspace"), workspace.numel())
    if den is not None:
        if den.dtype != torch.float32 or tuple(den.shape) != (B, H, T):
            raise ValueError("den must be fp32 [B,H,T]")
        args_ex = args[:5] + (_dev(den, "den"),) + args[5:]
        _check(lib().kata_bwd_chunked_ex(*args_ex, events if events is not None else None,
                                         _stream(stream, q.device)), "kata_bwd_chunked_ex")
    elif events is None:
        _check(lib().kata_bwd_chunked_ws(*args, _stream(stream, q.device)), "kata_bwd_chunked_ws")
    else:
        _check(lib().kata_bwd_chunked_timed(*args, events, _stream(stream, q.device)),
               "kata_bwd_chunked_timed")
    return dq, dk, dvv


def bwd_chunked_alloc(q, k, v, out, dout, C: int, g: int = 1, stream=None):
    """The same gradients via kata_bwd_chunked (stream-ordered library workspace)."""
    import torch
    B, H, T, d, dv = _qkv_shapes(q, k, v)
    code = _dtype_code(q)
    dq = torch.empty((B, H, T, d), dtype=torch.float32, device=q.device)
    dk = torch.empty((B, H, T, d), dtype=torch.float32, device=q.device)
    dvv = torch.empty((B, H, T, dv), dtype=torch.float32, device=q.device)
    _check(lib().kata_bwd_chunked(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(out, "out"),
                                  _dev(dout, "dout"), _dev(dq, "dq"), _dev(dk, "dk"),
                                  _dev(dvv, "dv"), B, H, T, d, dv, C, g, code,
                                  _stream(stream, q.device)), "kata_bwd_chunked")
    return dq, dk, dvv
