"""Thin Python binding of ``libfoe.so`` (C ABI in ``include/foe.h``).

Argument marshalling only: tensors are passed as device pointers plus the
current HIP stream, and every step of the block runs in the library's HIP
kernels.  PyTorch provides device memory and streams.  There is no fallback:
if the library is missing or a tensor is not a contiguous GPU tensor of the
right dtype, the call raises.
"""

from __future__ import annotations

import ctypes
import os

import torch

F32 = 0
BF16 = 1
GATE_RENORM = 0   # foe_gating
GATE_GLOBAL = 1

FOE_OK = 0
FOE_ERR_INVALID = -1
FOE_ERR_UNSUPPORTED = -2
FOE_ERR_WORKSPACE = -3
FOE_ERR_HIP = -4

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfoe.so")

_c_int, _c_float, _c_size = ctypes.c_int, ctypes.c_float, ctypes.c_size_t
_p = ctypes.c_void_p

_SIGNATURES = {
    "foe_route": (_c_int, [_c_int, _c_int, _c_int, _c_int, _c_int, _p, _p, _p, _p, _p, _p]),
    "foe_route_ex": (_c_int, [_c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _p, _p, _p,
                              _p, _p, _p]),
    "foe_permute": (_c_int, [_c_int, _c_int, _c_int, _c_int, _c_int, _p, _p, _p, _p, _p, _p, _p,
                             _p, _c_size, _p]),
    "foe_expert_ffn": (_c_int, [_c_int, _c_int, _c_int, _c_int, _c_int, _p, _p, _p, _p, _p, _p,
                                _p, _c_size, _p]),
    "foe_combine": (_c_int, [_c_int, _c_int, _c_int, _c_int, _p, _p, _p, _p, _p, _p]),
    "foe_reduce": (_c_int, [_c_int, _c_int, _c_int, _c_int, _p, _p, _c_float, _p, _p]),
    "foe_cluster_block": (_c_int, [_c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _p, _p,
                                   _p, _p, _p, _p, _c_float, _p, _p, _c_size, _p]),
    "foe_cluster_block_ex": (_c_int, [_c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int,
                                      _c_int, _p, _p, _p, _p, _p, _p, _c_float, _p, _p, _c_size,
                                      _p]),
    "foe_cluster_block_noalloc": (_c_int, [_c_int, _c_int, _c_int, _c_int, _c_int, _c_int,
                                           _c_int, _p, _p, _p, _p, _p, _p, _c_float, _p, _p]),
    "foe_workspace_bytes": (_c_size, [ctypes.c_char_p, _c_int, _c_int, _c_int, _c_int, _c_int,
                                      _c_int, _c_int]),
    "foe_group_attention": (_c_int, [_c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_float,
                                     _c_float, _p, _p, _p, _p, _p, _c_size, _p]),
    "foe_group_attention_workspace_bytes": (_c_size, [_c_int, _c_int, _c_int, _c_int, _c_int]),
    "foe_last_error": (ctypes.c_char_p, []),
    "foe_profile_enable": (_c_int, [_c_int]),
    "foe_profile_reset": (_c_int, []),
    "foe_profile_kernel": (_c_int, [ctypes.c_char_p, ctypes.POINTER(_c_int),
                                    ctypes.POINTER(ctypes.c_double)]),
    "foe_profile_names": (_c_int, [ctypes.c_char_p, _c_size]),
}

_lib = None


class FoeError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"[status {status}] {msg}")
        self.status = status


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2605_06206_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def last_error():
    return lib().foe_last_error().decode()


def _check(rc, name):
    if rc != FOE_OK:
        raise FoeError(rc, f"{name}: {last_error()}")


def _dt(t):
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype} (bf16 or fp32)")


def _dev(t, name, dtype=None):
    """Device pointer of a contiguous GPU tensor (None -> NULL)."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def workspace_bytes(op, dt, C=0, T=0, d=0, E=0, k=0, F=0):
    n = lib().foe_workspace_bytes(op.encode(), dt, C, T, d, E, k, F)
    if n == ctypes.c_size_t(-1).value:
        raise FoeError(FOE_ERR_INVALID, f"foe_workspace_bytes({op}): {last_error()}")
    return n


def _workspace(ws, nbytes, device):
    if ws is None or ws.numel() < nbytes:
        ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)
    return ws


def _gating(gating):
    codes = {"renorm": GATE_RENORM, "global": GATE_GLOBAL}
    if gating not in codes:
        raise ValueError(f"gating must be 'renorm' or 'global', got {gating!r}")
    return codes[gating]


def route(x, w_router, bias, k, topk_idx=None, topk_w=None, stream=None, gating="renorm"):
    """foe_route (w_router [E,d]) or foe_route_ex (w_router [G,E,d], or a
    gating other than "renorm"): returns (topk_idx, topk_w), [T,k] or [G,T,k]."""
    T, d = x.shape
    grouped = w_router.dim() == 3
    G = w_router.shape[0] if grouped else 1
    E = w_router.shape[-2]
    dt = _dt(x)
    shape = (G, T, k) if grouped else (T, k)
    if topk_idx is None:
        topk_idx = torch.empty(shape, dtype=torch.int32, device=x.device)
    if topk_w is None:
        topk_w = torch.empty(shape, dtype=torch.float32, device=x.device)
    args = (_dev(x, "x"), _dev(w_router, "w_router", x.dtype), _dev(bias, "bias", torch.float32),
            _dev(topk_idx, "topk_idx", torch.int32), _dev(topk_w, "topk_w", torch.float32),
            _stream(stream))
    if not grouped and gating == "renorm":
        _check(lib().foe_route(dt, T, d, E, k, *args), "foe_route")
    else:
        _check(lib().foe_route_ex(dt, G, T, d, E, k, _gating(gating), *args), "foe_route_ex")
    return topk_idx, topk_w


def permute(topk_idx, x, E, ws=None, stream=None, with_counts=True):
    """foe_permute: returns dict(counts, offsets, sorted_src, row_of, x_perm)."""
    T, k = topk_idx.shape
    d = x.shape[1]
    dt = _dt(x)
    dev = x.device
    R = T * k
    out = {
        "counts": torch.empty(E, dtype=torch.int32, device=dev) if with_counts else None,
        "offsets": torch.empty(E + 1, dtype=torch.int32, device=dev),
        "sorted_src": torch.empty(R, dtype=torch.int32, device=dev),
        "row_of": torch.empty(R, dtype=torch.int32, device=dev),
        "x_perm": torch.empty((R, d), dtype=x.dtype, device=dev),
    }
    need = workspace_bytes("permute", dt, 1, T, d, E, k, 0)
    ws = _workspace(ws, need, dev)
    rc = lib().foe_permute(dt, T, d, E, k, _dev(topk_idx, "topk_idx", torch.int32), _dev(x, "x"),
                           _dev(out["counts"], "counts"), _dev(out["offsets"], "offsets"),
                           _dev(out["sorted_src"], "sorted_src"), _dev(out["row_of"], "row_of"),
                           _dev(out["x_perm"], "x_perm"), _dev(ws, "ws"), ws.numel(),
                           _stream(stream))
    _check(rc, "foe_permute")
    return out


def expert_ffn(x_perm, offsets, w_gate, w_up, w_down, y_perm=None, ws=None, stream=None):
    """foe_expert_ffn: returns y_perm [rows,d]."""
    rows, d = x_perm.shape
    E, F, _ = w_gate.shape
    dt = _dt(x_perm)
    if y_perm is None:
        y_perm = torch.empty((rows, d), dtype=x_perm.dtype, device=x_perm.device)
    need = workspace_bytes("expert_ffn", dt, 1, rows, d, E, 1, F)
    ws = _workspace(ws, need, x_perm.device)
    rc = lib().foe_expert_ffn(dt, E, d, F, rows, _dev(x_perm, "x_perm"),
                              _dev(offsets, "offsets", torch.int32),
                              _dev(w_gate, "w_gate", x_perm.dtype), _dev(w_up, "w_up", x_perm.dtype),
                              _dev(w_down, "w_down", x_perm.dtype),
                              _dev(y_perm, "y_perm", x_perm.dtype), _dev(ws, "ws"), ws.numel(),
                              _stream(stream))
    _check(rc, "foe_expert_ffn")
    return y_perm


def combine(y_perm, row_of, topk_w, residual=None, out=None, stream=None):
    """foe_combine: returns out [T,d]."""
    T, k = topk_w.shape
    d = y_perm.shape[1]
    dt = _dt(y_perm)
    if out is None:
        out = torch.empty((T, d), dtype=y_perm.dtype, device=y_perm.device)
    rc = lib().foe_combine(dt, T, d, k, _dev(y_perm, "y_perm"), _dev(row_of, "row_of", torch.int32),
                           _dev(topk_w, "topk_w", torch.float32),
                           _dev(residual, "residual", y_perm.dtype), _dev(out, "out", y_perm.dtype),
                           _stream(stream))
    _check(rc, "foe_combine")
    return out


def reduce(partials, scale, residual=None, out=None, stream=None):
    """foe_reduce: out = scale * sum_h (residual + partials[h])."""
    C, T, d = partials.shape
    dt = _dt(partials)
    if out is None:
        out = torch.empty((T, d), dtype=partials.dtype, device=partials.device)
    rc = lib().foe_reduce(dt, C, T, d, _dev(partials, "partials"),
                          _dev(residual, "residual", partials.dtype), float(scale),
                          _dev(out, "out", partials.dtype), _stream(stream))
    _check(rc, "foe_reduce")
    return out


def cluster_block(x, w_router, bias, w_gate, w_up, w_down, k, reduce_scale=None, out=None,
                  ws=None, stream=None, gating="renorm"):
    """foe_cluster_block (foe_cluster_block_ex for a gating other than "renorm")
    for C clusters: weights stacked on a leading C axis."""
    T, d = x.shape
    C, E, F, _ = w_gate.shape
    dt = _dt(x)
    if reduce_scale is None:
        reduce_scale = 1.0 / C
    if out is None:
        out = torch.empty((T, d), dtype=x.dtype, device=x.device)
    need = workspace_bytes("cluster_block", dt, C, T, d, E, k, F)
    ws = _workspace(ws, need, x.device)
    args = (_dev(x, "x"), _dev(w_router, "w_router", x.dtype), _dev(bias, "bias", torch.float32),
            _dev(w_gate, "w_gate", x.dtype), _dev(w_up, "w_up", x.dtype),
            _dev(w_down, "w_down", x.dtype), float(reduce_scale), _dev(out, "out", x.dtype),
            _dev(ws, "ws"), ws.numel(), _stream(stream))
    if gating == "renorm":
        _check(lib().foe_cluster_block(dt, C, T, d, E, k, F, *args), "foe_cluster_block")
    else:
        _check(lib().foe_cluster_block_ex(dt, C, T, d, E, k, F, _gating(gating), *args),
               "foe_cluster_block_ex")
    return out


# bytes of the per-GPU scratch array of foe_cluster_block_noalloc
NOALLOC_SCRATCH_BYTES = 128 << 20


def cluster_block_noalloc(x, w_router, bias, w_gate, w_up, w_down, k, reduce_scale=None,
                          out=None, stream=None):
    """foe_cluster_block_noalloc: foe_cluster_block without a workspace (the
    library's per-GPU scratch array); weights stacked on a leading C axis."""
    T, d = x.shape
    C, E, F, _ = w_gate.shape
    if reduce_scale is None:
        reduce_scale = 1.0 / C
    if out is None:
        out = torch.empty((T, d), dtype=x.dtype, device=x.device)
    _check(lib().foe_cluster_block_noalloc(
        _dt(x), C, T, d, E, k, F, _dev(x, "x"), _dev(w_router, "w_router", x.dtype),
        _dev(bias, "bias", torch.float32), _dev(w_gate, "w_gate", x.dtype),
        _dev(w_up, "w_up", x.dtype), _dev(w_down, "w_down", x.dtype), float(reduce_scale),
        _dev(out, "out", x.dtype), _stream(stream)), "foe_cluster_block_noalloc")
    return out


def group_attention(x, w_qkv, w_o, nq, theta, scale=1.0, out=None, ws=None, stream=None):
    """foe_group_attention: x [H,S,d], w_qkv [H,(nq+2)*hd,d], w_o [d,H*nq*hd]
    (the groups' output projections side by side; bf16, hd = 96 or 128) ->
    r_full [S,d]."""
    H, S, d = x.shape
    hd = w_qkv.shape[1] // (nq + 2)
    if tuple(w_qkv.shape) != (H, (nq + 2) * hd, d) or tuple(w_o.shape) != (d, H * nq * hd):
        raise FoeError(FOE_ERR_INVALID, f"group_attention: w_qkv {tuple(w_qkv.shape)} / w_o "
                       f"{tuple(w_o.shape)} do not match x {tuple(x.shape)} with nq={nq}")
    if out is None:
        out = torch.empty((S, d), dtype=x.dtype, device=x.device)
    n = lib().foe_group_attention_workspace_bytes(H, S, d, nq, hd)
    if n == ctypes.c_size_t(-1).value:
        raise FoeError(FOE_ERR_INVALID, f"foe_group_attention_workspace_bytes: {last_error()}")
    ws = _workspace(ws, n, x.device)
    rc = lib().foe_group_attention(_dt(x), H, S, d, nq, hd, float(theta), float(scale),
                                   _dev(x, "x"), _dev(w_qkv, "w_qkv", x.dtype),
                                   _dev(w_o, "w_o", x.dtype), _dev(out, "r_full", x.dtype),
                                   _dev(ws, "ws"), ws.numel(), _stream(stream))
    _check(rc, "foe_group_attention")
    return out


# ---- kernel timing -------------------------------------------------------------

def profile_enable(on=True):
    _check(lib().foe_profile_enable(1 if on else 0), "foe_profile_enable")


def profile_reset():
    _check(lib().foe_profile_reset(), "foe_profile_reset")


def profile_kernel(name):
    """(launches, total_ms) recorded for kernel ``name``."""
    n = ctypes.c_int(0)
    ms = ctypes.c_double(0.0)
    _check(lib().foe_profile_kernel(name.encode(), ctypes.byref(n), ctypes.byref(ms)),
           "foe_profile_kernel")
    return n.value, ms.value


def profile_names():
    need = lib().foe_profile_names(None, 0)
    buf = ctypes.create_string_buffer(need)
    lib().foe_profile_names(buf, need)
    s = buf.value.decode()
    return [t for t in s.split(",") if t]
