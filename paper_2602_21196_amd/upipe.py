"""ctypes binding of libupipe.so (the C ABI in include/upipe.h).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  PyTorch supplies device memory and the current stream.  The
``upipe_*`` functions mirror the C entry points one to one; ``attn_fwd`` /
``attn_bwd`` / ``layer_fwd`` / ``layer_bwd`` are conveniences that allocate
outputs and the workspace with torch and raise on a non-zero status.

If the library has not been built this module raises when it is first used;
there is no fallback implementation.
"""

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libupipe.so")

UPIPE_OK = 0
STATUS = {0: "UPIPE_OK", -1: "UPIPE_ERR_INVALID_ARG", -2: "UPIPE_ERR_UNSUPPORTED",
          -3: "UPIPE_ERR_WORKSPACE", -4: "UPIPE_ERR_HIP"}

_c_void_p = ctypes.c_void_p
_i64 = ctypes.c_int64
_int = ctypes.c_int
_size = ctypes.c_size_t
_fptr = ctypes.c_void_p
_dbl = ctypes.c_double

_SIGNATURES = {
    "upipe_status_string": (ctypes.c_char_p, [_int]),
    "upipe_version": (_int, []),
    "upipe_gqa_schedule": (_int, [_int, _int, _int, _int,
                                  ctypes.POINTER(_int), ctypes.POINTER(_int)]),
    "upipe_attn_fwd_workspace_size": (_size, [_i64, _int, _int, _int, _int]),
    "upipe_attn_bwd_workspace_size": (_size, [_i64, _int, _int, _int, _int]),
    "upipe_layer_fwd_workspace_size": (_size, [_i64, _int, _int, _int, _int, _int]),
    "upipe_layer_bwd_workspace_size": (_size, [_i64, _int, _int, _int, _int, _int]),
    "upipe_attn_fwd": (_int, [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _fptr,
                              _i64, _int, _int, _int, _int, _int,
                              _c_void_p, _size, _c_void_p]),
    "upipe_attn_fwd_batch": (_int, [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _fptr,
                                    _i64, _i64, _int, _int, _int, _int, _int,
                                    _c_void_p, _size, _c_void_p]),
    "upipe_attn_bwd": (_int, [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _fptr,
                              _c_void_p, _c_void_p, _c_void_p, _c_void_p,
                              _i64, _int, _int, _int, _int, _int,
                              _c_void_p, _size, _c_void_p]),
    "upipe_attn_bwd_batch": (_int, [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _fptr,
                                    _c_void_p, _c_void_p, _c_void_p, _c_void_p,
                                    _i64, _i64, _int, _int, _int, _int, _int,
                                    _c_void_p, _size, _c_void_p]),
    "upipe_attn_fwd_noalloc_scratch_bytes": (_size, []),
    "upipe_attn_fwd_noalloc": (_int, [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _fptr,
                                      _i64, _int, _int, _int, _int, _int, _c_void_p]),
    "upipe_attn_fwd_ring_workspace_size": (_size, [_i64, _i64, _int, _int, _int, _int]),
    "upipe_attn_fwd_ring": (_int, [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _fptr,
                                   _i64, _i64, _i64, _i64, _int, _int, _int, _int,
                                   _int, _c_void_p, _size, _c_void_p]),
    "upipe_lse_merge": (_int, [_c_void_p, _fptr, _c_void_p, _fptr, _i64, _int, _int,
                               _c_void_p]),
    "upipe_rope": (_int, [_c_void_p, _i64, _int, _int, _i64, _dbl, _int, _c_void_p]),
    "upipe_layer_fwd": (_int, [_c_void_p, _c_void_p, _c_void_p, _c_void_p,
                               _c_void_p, _fptr, _i64, _int, _int, _int, _int,
                               _int, _c_void_p, _size, _c_void_p]),
    "upipe_layer_bwd": (_int, [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _fptr,
                               _c_void_p, _c_void_p, _c_void_p, _c_void_p,
                               _i64, _int, _int, _int, _int, _int,
                               _c_void_p, _size, _c_void_p]),
    "upipe_layer_fwd_ex": (_int, [_c_void_p, _c_void_p, _c_void_p, _c_void_p,
                                  _c_void_p, _fptr, _i64, _i64, _int, _int, _int, _int,
                                  _int, _dbl, _i64, _c_void_p, _size, _c_void_p]),
    "upipe_layer_bwd_ex": (_int, [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _fptr,
                                  _c_void_p, _c_void_p, _c_void_p, _c_void_p,
                                  _i64, _i64, _int, _int, _int, _int, _int, _dbl, _i64,
                                  _c_void_p, _size, _c_void_p]),
    "upipe_gemm_bf16": (_int, [_c_void_p, _c_void_p, _c_void_p, _i64, _i64, _i64,
                               _c_void_p]),
    "upipe_profile_enable": (_int, [_int]),
    "upipe_profile_reset": (_int, []),
    "upipe_profile_query": (_int, [ctypes.c_char_p, ctypes.POINTER(_int),
                                   ctypes.POINTER(ctypes.c_double)]),
    "upipe_profile_name": (ctypes.c_char_p, [_int]),
}

_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with "
                "`python -m paper_2602_21196_amd.build` (no fallback exists)")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


class UpipeError(RuntimeError):
    def __init__(self, fn, status):
        super().__init__(f"{fn} returned {STATUS.get(status, status)}")
        self.status = status


def _check(fn, status):
    if status != UPIPE_OK:
        raise UpipeError(fn, status)


# ------------------------------------------------------------ raw mirrors

def upipe_status_string(status):
    return lib().upipe_status_string(status).decode()


def upipe_version():
    return lib().upipe_version()


def upipe_gqa_schedule(H, Hkv, C, U):
    """Returns (status, stage_heads list[H], kv_stage list[Hkv])."""
    heads = (_int * max(H, 1))()
    kvs = (_int * max(Hkv, 1))()
    st = lib().upipe_gqa_schedule(H, Hkv, C, U, heads, kvs)
    return st, list(heads)[:H], list(kvs)[:Hkv]


def upipe_attn_fwd_workspace_size(S, Hq, Hkv, d, U):
    return lib().upipe_attn_fwd_workspace_size(S, Hq, Hkv, d, U)


def upipe_attn_bwd_workspace_size(S, Hq, Hkv, d, U):
    return lib().upipe_attn_bwd_workspace_size(S, Hq, Hkv, d, U)


def upipe_layer_fwd_workspace_size(S, d_model, Hq, Hkv, d, U):
    return lib().upipe_layer_fwd_workspace_size(S, d_model, Hq, Hkv, d, U)


def upipe_layer_bwd_workspace_size(S, d_model, Hq, Hkv, d, U):
    return lib().upipe_layer_bwd_workspace_size(S, d_model, Hq, Hkv, d, U)


def upipe_attn_fwd(q, k, v, o, lse, S, Hq, Hkv, d, causal, U, ws, ws_bytes, stream):
    return lib().upipe_attn_fwd(q, k, v, o, lse, S, Hq, Hkv, d, causal, U, ws,
                                ws_bytes, stream)


def upipe_attn_fwd_batch(q, k, v, o, lse, B, S, Hq, Hkv, d, causal, U, ws, ws_bytes,
                         stream):
    return lib().upipe_attn_fwd_batch(q, k, v, o, lse, B, S, Hq, Hkv, d, causal, U,
                                      ws, ws_bytes, stream)


def upipe_attn_bwd(q, k, v, o, lse, dout, dq, dk, dv, S, Hq, Hkv, d, causal,
                   U, ws, ws_bytes, stream):
    return lib().upipe_attn_bwd(q, k, v, o, lse, dout, dq, dk, dv, S, Hq, Hkv,
                                d, causal, U, ws, ws_bytes, stream)


def upipe_attn_bwd_batch(q, k, v, o, lse, dout, dq, dk, dv, B, S, Hq, Hkv, d,
                         causal, U, ws, ws_bytes, stream):
    return lib().upipe_attn_bwd_batch(q, k, v, o, lse, dout, dq, dk, dv, B, S, Hq,
                                      Hkv, d, causal, U, ws, ws_bytes, stream)


def upipe_attn_fwd_noalloc_scratch_bytes():
    return lib().upipe_attn_fwd_noalloc_scratch_bytes()


def upipe_attn_fwd_noalloc(q, k, v, o, lse, S, Hq, Hkv, d, causal, U, stream):
    return lib().upipe_attn_fwd_noalloc(q, k, v, o, lse, S, Hq, Hkv, d, causal, U, stream)


def upipe_attn_fwd_ring_workspace_size(Sq, Skv, Hq, Hkv, d, U):
    return lib().upipe_attn_fwd_ring_workspace_size(Sq, Skv, Hq, Hkv, d, U)


def upipe_attn_fwd_ring(q, k, v, o, lse, Sq, Skv, q_offset, kv_offset, Hq, Hkv,
                        d, causal, U, ws, ws_bytes, stream):
    return lib().upipe_attn_fwd_ring(q, k, v, o, lse, Sq, Skv, q_offset,
                                     kv_offset, Hq, Hkv, d, causal, U, ws,
                                     ws_bytes, stream)


def upipe_lse_merge(o, lse, o_part, lse_part, S, H, d, stream):
    return lib().upipe_lse_merge(o, lse, o_part, lse_part, S, H, d, stream)


def upipe_rope(x, S, H, d, pos0, base, inverse, stream):
    return lib().upipe_rope(x, S, H, d, pos0, base, inverse, stream)


def upipe_layer_fwd(x, wqkv, wo, y, o_saved, lse_saved, S, d_model, Hq, Hkv, d, U,
                    ws, ws_bytes, stream):
    return lib().upipe_layer_fwd(x, wqkv, wo, y, o_saved, lse_saved, S, d_model,
                                 Hq, Hkv, d, U, ws, ws_bytes, stream)


def upipe_layer_bwd(x, wqkv, wo, o_saved, lse_saved, dy, dx, dwqkv, dwo, S,
                    d_model, Hq, Hkv, d, U, ws, ws_bytes, stream):
    return lib().upipe_layer_bwd(x, wqkv, wo, o_saved, lse_saved, dy, dx,
                                 dwqkv, dwo, S, d_model, Hq, Hkv, d, U, ws,
                                 ws_bytes, stream)


def upipe_layer_fwd_ex(x, wqkv, wo, y, o_saved, lse_saved, B, S, d_model, Hq, Hkv,
                       d, U, rope_base, pos0, ws, ws_bytes, stream):
    return lib().upipe_layer_fwd_ex(x, wqkv, wo, y, o_saved, lse_saved, B, S,
                                    d_model, Hq, Hkv, d, U, rope_base, pos0, ws,
                                    ws_bytes, stream)


def upipe_layer_bwd_ex(x, wqkv, wo, o_saved, lse_saved, dy, dx, dwqkv, dwo, B, S,
                       d_model, Hq, Hkv, d, U, rope_base, pos0, ws, ws_bytes,
                       stream):
    return lib().upipe_layer_bwd_ex(x, wqkv, wo, o_saved, lse_saved, dy, dx,
                                    dwqkv, dwo, B, S, d_model, Hq, Hkv, d, U,
                                    rope_base, pos0, ws, ws_bytes, stream)


def upipe_gemm_bf16(a, b, c, M, N, K, stream):
    return lib().upipe_gemm_bf16(a, b, c, M, N, K, stream)


def upipe_profile_enable(on):
    return lib().upipe_profile_enable(int(on))


def upipe_profile_reset():
    return lib().upipe_profile_reset()


def upipe_profile_query(name):
    n = _int(0)
    ms = ctypes.c_double(0.0)
    st = lib().upipe_profile_query(name.encode(), ctypes.byref(n),
                                   ctypes.byref(ms))
    _check("upipe_profile_query", st)
    return n.value, ms.value


def upipe_profile_names():
    out, i = [], 0
    while True:
        nm = lib().upipe_profile_name(i)
        if nm is None:
            return out
        out.append(nm.decode())
        i += 1


# ------------------------------------------------------ torch conveniences

def _torch():
    import torch
    return torch


def _ptr(t, dtype, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must live on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream():
    return _torch().cuda.current_stream().cuda_stream


def workspace(nbytes, device):
    torch = _torch()
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def _batch(t, rank):
    """(B, shape without the batch) of a tensor with an optional leading batch."""
    if t.dim() == rank:
        return 1, tuple(t.shape)
    if t.dim() == rank + 1:
        return t.shape[0], tuple(t.shape[1:])
    raise ValueError(f"expected {rank} or {rank + 1} dimensions, got {t.dim()}")


def _lse_shape(q, B, Hq, S):
    return (Hq, S) if q.dim() == 3 else (B, Hq, S)


def _shape(t, want, name):
    """Raise ValueError unless tensor t has exactly the shape `want`: the C ABI
    sees raw pointers only, so a wrong size would be read or written out of
    bounds on the GPU."""
    if tuple(t.shape) != tuple(want):
        raise ValueError(f"{name} must have shape {tuple(want)}, got {tuple(t.shape)}")


def _attn_shapes(q, k, v, lead):
    """(B, S, Hq, Hkv, d) of q [(B,)S,Hq,d], k and v [(B,)S,Hkv,d]."""
    if q.dim() not in (3, 4):
        raise ValueError(f"q must be [S,Hq,d] or [B,S,Hq,d], got {tuple(q.shape)}")
    B, (S, Hq, d) = _batch(q, 3)
    if k.dim() != q.dim():
        raise ValueError(f"k must have shape {lead}[S,Hkv,d] like q, got {tuple(k.shape)}")
    Hkv = k.shape[-2]
    _shape(k, tuple(q.shape[:-2]) + (Hkv, d), "k")
    _shape(v, tuple(q.shape[:-2]) + (Hkv, d), "v")
    return B, S, Hq, Hkv, d


def attn_fwd(q, k, v, causal=True, U=1, ws=None):
    """o [(B,)S,Hq,d] bf16, lse [(B,)Hq,S] fp32 for q [(B,)S,Hq,d],
    k/v [(B,)S,Hkv,d] bf16.  Without a batch dimension this is the contract
    call upipe_attn_fwd, with one upipe_attn_fwd_batch."""
    torch = _torch()
    B, S, Hq, Hkv, d = _attn_shapes(q, k, v, "[B,]")
    need = upipe_attn_fwd_workspace_size(S, Hq, Hkv, d, U)
    if need == 0:
        raise UpipeError("upipe_attn_fwd_workspace_size", -1)
    if ws is None:
        ws = workspace(need, q.device)
    o = torch.empty_like(q)
    lse = torch.empty(_lse_shape(q, B, Hq, S), dtype=torch.float32, device=q.device)
    bf = torch.bfloat16
    ptrs = (_ptr(q, bf, "q"), _ptr(k, bf, "k"), _ptr(v, bf, "v"), _ptr(o, bf, "o"),
            _ptr(lse, torch.float32, "lse"))
    if q.dim() == 3:
        st = upipe_attn_fwd(*ptrs, S, Hq, Hkv, d, int(causal), U, ws.data_ptr(),
                            ws.numel(), _stream())
        _check("upipe_attn_fwd", st)
    else:
        st = upipe_attn_fwd_batch(*ptrs, B, S, Hq, Hkv, d, int(causal), U, ws.data_ptr(),
                                  ws.numel(), _stream())
        _check("upipe_attn_fwd_batch", st)
    return o, lse


def attn_fwd_ring(q, k, v, q_offset, kv_offset, causal=True, U=1, ws=None):
    """One ring step: o [Sq,Hq,d] bf16, lse [Hq,Sq] fp32 of q [Sq,Hq,d] (global
    rows q_offset..) against k/v [Skv,Hkv,d] (global rows kv_offset..)."""
    torch = _torch()
    if q.dim() != 3 or k.dim() != 3:
        raise ValueError("attn_fwd_ring: q [Sq,Hq,d], k and v [Skv,Hkv,d]")
    Sq, Hq, d = q.shape
    Skv, Hkv = k.shape[0], k.shape[1]
    _shape(k, (Skv, Hkv, d), "k")
    _shape(v, (Skv, Hkv, d), "v")
    need = upipe_attn_fwd_ring_workspace_size(Sq, Skv, Hq, Hkv, d, U)
    if need == 0:
        raise UpipeError("upipe_attn_fwd_ring_workspace_size", -1)
    if ws is None:
        ws = workspace(need, q.device)
    o = torch.empty_like(q)
    lse = torch.empty((Hq, Sq), dtype=torch.float32, device=q.device)
    bf = torch.bfloat16
    st = upipe_attn_fwd_ring(_ptr(q, bf, "q"), _ptr(k, bf, "k"), _ptr(v, bf, "v"),
                             _ptr(o, bf, "o"), _ptr(lse, torch.float32, "lse"),
                             Sq, Skv, int(q_offset), int(kv_offset), Hq, Hkv, d,
                             int(causal), U, ws.data_ptr(), ws.numel(), _stream())
    _check("upipe_attn_fwd_ring", st)
    return o, lse


def lse_merge(o, lse, o_part, lse_part):
    """In place: fold (o_part [S,H,d], lse_part [H,S]) into (o, lse)."""
    torch = _torch()
    if o.dim() != 3:
        raise ValueError("lse_merge: o, o_part [S,H,d] and lse, lse_part [H,S]")
    S, H, d = o.shape
    if tuple(o_part.shape) != (S, H, d) or tuple(lse.shape) != (H, S) or \
            tuple(lse_part.shape) != (H, S):
        raise ValueError("lse_merge: o, o_part [S,H,d] and lse, lse_part [H,S]")
    bf = torch.bfloat16
    st = upipe_lse_merge(_ptr(o, bf, "o"), _ptr(lse, torch.float32, "lse"),
                         _ptr(o_part, bf, "o_part"),
                         _ptr(lse_part, torch.float32, "lse_part"), S, H, d, _stream())
    _check("upipe_lse_merge", st)
    return o, lse


def attn_bwd(q, k, v, o, lse, dout, causal=True, U=1, ws=None):
    """dq [(B,)S,Hq,d], dk, dv [(B,)S,Hkv,d] bf16.  Without a batch dimension
    this is the contract call upipe_attn_bwd, with one upipe_attn_bwd_batch."""
    torch = _torch()
    B, S, Hq, Hkv, d = _attn_shapes(q, k, v, "[B,]")
    _shape(o, q.shape, "o")
    _shape(dout, q.shape, "dout")
    _shape(lse, _lse_shape(q, B, Hq, S), "lse")
    need = upipe_attn_bwd_workspace_size(S, Hq, Hkv, d, U)
    if need == 0:
        raise UpipeError("upipe_attn_bwd_workspace_size", -1)
    if ws is None:
        ws = workspace(need, q.device)
    dq = torch.empty_like(q)
    dk = torch.empty_like(k)
    dv = torch.empty_like(v)
    bf = torch.bfloat16
    ptrs = (_ptr(q, bf, "q"), _ptr(k, bf, "k"), _ptr(v, bf, "v"), _ptr(o, bf, "o"),
            _ptr(lse, torch.float32, "lse"), _ptr(dout, bf, "dout"), _ptr(dq, bf, "dq"),
            _ptr(dk, bf, "dk"), _ptr(dv, bf, "dv"))
    if q.dim() == 3:
        st = upipe_attn_bwd(*ptrs, S, Hq, Hkv, d, int(causal), U, ws.data_ptr(),
                            ws.numel(), _stream())
        _check("upipe_attn_bwd", st)
    else:
        st = upipe_attn_bwd_batch(*ptrs, B, S, Hq, Hkv, d, int(causal), U, ws.data_ptr(),
                                  ws.numel(), _stream())
        _check("upipe_attn_bwd_batch", st)
    return dq, dk, dv


def rope(x, base, pos0=0, inverse=False):
    """In place on x [S,H,d] bf16: rotary embedding at positions pos0 + s."""
    torch = _torch()
    if x.dim() != 3:
        raise ValueError(f"rope: x must be [S,H,d], got {tuple(x.shape)}")
    S, H, d = x.shape
    st = upipe_rope(_ptr(x, torch.bfloat16, "x"), S, H, d, int(pos0), float(base),
                    int(bool(inverse)), _stream())
    _check("upipe_rope", st)
    return x


def _layer_shapes(x, wqkv, wo, Hq, Hkv, d):
    """(B, S, d_model) of x [(B,)S,dm], with wqkv and wo checked against the
    head counts."""
    if x.dim() not in (2, 3):
        raise ValueError(f"x must be [S,d_model] or [B,S,d_model], got {tuple(x.shape)}")
    B, (S, dm) = _batch(x, 2)
    _shape(wqkv, (dm, (Hq + 2 * Hkv) * d), "wqkv")
    _shape(wo, (Hq * d, dm), "wo")
    return B, S, dm


def _plain_layer(x, rope_base, pos0):
    """The contract calls cover one sequence without rotary embedding."""
    return x.dim() == 2 and float(rope_base) == 0.0 and int(pos0) == 0


def layer_fwd(x, wqkv, wo, Hq, Hkv, d=128, U=1, ws=None, rope_base=0.0, pos0=0):
    """y [(B,)S,dm] bf16, o_saved [(B,)S,Hq,d] bf16, lse_saved [(B,)Hq,S]
    fp32.  rope_base > 0 rotates Q and K at positions pos0 + s.  One sequence
    without rotation goes through the contract call upipe_layer_fwd, anything
    else through upipe_layer_fwd_ex."""
    torch = _torch()
    B, S, dm = _layer_shapes(x, wqkv, wo, Hq, Hkv, d)
    need = upipe_layer_fwd_workspace_size(S, dm, Hq, Hkv, d, U)
    if need == 0:
        raise UpipeError("upipe_layer_fwd_workspace_size", -1)
    if ws is None:
        ws = workspace(need, x.device)
    y = torch.empty_like(x)
    lead = (B,) if x.dim() == 3 else ()
    o = torch.empty(lead + (S, Hq, d), dtype=torch.bfloat16, device=x.device)
    lse = torch.empty(lead + (Hq, S), dtype=torch.float32, device=x.device)
    bf = torch.bfloat16
    ptrs = (_ptr(x, bf, "x"), _ptr(wqkv, bf, "wqkv"), _ptr(wo, bf, "wo"), _ptr(y, bf, "y"),
            _ptr(o, bf, "o_saved"), _ptr(lse, torch.float32, "lse_saved"))
    if _plain_layer(x, rope_base, pos0):
        st = upipe_layer_fwd(*ptrs, S, dm, Hq, Hkv, d, U, ws.data_ptr(), ws.numel(),
                             _stream())
        _check("upipe_layer_fwd", st)
    else:
        st = upipe_layer_fwd_ex(*ptrs, B, S, dm, Hq, Hkv, d, U, float(rope_base), int(pos0),
                                ws.data_ptr(), ws.numel(), _stream())
        _check("upipe_layer_fwd_ex", st)
    return y, o, lse


def layer_bwd(x, wqkv, wo, o_saved, lse_saved, dy, Hq, Hkv, d=128, U=1,
              ws=None, rope_base=0.0, pos0=0):
    """dx [(B,)S,dm], dwqkv [dm,(Hq+2Hkv)d], dwo [Hq d, dm] (summed over the
    batch), all bf16.  o_saved = lse_saved = None recomputes the attention
    output (full checkpointing) instead of reading the kept one.  One
    sequence without rotation goes through the contract call upipe_layer_bwd,
    anything else through upipe_layer_bwd_ex."""
    torch = _torch()
    B, S, dm = _layer_shapes(x, wqkv, wo, Hq, Hkv, d)
    _shape(dy, x.shape, "dy")
    kept = o_saved is not None
    if kept != (lse_saved is not None):
        raise ValueError("layer_bwd: pass both o_saved and lse_saved, or neither")
    lead = (B,) if x.dim() == 3 else ()
    if kept:
        _shape(o_saved, lead + (S, Hq, d), "o_saved")
        _shape(lse_saved, lead + (Hq, S), "lse_saved")
    need = upipe_layer_bwd_workspace_size(S, dm, Hq, Hkv, d, U)
    if need == 0:
        raise UpipeError("upipe_layer_bwd_workspace_size", -1)
    if ws is None:
        ws = workspace(need, x.device)
    dx = torch.empty_like(x)
    dwqkv = torch.empty_like(wqkv)
    dwo = torch.empty_like(wo)
    bf = torch.bfloat16
    ptrs = (_ptr(x, bf, "x"), _ptr(wqkv, bf, "wqkv"), _ptr(wo, bf, "wo"),
            _ptr(o_saved, bf, "o_saved") if kept else None,
            _ptr(lse_saved, torch.float32, "lse_saved") if kept else None,
            _ptr(dy, bf, "dy"), _ptr(dx, bf, "dx"), _ptr(dwqkv, bf, "dwqkv"),
            _ptr(dwo, bf, "dwo"))
    if _plain_layer(x, rope_base, pos0):
        st = upipe_layer_bwd(*ptrs, S, dm, Hq, Hkv, d, U, ws.data_ptr(), ws.numel(),
                             _stream())
        _check("upipe_layer_bwd", st)
    else:
        st = upipe_layer_bwd_ex(*ptrs, B, S, dm, Hq, Hkv, d, U, float(rope_base), int(pos0),
                                ws.data_ptr(), ws.numel(), _stream())
        _check("upipe_layer_bwd_ex", st)
    return dx, dwqkv, dwo


def gemm(a, b):
    """c [M,N] = a [M,K] . b [K,N], bf16 with fp32 accumulation (M, N, K
    multiples of 128)."""
    torch = _torch()
    if a.dim() != 2 or b.dim() != 2 or a.shape[1] != b.shape[0]:
        raise ValueError(f"gemm: a [M,K] and b [K,N], got {tuple(a.shape)}, {tuple(b.shape)}")
    M, K = a.shape
    N = b.shape[1]
    c = torch.empty((M, N), dtype=torch.bfloat16, device=a.device)
    bf = torch.bfloat16
    st = upipe_gemm_bf16(_ptr(a, bf, "a"), _ptr(b, bf, "b"), _ptr(c, bf, "c"), M, N, K,
                         _stream())
    _check("upipe_gemm_bf16", st)
    return c
