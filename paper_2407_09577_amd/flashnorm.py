"""Thin Python binding of ``libflashnorm.so`` (the C ABI in ``include/flashnorm.h``).

Argument marshalling only: tensors become device pointers, leading dimensions
and dtype codes; outputs the caller does not pass are allocated with torch; the
work is enqueued on the current torch stream (or the given one).  Every step of
the computation runs in the library's HIP kernels.  If the library is not built
this module raises on first use -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libflashnorm.so")

FN_F32, FN_BF16 = 0, 1
FN_LAYOUT_LINEAR, FN_LAYOUT_GLU = 0, 1
FN_PATH_AUTO, FN_PATH_PREFILL, FN_PATH_DECODE = 0, 1, 2
FN_DECODE_MAX_M = 16
FN_GLU_SWIGLU, FN_GLU_REGLU, FN_GLU_BILINEAR, FN_GLU_SWIGLU_DEFER_UP = 0, 1, 2, 3

STATUS = {0: "FN_OK", -1: "FN_ERR_NULL", -2: "FN_ERR_SHAPE", -3: "FN_ERR_DTYPE", -4: "FN_ERR_ALIGN",
          -5: "FN_ERR_UNSUPPORTED", -6: "FN_ERR_VALUE", -7: "FN_ERR_HIP", -8: "FN_ERR_ALIAS",
          -9: "FN_ERR_SIZE"}

_lib = None


class FlashNormError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {_load().flashnorm_status_string(status).decode()}")


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built: run `python -c 'import __graft_entry__ as g; g.build()'`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I64, I, F = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float
    sig = {
        "fold_weights_size": ([I64, I64, I, I], ctypes.c_size_t),
        "fold_weights": ([P, I64, I64, I, P, P, I64, I64, I, P, I, P, P, P], I),
        "unpack_weights": ([P, I64, I64, I, I, P, I64, P], I),
        "flashnorm_linear": ([P, I64, I64, I64, I, P, I64, F, P, P, I64, I, P, P], I),
        "flashnorm_linear_ex": ([P, I64, I64, I64, I, P, I64, F, P, P, I64, I, P, I, P], I),
        "flashnorm_glu": ([P, I64, I64, I64, I, P, I64, F, P, I64, I, P], I),
        "flashnorm_glu_ex": ([P, I64, I64, I64, I, P, I64, F, P, I64, I, I, P], I),
        "flashnorm_layernorm_linear": ([P, I64, I64, I64, I, P, P, P, I64, F, P, I64, I, P], I),
        "flashnorm_layernorm_linear_ex": ([P, I64, I64, I64, I, P, P, P, I64, F, P, I64, I, I, P], I),
        "baseline_rmsnorm_linear": ([P, I64, I64, I64, I, P, P, I64, F, P, P, I64, I, P], I),
        "baseline_rmsnorm_glu": ([P, I64, I64, I64, I, P, P, I64, F, P, P, I64, I, P], I),
        "baseline_layernorm_linear": ([P, I64, I64, I64, I, P, P, P, I64, F, P, P, I64, I, P], I),
        "baseline_rmsnorm_linear_noalloc": ([P, I64, I64, I64, I, P, P, I64, F, P, I64, I, P], I),
        "flashnorm_glu_act": ([P, I64, I64, I64, I, P, I64, F, I, P, I64, I, P, I, P], I),
        "flashnorm_linear_relu": ([P, I64, I64, I64, I, P, I64, F, P, I64, I, P, I, P], I),
        "rowscale_linear": ([P, I64, I64, I64, I, P, I64, P, P, I64, I, I, P], I),
        "flashnorm_qkv_rope": ([P, I64, I64, I64, I, P, I64, I64, I64, F, P, P, P, P, I64, F, P, I64, I, P, I, P],
                               I),
        "baseline_rope": ([P, I64, I64, I, I64, I64, I64, P, P, P, I64, F, P], I),
        "baseline_qkv_headnorm": ([P, I64, I64, I, I64, I64, I64, P, P, P, F, P, P, P, I64, F, P], I),
        "flashnorm_qkv_headnorm": ([P, I64, I64, I64, I, P, I64, I64, I64, F, P, P, P, F, P, P, P, I64, F, P, I64,
                                    I, P, I, P], I),
        "flashnorm_mla_latent": ([P, I64, I64, I64, I, P, I64, I64, P, F, F, P, P, P, I64, P, I64, I, P, I, P], I),
        "baseline_mla_latent": ([P, I64, I64, I, I64, I64, P, F, P, P, P, I64, P], I),
        "flashnorm_linear_unfolded": ([P, I64, I64, I64, I, P, P, I64, F, P, P, I64, I, P, I, P], I),
        "flashnorm_glu_unfolded": ([P, I64, I64, I64, I, P, P, I64, F, P, I64, I, I, P], I),
        "flashnorm_status_string": ([I], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def lib():
    """The raw ctypes handle (for tests of the C ABI itself)."""
    return _load()


def _check(status: int, where: str):
    if status != 0:
        raise FlashNormError(status, where)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return FN_BF16
    if t.dtype == torch.float32:
        return FN_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _torch_dtype(code: int) -> torch.dtype:
    return torch.bfloat16 if code == FN_BF16 else torch.float32


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _ld(t: torch.Tensor) -> int:
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("expected a row-major 2-D tensor (unit column stride)")
    return t.stride(0)


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _vec(t, n, name):
    if t is None:
        return None
    if t.dtype != torch.float32 or t.numel() != n or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous fp32 vector of {n} elements")
    return t


def _new_out(M: int, N: int, like: torch.Tensor) -> torch.Tensor:
    """A new [M, N] output in like's dtype and device.  Its rows are padded to a multiple of
    16 bytes, the row pitch the kernels' vector stores require (FN_ERR_ALIGN otherwise), so
    any N works; the result is then a view of the first N columns."""
    per = 16 // like.element_size()
    ld = (N + per - 1) // per * per
    buf = torch.empty(M, ld, dtype=like.dtype, device=like.device)
    return buf if ld == N else buf[:, :N]


def fold_weights_size(K: int, N: int, layout: int = FN_LAYOUT_LINEAR, ws_dtype: int = FN_BF16) -> int:
    return _load().fold_weights_size(K, N, layout, ws_dtype)


# The C ABI takes raw device pointers and sizes the kernels' reads from the shape
# arguments, so the binding refuses, before any call, tensors that the library would
# read or write out of bounds: host tensors, tensors on different GPUs, outputs whose
# shape is not [M, N], and packed weights or workspaces smaller than the shapes need.
def _guard(where, tensors=(), packed=None, outs=(), nbytes=()):
    """packed = (W_star, K, N, layout, dtype code); outs = ((tensor, rows, cols), ...);
    nbytes = ((tensor, bytes needed, name), ...).  Size checks come first, then devices."""
    if packed is not None:
        Wst, K, N, layout, code = packed
        need = fold_weights_size(K, N, layout, code)
        # need == 0: invalid geometry, which the library itself rejects with its status
        if need and Wst.numel() * Wst.element_size() < need:
            raise ValueError(f"{where}: the packed weight holds {Wst.numel() * Wst.element_size()} bytes; "
                             f"K = {K}, N = {N} need {need} (fold_weights_size)")
        if not Wst.is_contiguous():
            raise ValueError(f"{where}: the packed weight must be contiguous")
    for t, rows, cols in outs:
        if t is not None and tuple(t.shape) != (rows, cols):
            raise ValueError(f"{where}: output of shape {tuple(t.shape)}, expected ({rows}, {cols})")
    for t, need, name in nbytes:
        if t is not None and t.numel() * t.element_size() < need:
            raise ValueError(f"{where}: {name} holds {t.numel() * t.element_size()} bytes; {need} needed")
    dev = None
    for t in tensors:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError(f"{where}: every tensor must be a GPU tensor (got one on {t.device})")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError(f"{where}: tensors on {dev} and {t.device}; all must be on one GPU")


def fold_weights(W: torch.Tensor, g, beta=None, layout: int = FN_LAYOUT_LINEAR, ws_dtype=None,
                 colsum: bool = False, c_star: bool = False, stream=None):
    """Fold g into W (and beta into c*) and pack.  W is the logical [K, N] weight
    ([K, 2F] = [Wg | Wu] for a GLU), any strides: a torch linear layer's [N, K]
    weight is passed as ``weight.t()`` and read in place.  g = None packs W
    unchanged.  Returns (W_star, colsum or None, c_star or None); W_star is an
    opaque uint8 device buffer."""
    K, N = W.shape
    ws_code = _dt(W) if ws_dtype is None else (ws_dtype if isinstance(ws_dtype, int) else _dt(torch.empty(0, dtype=ws_dtype)))
    nbytes = fold_weights_size(K, N, layout, ws_code)
    if nbytes == 0:
        raise ValueError("invalid fold geometry")
    _guard("fold_weights", (W, g, beta))
    Ws = torch.empty(nbytes, dtype=torch.uint8, device=W.device)
    cs = torch.empty(N, dtype=torch.float32, device=W.device) if colsum else None
    cb = torch.empty(N, dtype=torch.float32, device=W.device) if c_star else None
    if W.dim() != 2:
        raise ValueError("W must be a 2-D [K, N] tensor")
    _check(_load().fold_weights(_ptr(W), W.stride(0), W.stride(1), _dt(W), _ptr(_vec(g, K, "g")), _ptr(_vec(beta, K, "beta")),
                                K, N, layout, _ptr(Ws), ws_code, _ptr(cs), _ptr(cb), _stream(stream)),
           "fold_weights")
    return Ws, cs, cb


def unpack_weights(W_star: torch.Tensor, K: int, N: int, layout: int = FN_LAYOUT_LINEAR,
                   ws_dtype: int = FN_BF16, stream=None) -> torch.Tensor:
    _guard("unpack_weights", (W_star,), packed=(W_star, K, N, layout, ws_dtype))
    out = torch.zeros(K, N, dtype=_torch_dtype(ws_dtype), device=W_star.device)
    _check(_load().unpack_weights(_ptr(W_star), K, N, layout, ws_dtype, _ptr(out), N, _stream(stream)),
           "unpack_weights")
    return out


def flashnorm_linear(a: torch.Tensor, W_star: torch.Tensor, N: int, eps: float, bias=None, out=None,
                     inv_rms=None, path: int = FN_PATH_AUTO, stream=None) -> torch.Tensor:
    M, K = a.shape
    _guard("flashnorm_linear", (a, W_star, bias, out, inv_rms), packed=(W_star, K, N, FN_LAYOUT_LINEAR, _dt(a)),
           outs=((out, M, N),))
    y = out if out is not None else _new_out(M, N, a)
    _check(_load().flashnorm_linear_ex(_ptr(a), M, K, _ld(a), _dt(a), _ptr(W_star), N, eps,
                                       _ptr(_vec(bias, N, "bias")), _ptr(y), _ld(y), _dt(y),
                                       _ptr(_vec(inv_rms, M, "inv_rms")), path, _stream(stream)),
           "flashnorm_linear")
    return y


def flashnorm_glu(a: torch.Tensor, W_star_gu: torch.Tensor, F: int, eps: float, out=None,
                  path: int = FN_PATH_AUTO, stream=None) -> torch.Tensor:
    M, K = a.shape
    _guard("flashnorm_glu", (a, W_star_gu, out), packed=(W_star_gu, K, 2 * F, FN_LAYOUT_GLU, _dt(a)),
           outs=((out, M, F),))
    o = out if out is not None else _new_out(M, F, a)
    _check(_load().flashnorm_glu_ex(_ptr(a), M, K, _ld(a), _dt(a), _ptr(W_star_gu), F, eps, _ptr(o), _ld(o),
                                    _dt(o), path, _stream(stream)), "flashnorm_glu")
    return o


def flashnorm_glu_act(a: torch.Tensor, W_star_gu: torch.Tensor, F: int, eps: float, act: int, out=None,
                      inv_rms=None, path: int = FN_PATH_AUTO, stream=None) -> torch.Tensor:
    """GLU-variant FFN input projection (act = FN_GLU_*); inv_rms receives s = 1/RMSe(a) where allowed."""
    M, K = a.shape
    _guard("flashnorm_glu_act", (a, W_star_gu, out, inv_rms), packed=(W_star_gu, K, 2 * F, FN_LAYOUT_GLU, _dt(a)),
           outs=((out, M, F),))
    o = out if out is not None else _new_out(M, F, a)
    _check(_load().flashnorm_glu_act(_ptr(a), M, K, _ld(a), _dt(a), _ptr(W_star_gu), F, eps, act, _ptr(o),
                                     _ld(o), _dt(o), _ptr(_vec(inv_rms, M, "inv_rms")), path, _stream(stream)),
           "flashnorm_glu_act")
    return o


def flashnorm_linear_relu(a: torch.Tensor, W_star: torch.Tensor, N: int, eps: float, inv_rms: torch.Tensor,
                          out=None, path: int = FN_PATH_AUTO, stream=None) -> torch.Tensor:
    """ReLU FFN up projection with the scale deferred: y = relu(a W*), inv_rms = 1/RMSe(a)."""
    M, K = a.shape
    _guard("flashnorm_linear_relu", (a, W_star, out, inv_rms), packed=(W_star, K, N, FN_LAYOUT_LINEAR, _dt(a)),
           outs=((out, M, N),))
    y = out if out is not None else _new_out(M, N, a)
    _check(_load().flashnorm_linear_relu(_ptr(a), M, K, _ld(a), _dt(a), _ptr(W_star), N, eps, _ptr(y), _ld(y),
                                         _dt(y), _ptr(_vec(inv_rms, M, "inv_rms")), path, _stream(stream)),
           "flashnorm_linear_relu")
    return y


def rowscale_linear(x: torch.Tensor, W_packed: torch.Tensor, N: int, row_scale: torch.Tensor, out=None,
                    path: int = FN_PATH_AUTO, stream=None) -> torch.Tensor:
    """y = (x W) * row_scale[m]: applies a normalisation scale deferred to this layer's output."""
    M, K = x.shape
    _guard("rowscale_linear", (x, W_packed, row_scale, out), packed=(W_packed, K, N, FN_LAYOUT_LINEAR, _dt(x)),
           outs=((out, M, N),))
    y = out if out is not None else _new_out(M, N, x)
    _check(_load().rowscale_linear(_ptr(x), M, K, _ld(x), _dt(x), _ptr(W_packed), N,
                                   _ptr(_vec(row_scale, M, "row_scale")), _ptr(y), _ld(y), _dt(y), path,
                                   _stream(stream)), "rowscale_linear")
    return y


def flashnorm_qkv_rope(a: torch.Tensor, W_packed: torch.Tensor, Hq: int, Hkv: int, h: int, eps: float,
                       positions: torch.Tensor, cos_tab: torch.Tensor, sin_tab: torch.Tensor, q_scale: float,
                       bias=None, out=None, inv_rms=None, path: int = FN_PATH_AUTO, stream=None) -> torch.Tensor:
    """Deferred RMSNorm -> fused [Wq|Wk|Wv] projection -> RoPE on Q and K (Fig. 5(b))."""
    M, K = a.shape
    N = (Hq + 2 * Hkv) * h
    _guard("flashnorm_qkv_rope", (a, W_packed, positions, cos_tab, sin_tab, bias, out, inv_rms),
           packed=(W_packed, K, N, FN_LAYOUT_LINEAR, _dt(a)), outs=((out, M, N),))
    y = out if out is not None else _new_out(M, N, a)
    if positions.dtype != torch.int32 or not positions.is_contiguous() or positions.numel() != M:
        raise ValueError("positions must be a contiguous int32 tensor of M entries")
    for name, t in (("cos_tab", cos_tab), ("sin_tab", sin_tab)):
        if t.dtype != torch.float32 or not t.is_contiguous() or t.dim() != 2 or t.shape[1] != h // 2:
            raise ValueError(f"{name} must be a contiguous fp32 [P, h/2] tensor")
    if cos_tab.shape != sin_tab.shape:
        raise ValueError("cos_tab and sin_tab differ in shape")
    _check(_load().flashnorm_qkv_rope(_ptr(a), M, K, _ld(a), _dt(a), _ptr(W_packed), Hq, Hkv, h, eps,
                                      _ptr(_vec(bias, N, "bias")), _ptr(positions), _ptr(cos_tab), _ptr(sin_tab),
                                      cos_tab.shape[0], q_scale, _ptr(y), _ld(y), _dt(y),
                                      _ptr(_vec(inv_rms, M, "inv_rms")), path, _stream(stream)),
           "flashnorm_qkv_rope")
    return y


def flashnorm_qkv_headnorm(a: torch.Tensor, W_packed: torch.Tensor, Hq: int, Hkv: int, h: int, eps: float,
                           gq: torch.Tensor, gk: torch.Tensor, gv, eps_head: float, positions=None, cos_tab=None,
                           sin_tab=None, q_scale: float = 1.0, out=None, inv_rms=None, path: int = FN_PATH_AUTO,
                           stream=None) -> torch.Tensor:
    """Deferred RMSNorm -> fused [Wq|Wk|Wv] -> per-head RMSNorm of Q, K (and V with gv) -> RoPE (Prop. 3)."""
    M, K = a.shape
    N = (Hq + 2 * Hkv) * h
    _guard("flashnorm_qkv_headnorm", (a, W_packed, gq, gk, gv, positions, cos_tab, sin_tab, out, inv_rms),
           packed=(W_packed, K, N, FN_LAYOUT_LINEAR, _dt(a)), outs=((out, M, N),))
    y = out if out is not None else _new_out(M, N, a)
    P_rows = 0
    if positions is not None:
        P_rows = _rope_tables(M, h // 2, positions, cos_tab, sin_tab)
    _check(_load().flashnorm_qkv_headnorm(_ptr(a), M, K, _ld(a), _dt(a), _ptr(W_packed), Hq, Hkv, h, eps,
                                          _ptr(_vec(gq, h, "gq")), _ptr(_vec(gk, h, "gk")), _ptr(_vec(gv, h, "gv")),
                                          eps_head, _ptr(positions), _ptr(cos_tab), _ptr(sin_tab), P_rows, q_scale,
                                          _ptr(y), _ld(y), _dt(y), _ptr(_vec(inv_rms, M, "inv_rms")), path,
                                          _stream(stream)), "flashnorm_qkv_headnorm")
    return y


def baseline_qkv_headnorm(y: torch.Tensor, Hq: int, Hkv: int, h: int, gq, gk, gv, eps_head: float, positions=None,
                          cos_tab=None, sin_tab=None, q_scale: float = 1.0, stream=None) -> torch.Tensor:
    """Unfused per-head norms (+ RoPE) on the Q and K (and V) heads of y, in place."""
    M = y.shape[0]
    _guard("baseline_qkv_headnorm", (y, gq, gk, gv, positions, cos_tab, sin_tab),
           outs=((y, M, (Hq + 2 * Hkv) * h),))
    P_rows = _rope_tables(M, h // 2, positions, cos_tab, sin_tab) if positions is not None else 0
    _check(_load().baseline_qkv_headnorm(_ptr(y), M, _ld(y), _dt(y), Hq, Hkv, h, _ptr(_vec(gq, h, "gq")),
                                         _ptr(_vec(gk, h, "gk")), _ptr(_vec(gv, h, "gv")), eps_head, _ptr(positions),
                                         _ptr(cos_tab), _ptr(sin_tab), P_rows, q_scale, _stream(stream)),
           "baseline_qkv_headnorm")
    return y


def baseline_rope(y: torch.Tensor, Hq: int, Hkv: int, h: int, positions: torch.Tensor, cos_tab: torch.Tensor,
                  sin_tab: torch.Tensor, q_scale: float, stream=None) -> torch.Tensor:
    """Unfused RoPE on the Q and K heads of y, in place (the rotation kernel of Fig. 5(a))."""
    M = y.shape[0]
    _rope_tables(M, h // 2, positions, cos_tab, sin_tab)
    _guard("baseline_rope", (y, positions, cos_tab, sin_tab), outs=((y, M, (Hq + 2 * Hkv) * h),))
    _check(_load().baseline_rope(_ptr(y), M, _ld(y), _dt(y), Hq, Hkv, h, _ptr(positions), _ptr(cos_tab),
                                 _ptr(sin_tab), cos_tab.shape[0], q_scale, _stream(stream)), "baseline_rope")
    return y


def _rope_tables(M, half, positions, cos_tab, sin_tab):
    """positions: contiguous int32 [M]; cos_tab, sin_tab: contiguous fp32 [P, half] of one shape."""
    if positions is None or positions.dtype != torch.int32 or not positions.is_contiguous() or positions.numel() != M:
        raise ValueError("positions must be a contiguous int32 tensor of M entries")
    for name, t in (("cos_tab", cos_tab), ("sin_tab", sin_tab)):
        if t is None or t.dtype != torch.float32 or not t.is_contiguous() or t.dim() != 2 or t.shape[1] != half:
            raise ValueError(f"{name} must be a contiguous fp32 [P, {half}] tensor")
    if cos_tab.shape != sin_tab.shape:
        raise ValueError("cos_tab and sin_tab differ in shape")
    return cos_tab.shape[0]


def _rotary_args(M, R, positions, cos_tab, sin_tab):
    if R == 0:
        return None, None, None, 0
    if positions is None or positions.dtype != torch.int32 or not positions.is_contiguous() or positions.numel() != M:
        raise ValueError("positions must be a contiguous int32 tensor of M entries")
    for name, t in (("cos_tab", cos_tab), ("sin_tab", sin_tab)):
        if t is None or t.dtype != torch.float32 or not t.is_contiguous() or t.dim() != 2 or t.shape[1] != R // 2:
            raise ValueError(f"{name} must be a contiguous fp32 [P, R/2] tensor")
    if cos_tab.shape != sin_tab.shape:
        raise ValueError("cos_tab and sin_tab differ in shape")
    return positions, cos_tab, sin_tab, cos_tab.shape[0]


def flashnorm_mla_latent(a: torch.Tensor, W_packed: torch.Tensor, L: int, R: int, g_lat: torch.Tensor,
                         eps_lat: float, eps: float, positions=None, cos_tab=None, sin_tab=None, out=None,
                         inv_rms=None, path: int = FN_PATH_AUTO, stream=None) -> torch.Tensor:
    """MLA down-projection [latent | rotary key] with the latent RMSNorm (Prop. 3: the input
    norm cancels in the latent) and RoPE on the R rotary columns."""
    M, K = a.shape
    _guard("flashnorm_mla_latent", (a, W_packed, g_lat, positions, cos_tab, sin_tab, out, inv_rms),
           packed=(W_packed, K, L + R, FN_LAYOUT_LINEAR, _dt(a)), outs=((out, M, L + R),))
    y = out if out is not None else _new_out(M, L + R, a)
    pos, cos_t, sin_t, P_rows = _rotary_args(M, R, positions, cos_tab, sin_tab)
    if R > 0 and inv_rms is None:
        inv_rms = torch.empty(M, dtype=torch.float32, device=a.device)
    _check(_load().flashnorm_mla_latent(_ptr(a), M, K, _ld(a), _dt(a), _ptr(W_packed), L, R,
                                        _ptr(_vec(g_lat, L, "g_lat")), eps_lat, eps, _ptr(pos), _ptr(cos_t),
                                        _ptr(sin_t), P_rows, _ptr(y), _ld(y), _dt(y),
                                        _ptr(_vec(inv_rms, M, "inv_rms")), path, _stream(stream)),
           "flashnorm_mla_latent")
    return y


def baseline_mla_latent(y: torch.Tensor, L: int, R: int, g_lat: torch.Tensor, eps_lat: float, positions=None,
                        cos_tab=None, sin_tab=None, stream=None) -> torch.Tensor:
    """Unfused latent RMSNorm + rotary key RoPE on y = [latent | key], in place."""
    M = y.shape[0]
    _guard("baseline_mla_latent", (y, g_lat, positions, cos_tab, sin_tab), outs=((y, M, L + R),))
    pos, cos_t, sin_t, P_rows = _rotary_args(M, R, positions, cos_tab, sin_tab)
    _check(_load().baseline_mla_latent(_ptr(y), M, _ld(y), _dt(y), L, R, _ptr(_vec(g_lat, L, "g_lat")), eps_lat,
                                       _ptr(pos), _ptr(cos_t), _ptr(sin_t), P_rows, _stream(stream)),
           "baseline_mla_latent")
    return y


def flashnorm_linear_unfolded(a: torch.Tensor, g: torch.Tensor, W_packed: torch.Tensor, N: int, eps: float,
                              bias=None, out=None, inv_rms=None, path: int = FN_PATH_AUTO, stream=None) -> torch.Tensor:
    """Deferred RMSNorm -> linear with g applied at run time to an unfolded packed W."""
    M, K = a.shape
    _guard("flashnorm_linear_unfolded", (a, g, W_packed, bias, out, inv_rms),
           packed=(W_packed, K, N, FN_LAYOUT_LINEAR, _dt(a)), outs=((out, M, N),))
    y = out if out is not None else _new_out(M, N, a)
    _check(_load().flashnorm_linear_unfolded(_ptr(a), M, K, _ld(a), _dt(a), _ptr(_vec(g, K, "g")), _ptr(W_packed),
                                             N, eps, _ptr(_vec(bias, N, "bias")), _ptr(y), _ld(y), _dt(y),
                                             _ptr(_vec(inv_rms, M, "inv_rms")), path, _stream(stream)),
           "flashnorm_linear_unfolded")
    return y


def flashnorm_glu_unfolded(a: torch.Tensor, g: torch.Tensor, W_packed_gu: torch.Tensor, F: int, eps: float,
                           out=None, path: int = FN_PATH_AUTO, stream=None) -> torch.Tensor:
    """Deferred RMSNorm -> SwiGLU with g applied at run time to an unfolded packed [Wg | Wu]."""
    M, K = a.shape
    _guard("flashnorm_glu_unfolded", (a, g, W_packed_gu, out), packed=(W_packed_gu, K, 2 * F, FN_LAYOUT_GLU, _dt(a)),
           outs=((out, M, F),))
    o = out if out is not None else _new_out(M, F, a)
    _check(_load().flashnorm_glu_unfolded(_ptr(a), M, K, _ld(a), _dt(a), _ptr(_vec(g, K, "g")), _ptr(W_packed_gu),
                                          F, eps, _ptr(o), _ld(o), _dt(o), path, _stream(stream)),
           "flashnorm_glu_unfolded")
    return o


def flashnorm_layernorm_linear(a: torch.Tensor, W_star: torch.Tensor, colsum: torch.Tensor, c_star, N: int,
                               eps: float, out=None, path: int = FN_PATH_AUTO, stream=None) -> torch.Tensor:
    M, K = a.shape
    _guard("flashnorm_layernorm_linear", (a, W_star, colsum, c_star, out),
           packed=(W_star, K, N, FN_LAYOUT_LINEAR, _dt(a)), outs=((out, M, N),))
    y = out if out is not None else _new_out(M, N, a)
    _check(_load().flashnorm_layernorm_linear_ex(_ptr(a), M, K, _ld(a), _dt(a), _ptr(W_star),
                                                 _ptr(_vec(colsum, N, "colsum")), _ptr(_vec(c_star, N, "c_star")),
                                                 N, eps, _ptr(y), _ld(y), _dt(y), path, _stream(stream)),
           "flashnorm_layernorm_linear")
    return y


def _ws(a, x_ws):
    return x_ws if x_ws is not None else torch.empty_like(a, memory_format=torch.contiguous_format)


def _baseline_guard(where, a, g, beta, W_packed, N, layout, x_ws, out, ncols):
    M, K = a.shape
    _guard(where, (a, g, beta, W_packed, x_ws, out), packed=(W_packed, K, N, layout, _dt(a)),
           outs=((out, M, ncols),), nbytes=((x_ws, M * K * a.element_size(), "the workspace x_ws"),))
    if x_ws is not None and (x_ws.dtype != a.dtype or not x_ws.is_contiguous()):
        raise ValueError(f"{where}: the workspace must be contiguous, in the activations' dtype")


def baseline_rmsnorm_linear(a, g, W_packed, N, eps, x_ws=None, out=None, path=FN_PATH_AUTO, stream=None):
    M, K = a.shape
    _baseline_guard("baseline_rmsnorm_linear", a, g, None, W_packed, N, FN_LAYOUT_LINEAR, x_ws, out, N)
    x = _ws(a, x_ws)
    y = out if out is not None else _new_out(M, N, a)
    _check(_load().baseline_rmsnorm_linear(_ptr(a), M, K, _ld(a), _dt(a), _ptr(_vec(g, K, "g")), _ptr(W_packed),
                                           N, eps, _ptr(x), _ptr(y), _ld(y), path, _stream(stream)),
           "baseline_rmsnorm_linear")
    return y


FN_NOALLOC_SCRATCH_BYTES = 32 * 1024 * 1024


def baseline_rmsnorm_linear_noalloc(a, g, W_packed, N, eps, out=None, path=FN_PATH_AUTO, stream=None):
    """baseline_rmsnorm_linear with the library's static device workspace (no x_ws):
    the C call allocates nothing; pass ``out`` to allocate nothing here either."""
    M, K = a.shape
    _guard("baseline_rmsnorm_linear_noalloc", (a, g, W_packed, out),
           packed=(W_packed, K, N, FN_LAYOUT_LINEAR, _dt(a)), outs=((out, M, N),))
    y = out if out is not None else _new_out(M, N, a)
    _check(_load().baseline_rmsnorm_linear_noalloc(_ptr(a), M, K, _ld(a), _dt(a), _ptr(_vec(g, K, "g")),
                                                   _ptr(W_packed), N, eps, _ptr(y), _ld(y), path, _stream(stream)),
           "baseline_rmsnorm_linear_noalloc")
    return y


def baseline_rmsnorm_glu(a, g, W_packed_gu, F, eps, x_ws=None, out=None, path=FN_PATH_AUTO, stream=None):
    M, K = a.shape
    _baseline_guard("baseline_rmsnorm_glu", a, g, None, W_packed_gu, 2 * F, FN_LAYOUT_GLU, x_ws, out, F)
    x = _ws(a, x_ws)
    o = out if out is not None else _new_out(M, F, a)
    _check(_load().baseline_rmsnorm_glu(_ptr(a), M, K, _ld(a), _dt(a), _ptr(_vec(g, K, "g")), _ptr(W_packed_gu),
                                        F, eps, _ptr(x), _ptr(o), _ld(o), path, _stream(stream)),
           "baseline_rmsnorm_glu")
    return o


def baseline_layernorm_linear(a, g, beta, W_packed, N, eps, x_ws=None, out=None, path=FN_PATH_AUTO,
                              stream=None):
    M, K = a.shape
    _baseline_guard("baseline_layernorm_linear", a, g, beta, W_packed, N, FN_LAYOUT_LINEAR, x_ws, out, N)
    x = _ws(a, x_ws)
    y = out if out is not None else _new_out(M, N, a)
    _check(_load().baseline_layernorm_linear(_ptr(a), M, K, _ld(a), _dt(a), _ptr(_vec(g, K, "g")),
                                             _ptr(_vec(beta, K, "beta")), _ptr(W_packed), N, eps, _ptr(x),
                                             _ptr(y), _ld(y), path, _stream(stream)),
           "baseline_layernorm_linear")
    return y
