"""FlashNorm CPU oracle (fp64) -- TEST INFRASTRUCTURE ONLY.

Plain, slow, obviously correct reference for the norm-then-project hot path of
"FlashNorm: Fast Normalization for Transformers" (arXiv 2407.09577), written in C
(``flashnorm_oracle.c``) and driven from here through ctypes.  Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import
this package.  It shares no code with the GPU library in
``paper_2407_09577_amd/``: neither imports, includes or links the other.

Every function takes the values the GPU receives (bf16 or fp32 tensors, fp32
``g``/``beta``, the fp32 ``eps``) and computes in fp64.  ``rows`` selects a subset
of input rows (sampled parity at full workload sizes); the result has one row
per selected input row.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "flashnorm_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

STORAGE_F32 = 0
STORAGE_BF16 = 1


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no fast-math, no FP contraction)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-shared", "-fPIC",
               "-fvisibility=hidden", _SRC, "-o", tmp, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    I = ctypes.c_int64
    D = ctypes.c_double
    lib.fn_oracle_num_threads.argtypes = []
    lib.fn_oracle_num_threads.restype = ctypes.c_int
    lib.fn_oracle_rms.argtypes = [P, I, D]
    lib.fn_oracle_rms.restype = D
    for name in ("fn_oracle_rmsnorm_linear", "fn_oracle_weightless", "fn_oracle_deferred"):
        getattr(lib, name).argtypes = [P, I, I, P, P, I, D, P, P, I, P]
        getattr(lib, name).restype = None
    lib.fn_oracle_rmsnorm_swiglu.argtypes = [P, I, I, P, P, I, D, P, I, P]
    lib.fn_oracle_rmsnorm_swiglu.restype = None
    for name in ("fn_oracle_layernorm_linear", "fn_oracle_layernorm_linear_deferred"):
        getattr(lib, name).argtypes = [P, I, I, P, P, P, I, D, P, P, I, P]
        getattr(lib, name).restype = None
    for name in ("fn_oracle_rmsnorm_glu_act", "fn_oracle_glu_act_deferred"):
        getattr(lib, name).argtypes = [P, I, I, P, P, I, D, ctypes.c_int, P, I, P]
        getattr(lib, name).restype = None
    lib.fn_oracle_rmsnorm_ffn.argtypes = [P, I, I, P, P, I, P, I, D, ctypes.c_int, P, I, P]
    lib.fn_oracle_rmsnorm_ffn.restype = None
    lib.fn_oracle_round_bf16.argtypes = [D]
    lib.fn_oracle_round_bf16.restype = D
    lib.fn_oracle_round_f32.argtypes = [D]
    lib.fn_oracle_round_f32.restype = D
    lib.fn_oracle_fold.argtypes = [P, P, P, I, I, ctypes.c_int, P, P, P]
    lib.fn_oracle_fold.restype = None
    _lib = lib
    return lib


def _f64(x) -> np.ndarray:
    """fp64 C-contiguous copy of a numpy array or a (CPU) torch tensor of any float dtype."""
    if x is None:
        return None
    if hasattr(x, "detach"):  # torch tensor: bf16 has no numpy dtype, go through fp32 (exact)
        import torch
        x = x.detach().to("cpu", torch.float64).numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _ptr(x):
    return None if x is None else x.ctypes.data_as(ctypes.c_void_p)


def _rows(rows, M):
    if rows is None:
        return None, M
    r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    if r.ndim != 1 or (r.size and (r.min() < 0 or r.max() >= M)):
        raise ValueError("rows must be a 1-D list of indices into a")
    return r, int(r.size)


def _eps(eps) -> float:
    # the kernels receive eps as an fp32 scalar; the oracle uses that exact value
    return float(np.float32(eps))


def num_threads() -> int:
    """OpenMP threads the oracle's row loops use."""
    return int(_load().fn_oracle_num_threads())


def rms(a, eps: float = 0.0) -> float:
    """RMSe(a) = sqrt(eps + mean(a^2)) of one row (App. "RMS with epsilon")."""
    a = _f64(a).ravel()
    return _load().fn_oracle_rms(_ptr(a), a.size, float(eps))


def _linear_like(fn, a, g, W, eps, bias, rows):
    a, g, W, bias = _f64(a), _f64(g), _f64(W), _f64(bias)
    M, K = a.shape
    K2, N = W.shape
    if K2 != K or g.shape != (K,) or (bias is not None and bias.shape != (N,)):
        raise ValueError("shape mismatch")
    r, nr = _rows(rows, M)
    y = np.empty((nr, N), dtype=np.float64)
    fn(_ptr(a), M, K, _ptr(g), _ptr(W), N, _eps(eps), _ptr(bias), _ptr(r), nr, _ptr(y))
    return y


def rmsnorm_linear(a, g, W, eps, bias=None, rows=None) -> np.ndarray:
    """Standard form (a): y = RMSNorm(a; g) W (+ c after the normalisation), Sec. 3.1."""
    return _linear_like(_load().fn_oracle_rmsnorm_linear, a, g, W, eps, bias, rows)


def weightless(a, g, W, eps, bias=None, rows=None) -> np.ndarray:
    """Form (b): y = (a / RMS(a)) W* with W* = diag(g) W in fp64 (Prop. 1). Self-check."""
    return _linear_like(_load().fn_oracle_weightless, a, g, W, eps, bias, rows)


def deferred(a, g, W, eps, bias=None, rows=None) -> np.ndarray:
    """Form (c): y = (a W*) / RMS(a) (Prop. 2). Self-check."""
    return _linear_like(_load().fn_oracle_deferred, a, g, W, eps, bias, rows)


def rmsnorm_swiglu(a, g, Wgu, eps, rows=None) -> np.ndarray:
    """out = silu(x Wg) * (x Wu), x = RMSNorm(a; g), Wgu = [Wg | Wu] of shape [K, 2F] (Sec. 4.1)."""
    a, g, Wgu = _f64(a), _f64(g), _f64(Wgu)
    M, K = a.shape
    K2, N2 = Wgu.shape
    if K2 != K or N2 % 2 or g.shape != (K,):
        raise ValueError("shape mismatch")
    F = N2 // 2
    r, nr = _rows(rows, M)
    out = np.empty((nr, F), dtype=np.float64)
    _load().fn_oracle_rmsnorm_swiglu(_ptr(a), M, K, _ptr(g), _ptr(Wgu), F, _eps(eps), _ptr(r), nr, _ptr(out))
    return out


GLU_SWIGLU, GLU_REGLU, GLU_BILINEAR, FFN_RELU = 0, 1, 2, 3


def _glu_like(fn, a, g, Wgu, eps, act, rows):
    a, g, Wgu = _f64(a), _f64(g), _f64(Wgu)
    M, K = a.shape
    K2, N2 = Wgu.shape
    if K2 != K or N2 % 2 or g.shape != (K,) or act not in (GLU_SWIGLU, GLU_REGLU, GLU_BILINEAR):
        raise ValueError("shape mismatch or unknown act")
    F = N2 // 2
    r, nr = _rows(rows, M)
    out = np.empty((nr, F), dtype=np.float64)
    fn(_ptr(a), M, K, _ptr(g), _ptr(Wgu), F, _eps(eps), int(act), _ptr(r), nr, _ptr(out))
    return out


def rmsnorm_glu_act(a, g, Wgu, eps, act, rows=None) -> np.ndarray:
    """out = act(x Wg) * (x Wu), x = RMSNorm(a; g); act = silu, ReLU or identity (Sec. 4.1, App.)."""
    return _glu_like(_load().fn_oracle_rmsnorm_glu_act, a, g, Wgu, eps, act, rows)


def glu_act_deferred(a, g, Wgu, eps, act, rows=None) -> np.ndarray:
    """The same with W* = diag(g) W and the scale deferred (1/MS for ReGLU / bilinear). Self-check."""
    return _glu_like(_load().fn_oracle_glu_act_deferred, a, g, Wgu, eps, act, rows)


def rmsnorm_ffn(a, g, Wup, Wdown, eps, act, rows=None) -> np.ndarray:
    """y = h Wdown after x = RMSNorm(a; g): h = ReLU(x Wup) (act 3) or act(x Wg) * (x Wu) (act 0-2)."""
    a, g, Wup, Wdown = _f64(a), _f64(g), _f64(Wup), _f64(Wdown)
    M, K = a.shape
    K2, NU = Wup.shape
    F, N = Wdown.shape
    if K2 != K or g.shape != (K,) or act not in (0, 1, 2, 3) or NU != (F if act == FFN_RELU else 2 * F):
        raise ValueError("shape mismatch or unknown act")
    r, nr = _rows(rows, M)
    y = np.empty((nr, N), dtype=np.float64)
    _load().fn_oracle_rmsnorm_ffn(_ptr(a), M, K, _ptr(g), _ptr(Wup), F, _ptr(Wdown), N, _eps(eps), int(act),
                                  _ptr(r), nr, _ptr(y))
    return y


def rope(x, h, pos, cos_tab, sin_tab) -> np.ndarray:
    """Rotary position embedding of every h-wide head of each row of x (Sec. 4.2 with the
    rotation of the RoPE paper): row i is a token at position pos[i]; within each head the
    consecutive pairs (x_2j, x_2j+1) turn by the angle whose cosine and sine are
    cos_tab[pos[i], j] and sin_tab[pos[i], j]:
        y_2j = x_2j cos - x_2j+1 sin,   y_2j+1 = x_2j sin + x_2j+1 cos.
    A row whose position lies outside the table is NaN."""
    x, c_tab, s_tab = _f64(x), _f64(cos_tab), _f64(sin_tab)
    M, N = x.shape
    if h % 2 or N % h or c_tab.shape != s_tab.shape or c_tab.shape[1] != h // 2:
        raise ValueError("shape mismatch")
    pos = np.asarray(pos).ravel()
    out = np.empty_like(x)
    for i in range(M):
        p = int(pos[i])
        if not 0 <= p < c_tab.shape[0]:
            out[i] = np.nan
            continue
        pairs = x[i].reshape(N // h, h // 2, 2)  # [head, j, (even, odd)]
        c, s = c_tab[p], s_tab[p]
        out[i, 0::2] = (pairs[:, :, 0] * c - pairs[:, :, 1] * s).ravel()
        out[i, 1::2] = (pairs[:, :, 0] * s + pairs[:, :, 1] * c).ravel()
    return out


def rmsnorm_qkv_rope(a, g, W, eps, Hq, Hkv, h, pos, cos_tab, sin_tab, q_scale, bias=None,
                     rows=None) -> np.ndarray:
    """Standard form of Fig. 5(a): x = RMSNorm(a; g), t = x W (+ c), W = [Wq | Wk | Wv] with Hq
    query heads and Hkv key/value heads of width h; Q and K heads rotated by RoPE at each
    row's position, Q also multiplied by q_scale (the 1/sqrt(h) of the attention scores).
    V is t itself."""
    qk = (Hq + Hkv) * h
    if _f64(W).shape[1] != (Hq + 2 * Hkv) * h:
        raise ValueError("W must have (Hq + 2 Hkv) h columns")
    t = rmsnorm_linear(a, g, W, eps, bias=bias, rows=rows)
    p = np.asarray(pos).ravel()
    if rows is not None:
        p = p[np.asarray(rows, dtype=np.int64)]
    out = t.copy()
    out[:, :qk] = rope(t[:, :qk], h, p, cos_tab, sin_tab)
    out[:, :Hq * h] *= float(np.float32(q_scale))
    return out


def qkv_rope_deferred(a, g, W, eps, Hq, Hkv, h, pos, cos_tab, sin_tab, q_scale, rows=None) -> np.ndarray:
    """Deferred form of Fig. 5(b): z = a W* with W* = diag(g) W, then RoPE with per-token tables
    cos/RMSe(a) and sin/RMSe(a) (times q_scale for Q); V is z / RMSe(a). Self-check."""
    a, g, W = _f64(a), _f64(g), _f64(W)
    r, nr = _rows(rows, a.shape[0])
    if r is None:
        r = np.arange(nr)
    a = a[r]
    p = np.asarray(pos).ravel()[r]
    qk = (Hq + Hkv) * h
    z = a @ (g[:, None] * W)
    s = np.array([1.0 / rms(row, _eps(eps)) for row in a])
    c_tab, s_tab = _f64(cos_tab), _f64(sin_tab)
    valid = (p >= 0) & (p < c_tab.shape[0])
    pc = np.where(valid, p, 0)
    c_rows = np.where(valid[:, None], c_tab[pc] * s[:, None], np.nan)  # per-token tables
    s_rows = np.where(valid[:, None], s_tab[pc] * s[:, None], np.nan)
    out = z * s[:, None]
    out[:, :qk] = rope(z[:, :qk], h, np.arange(nr), c_rows, s_rows)
    out[:, :Hq * h] *= float(np.float32(q_scale))
    return out


def _head_rmsnorm(t, h, w, eps_head):
    """RMSNorm of every h-wide head of each row of t (the QK-norm / QKV-norm of Sec. 4.3 and
    Sec. 3.3's QKV-normalization): t_head / sqrt(eps_head + mean(t_head^2)) * w, w of length h."""
    t, w = _f64(t), _f64(w)
    M, N = t.shape
    heads = t.reshape(M, N // h, h)
    ms = np.mean(heads * heads, axis=2, keepdims=True)
    return (heads / np.sqrt(_eps(eps_head) + ms) * w).reshape(M, N)


def rmsnorm_qkv_headnorm(a, g, W, eps, Hq, Hkv, h, gq, gk, gv, eps_head, pos=None, cos_tab=None, sin_tab=None,
                         q_scale=1.0, rows=None) -> np.ndarray:
    """Standard form (Fig. 6(a) with per-head second norms): x = RMSNorm(a; g), t = x W with
    W = [Wq | Wk | Wv]; every Q head RMS-normalised with weight gq, every K head with gk (QK-norm),
    every V head with gv when gv is given (QKV-normalization), else V = t; then RoPE on Q and K
    when positions are given, and Q times q_scale."""
    qe, ke = Hq * h, (Hq + Hkv) * h
    if _f64(W).shape[1] != (Hq + 2 * Hkv) * h:
        raise ValueError("W must have (Hq + 2 Hkv) h columns")
    t = rmsnorm_linear(a, g, W, eps, rows=rows)
    out = t.copy()
    out[:, :qe] = _head_rmsnorm(t[:, :qe], h, gq, eps_head)
    out[:, qe:ke] = _head_rmsnorm(t[:, qe:ke], h, gk, eps_head)
    if gv is not None:
        out[:, ke:] = _head_rmsnorm(t[:, ke:], h, gv, eps_head)
    if pos is not None:
        p = np.asarray(pos).ravel()
        if rows is not None:
            p = p[np.asarray(rows, dtype=np.int64)]
        out[:, :ke] = rope(out[:, :ke], h, p, cos_tab, sin_tab)
    out[:, :qe] *= float(np.float32(q_scale))
    return out


def qkv_headnorm_cancelled(a, g, W, eps, Hq, Hkv, h, gq, gk, gv, eps_head, pos=None, cos_tab=None,
                           sin_tab=None, q_scale=1.0, rows=None) -> np.ndarray:
    """Prop. 3 form (Fig. 6(b)): the per-head norms act on z = a W* (W* = diag(g) W) directly,
    the input RMSNorm's scale dropped; V without gv keeps z / RMSe(a). Equal to the standard
    form when eps_head = 0 (the epsilon caveat otherwise). Self-check."""
    a, g, W = _f64(a), _f64(g), _f64(W)
    r, nr = _rows(rows, a.shape[0])
    if r is None:
        r = np.arange(nr)
    a = a[r]
    qe, ke = Hq * h, (Hq + Hkv) * h
    z = a @ (g[:, None] * W)
    out = z.copy()
    out[:, :qe] = _head_rmsnorm(z[:, :qe], h, gq, eps_head)
    out[:, qe:ke] = _head_rmsnorm(z[:, qe:ke], h, gk, eps_head)
    if gv is not None:
        out[:, ke:] = _head_rmsnorm(z[:, ke:], h, gv, eps_head)
    else:
        out[:, ke:] = z[:, ke:] / np.array([rms(row, _eps(eps)) for row in a])[:, None]
    if pos is not None:
        out[:, :ke] = rope(out[:, :ke], h, np.asarray(pos).ravel()[r], cos_tab, sin_tab)
    out[:, :qe] *= float(np.float32(q_scale))
    return out


def rmsnorm_mla_latent(a, g, W, eps, L, g_lat, eps_lat, pos=None, cos_tab=None, sin_tab=None,
                       rows=None) -> np.ndarray:
    """Standard form of the MLA down-projection with latent normalization (Sec. 3.3, the
    paragraph on MLA): x = RMSNorm(a; g), t = x W with W = [W_lat | W_rope]; the first L
    columns (the latent) are RMS-normalised over their whole width with weight g_lat:
    t_lat / sqrt(eps_lat + mean(t_lat^2)) * g_lat; the remaining R columns (the shared
    rotary key, one head of width R; R may be 0) are rotated by RoPE at each row's
    position and carry no second norm."""
    t = rmsnorm_linear(a, g, W, eps, rows=rows)
    R = t.shape[1] - L
    if L < 1 or R < 0 or R % 2:
        raise ValueError("need 0 < L <= N and an even N - L")
    out = t.copy()
    out[:, :L] = _head_rmsnorm(t[:, :L], L, g_lat, eps_lat)
    if R:
        p = np.asarray(pos).ravel()
        if rows is not None:
            p = p[np.asarray(rows, dtype=np.int64)]
        out[:, L:] = rope(t[:, L:], R, p, cos_tab, sin_tab)
    return out


def mla_latent_cancelled(a, g, W, eps, L, g_lat, eps_lat, pos=None, cos_tab=None, sin_tab=None,
                         rows=None) -> np.ndarray:
    """Prop. 3 form (Fig. 6(b)) of rmsnorm_mla_latent: the latent norm acts on z = a W*
    (W* = diag(g) W) directly, the input RMSNorm dropped; the rotary columns, which no norm
    follows, keep z / RMSe(a). Equal to the standard form when eps_lat = 0 (the epsilon
    caveat otherwise). Self-check."""
    a, g, W = _f64(a), _f64(g), _f64(W)
    r, nr = _rows(rows, a.shape[0])
    if r is None:
        r = np.arange(nr)
    a = a[r]
    z = a @ (g[:, None] * W)
    R = z.shape[1] - L
    out = z.copy()
    out[:, :L] = _head_rmsnorm(z[:, :L], L, g_lat, eps_lat)
    if R:
        s = np.array([1.0 / rms(row, _eps(eps)) for row in a])
        out[:, L:] = rope(z[:, L:] * s[:, None], R, np.asarray(pos).ravel()[r], cos_tab, sin_tab)
    return out


def _ln_like(fn, a, g, beta, W, eps, bias, rows):
    a, g, beta, W, bias = _f64(a), _f64(g), _f64(beta), _f64(W), _f64(bias)
    M, K = a.shape
    K2, N = W.shape
    if K2 != K or g.shape != (K,) or beta.shape != (K,):
        raise ValueError("shape mismatch")
    r, nr = _rows(rows, M)
    y = np.empty((nr, N), dtype=np.float64)
    fn(_ptr(a), M, K, _ptr(g), _ptr(beta), _ptr(W), N, _eps(eps), _ptr(bias), _ptr(r), nr, _ptr(y))
    return y


def layernorm_linear(a, g, beta, W, eps, bias=None, rows=None) -> np.ndarray:
    """Standard LayerNorm -> linear: x = (a - mu)/sqrt(var + eps) * g + beta, y = x W (+ c)."""
    return _ln_like(_load().fn_oracle_layernorm_linear, a, g, beta, W, eps, bias, rows)


def layernorm_linear_deferred(a, g, beta, W, eps, bias=None, rows=None) -> np.ndarray:
    """Deferred LayerNorm -> linear: ((a W*) - mu colsum(W*)) / sigma + beta W (+ c). Self-check."""
    return _ln_like(_load().fn_oracle_layernorm_linear_deferred, a, g, beta, W, eps, bias, rows)


def round_bf16(x) -> np.ndarray:
    """Round fp64 values to the nearest bfloat16 value (ties to even), returned as fp64."""
    f = _load().fn_oracle_round_bf16
    x = np.asarray(x, dtype=np.float64)
    return np.vectorize(f, otypes=[np.float64])(x) if x.ndim else np.float64(f(float(x)))


def fold(W, g, beta=None, storage: int = STORAGE_BF16):
    """Expected fold (Prop. 1, Sec. 3.4): stored W* = round(g_k W[k,n]) in the storage type,
    colsum of the stored W*, and c* = beta W with the unfolded W (None without beta)."""
    W, g, beta = _f64(W), _f64(g), _f64(beta)
    K, N = W.shape
    Ws = np.empty((K, N), dtype=np.float64)
    colsum = np.empty(N, dtype=np.float64)
    cstar = np.empty(N, dtype=np.float64) if beta is not None else None
    _load().fn_oracle_fold(_ptr(W), _ptr(g), _ptr(beta), K, N, int(storage), _ptr(Ws), _ptr(colsum), _ptr(cstar))
    return Ws, colsum, cstar
