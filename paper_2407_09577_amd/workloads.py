"""Seeded synthetic inputs for the FlashNorm norm-then-project workloads.

This module only draws random numbers and casts them: it holds none of the
method's arithmetic, so both the GPU path (through the tests and the benchmark)
and the CPU oracle consume exactly the same tensors without sharing any code.

Recipe (one CPU ``torch.Generator`` seeded per workload, draw order fixed):
``a`` ~ N(mean, 1) of shape [M, K]; ``g`` ~ U(0.5, 1.5) of shape [K]; ``W`` ~ N(0, 1/K)
of shape [K, N] (for a GLU: Wg then Wu, each [K, F], concatenated as [Wg | Wu]);
then ``beta`` ~ N(0, 0.1) of shape [K] for LayerNorm; then, if requested, a random
permutation whose first ``round(frac * M)`` rows of ``a`` are multiplied by the
outlier factor.  Everything is drawn in fp32 and cast once (round to nearest
even) to bf16 where the workload is bf16; ``g`` and ``beta`` stay fp32.  The second
argument of N(., .) is the variance, so W's standard deviation is K^-1/2 and
every output column has unit variance.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import torch

KIND_LINEAR = "linear"
KIND_GLU = "glu"
KIND_LAYERNORM = "layernorm"


@dataclasses.dataclass
class Workload:
    name: str
    kind: str              # "linear" | "glu" | "layernorm"
    a: torch.Tensor        # [M, K], bf16 or fp32, CPU
    g: torch.Tensor        # [K] fp32
    W: torch.Tensor        # [K, N] logical weight (GLU: [K, 2F] = [Wg | Wu]), dtype of a
    eps: float
    beta: Optional[torch.Tensor] = None       # [K] fp32 (LayerNorm only)
    outlier_rows: Optional[torch.Tensor] = None  # int64 row indices scaled as outliers

    @property
    def M(self) -> int:
        return self.a.shape[0]

    @property
    def K(self) -> int:
        return self.a.shape[1]

    @property
    def N(self) -> int:
        """Columns of the logical weight (2F for a GLU)."""
        return self.W.shape[1]

    @property
    def out_features(self) -> int:
        return self.N // 2 if self.kind == KIND_GLU else self.N

    @property
    def dtype(self) -> torch.dtype:
        return self.a.dtype


def weight(K: int, N: int, *, dtype=torch.bfloat16, seed: int = 0) -> torch.Tensor:
    """A further seeded weight [K, N] ~ N(0, 1/K) (e.g. an FFN down projection), drawn in fp32
    and cast once to dtype."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(seed)
    return (torch.randn(K, N, generator=gen, dtype=torch.float32) * K ** -0.5).to(dtype)


def rope_tables(P: int, h: int, base: float = 10000.0):
    """Precomputed RoPE inputs shared by every head: cos and sin of p * base^(-2j/h) for
    positions p < P and pairs j < h/2, evaluated in fp64 and cast once to fp32 ([P, h/2] each).
    These are the caller's tables, inputs of the fused op like the weights."""
    p = torch.arange(P, dtype=torch.float64)[:, None]
    j = torch.arange(h // 2, dtype=torch.float64)[None, :]
    ang = p * base ** (-2.0 * j / h)
    return torch.cos(ang).to(torch.float32), torch.sin(ang).to(torch.float32)


def positions(M: int, seq_len: int) -> torch.Tensor:
    """Token positions of M rows packed as sequences of seq_len tokens: m % seq_len (int32)."""
    return (torch.arange(M, dtype=torch.int64) % seq_len).to(torch.int32)


def make(kind: str, M: int, K: int, N: int, *, dtype=torch.bfloat16, eps: float = 1e-6,
         seed: int = 0, a_mean: float = 0.0, outlier_frac: float = 0.0,
         outlier_scale: float = 20.0, name: str = "") -> Workload:
    """Draw one workload.  For kind == "glu", N is the number of output features F and
    the weight has 2F columns [Wg | Wu]."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(seed)
    a = torch.randn(M, K, generator=gen, dtype=torch.float32)
    if a_mean:
        a = a + a_mean
    g = torch.rand(K, generator=gen, dtype=torch.float32) + 0.5
    std = K ** -0.5
    if kind == KIND_GLU:
        Wg = torch.randn(K, N, generator=gen, dtype=torch.float32) * std
        Wu = torch.randn(K, N, generator=gen, dtype=torch.float32) * std
        W = torch.cat([Wg, Wu], dim=1)
    else:
        W = torch.randn(K, N, generator=gen, dtype=torch.float32) * std
    beta = None
    if kind == KIND_LAYERNORM:
        beta = torch.randn(K, generator=gen, dtype=torch.float32) * (0.1 ** 0.5)
    outliers = None
    if outlier_frac > 0 and M > 0:
        n_out = int(outlier_frac * M)
        outliers = torch.randperm(M, generator=gen)[:n_out].sort().values
        a[outliers] *= outlier_scale
    a = a.to(dtype)
    W = W.to(dtype)
    return Workload(name=name or f"{kind}_{M}x{K}x{N}", kind=kind, a=a, g=g, W=W, eps=eps,
                    beta=beta, outlier_rows=outliers)


# The five synthetic workloads of the benchmark (model-scale shapes; synthetic data).
def tiny_fp32(seed: int = 0) -> Workload:
    """fp32 RMSNorm->linear, a[16,576], W[576,576], eps 1e-6 (deferred vs standard form)."""
    return make(KIND_LINEAR, 16, 576, 576, dtype=torch.float32, eps=1e-6, seed=seed,
                name="tiny_fp32_rmsnorm_linear_16x576x576")


def smollm2_prefill(seed: int = 0) -> Workload:
    """SmolLM2-135M-scale prefill: bf16 a[2048,576] with 1% outlier rows x20, W[576,1536], eps 1e-5."""
    return make(KIND_LINEAR, 2048, 576, 1536, dtype=torch.bfloat16, eps=1e-5, seed=seed,
                outlier_frac=0.01, outlier_scale=20.0,
                name="smollm2_135m_prefill_rmsnorm_linear_2048x576x1536")


def llama7b_qkv_prefill(seed: int = 0) -> Workload:
    """Llama-7B-scale fused QKV prefill: bf16 a[4096,4096], W[4096,12288], eps 1e-6."""
    return make(KIND_LINEAR, 4096, 4096, 12288, dtype=torch.bfloat16, eps=1e-6, seed=seed,
                name="llama7b_qkv_prefill_rmsnorm_linear_4096x4096x12288")


def llama7b_swiglu_decode(M: int = 16, seed: int = 0) -> Workload:
    """Llama-7B-scale decode SwiGLU FFN input: bf16 a[M,4096], [Wg|Wu] of [4096, 2x11008], eps 1e-6.
    The M in {1, 4} cases are the first rows of the M = 16 draw."""
    w = make(KIND_GLU, 16, 4096, 11008, dtype=torch.bfloat16, eps=1e-6, seed=seed,
             name=f"llama7b_swiglu_decode_{M}x4096x11008")
    w.a = w.a[:M].contiguous()
    return w


def layernorm_linear(seed: int = 0) -> Workload:
    """Deferred LayerNorm->linear: bf16 a[4096,4096] ~ N(0.5,1), beta ~ N(0,0.1), W[4096,4096], eps 1e-5."""
    return make(KIND_LAYERNORM, 4096, 4096, 4096, dtype=torch.bfloat16, eps=1e-5, seed=seed,
                a_mean=0.5, name="layernorm_linear_4096x4096x4096")


def mla_kv_down(seed: int = 0) -> Workload:
    """MLA down-projection at DeepSeek-V2 width: bf16 a[4096,5120] ~ N(0,1), W[5120,576] ~ N(0,1/5120)
    = a 512-wide latent and a 64-wide rotary key, g ~ U(0.5,1.5), eps 1e-6."""
    return make(KIND_LINEAR, 4096, 5120, 576, dtype=torch.bfloat16, eps=1e-6, seed=seed,
                name="mla_kv_down_4096x5120x(512+64)")


WORKLOADS = {
    "tiny_fp32": tiny_fp32,
    "smollm2_prefill": smollm2_prefill,
    "llama7b_qkv_prefill": llama7b_qkv_prefill,
    "llama7b_swiglu_decode": llama7b_swiglu_decode,
    "layernorm_linear": layernorm_linear,
    "mla_kv_down": mla_kv_down,
}
