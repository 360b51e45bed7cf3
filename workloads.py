"""Seeded synthetic inputs for the binary-delta matmul.

This module only draws random numbers: it holds none of the operator's
arithmetic (no sign decode, no packing, no products).  Both the test suite
(feeding the oracle and the HIP path) and ``bench.py`` use it.

The paper reports no problem sizes for its BitDelta kernels beyond saying that
they are representative LLM dimensions (Section 4, evaluation set-up), so the
workloads below are LLaMA-7B-shaped stand-ins:

  tiny         x 4x256, W 512x256, one tenant, fp32 output
  decode       x {1,16}x4096, W 4096x4096, one tenant, bf16 output
  mt_decode    x 32x4096, W 11008x4096, 16 tenants, per-row tenant id, bf16 output
  prefill      x 4096x4096, W 4096x4096, one tenant, bf16 output
  mt_prefill   x 4096x4096 as 16 prompts of random length, one tenant per
               prompt drawn from 8, W 4096x4096, bf16 output
  llama_sweep  32 layers x {q,k,v,o 4096x4096; gate,up 11008x4096;
               down 4096x11008}, 8 tenants, 64 token rows, bf16 output

Distributions: x ~ N(0, 1); W ~ N(0, 0.02) (0.02 is the standard deviation);
sign bits i.i.d. Bernoulli(0.5); alpha ~ U(1e-4, 1e-3) per tenant (and per
matrix in the sweep); tenant ids uniform over [0, T).  Normal draws are made in
float32 and rounded to bfloat16 (or, for the fp16 variants of the same shapes,
to IEEE fp16) with round-to-nearest-even.  Draw order inside
one generator: x, W, signs, alpha, tenant ids.

The tiny workload draws its signs as int8 +1/-1 (so that the packer is
exercised); every other workload draws the packed words directly as uniform
uint32 (each bit an independent fair coin).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

LLAMA_MATRICES = (  # name, N (output features), K (input features)
    ("q", 4096, 4096),
    ("k", 4096, 4096),
    ("v", 4096, 4096),
    ("o", 4096, 4096),
    ("gate", 11008, 4096),
    ("up", 11008, 4096),
    ("down", 4096, 11008),
)
LLAMA_LAYERS = 32
LLAMA_TENANTS = 8
LLAMA_ROWS = 64


@dataclass
class Problem:
    """One binary-delta matmul instance (host arrays)."""
    name: str
    x: np.ndarray                    # uint16 [M, K] bf16 bits
    w: np.ndarray                    # uint16 [N, K] bf16 bits
    alpha: np.ndarray                # float32 [T]
    packed: Optional[np.ndarray] = None   # uint32 [T, N, K/32]
    signs: Optional[np.ndarray] = None    # int8 [T, N, K] (+1/-1), tiny only
    tenant_ids: Optional[np.ndarray] = None  # int32 [M] or None
    y_dtype: str = "bf16"            # "f32" or the input type
    dtype: str = "bf16"              # 16-bit type of x and W: "bf16" or "f16"
    meta: dict = field(default_factory=dict)

    @property
    def M(self):
        return self.x.shape[0]

    @property
    def K(self):
        return self.x.shape[1]

    @property
    def N(self):
        return self.w.shape[0]

    @property
    def T(self):
        return self.alpha.shape[0]


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 draws to bfloat16 (nearest-even) and return the bit patterns."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def bf16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> float32 values (exact)."""
    return (np.asarray(h, dtype=np.uint32) << 16).view(np.float32)


def normal_bf16(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    return f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32) * np.float32(std))


def normal_f16(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    """fp32 normal draws rounded to IEEE fp16 (nearest even), as bit patterns."""
    return (rng.standard_normal(shape, dtype=np.float32) * np.float32(std)).astype(np.float16).view(np.uint16)


def half_bits_to_f32(h: np.ndarray, dtype: str) -> np.ndarray:
    """bf16 or fp16 bit patterns -> float32 values (exact)."""
    if dtype == "f16":
        return np.asarray(h, dtype=np.uint16).view(np.float16).astype(np.float32)
    return bf16_bits_to_f32(h)


def uniform_words(rng: np.random.Generator, shape) -> np.ndarray:
    return rng.integers(0, 2**32, size=shape, dtype=np.uint64).astype(np.uint32)


def random_signs_i8(rng: np.random.Generator, shape) -> np.ndarray:
    return np.where(rng.random(shape) < 0.5, 1, -1).astype(np.int8)


def alphas(rng: np.random.Generator, T: int) -> np.ndarray:
    return rng.uniform(1e-4, 1e-3, size=T).astype(np.float32)


def tenant_draw(rng: np.random.Generator, M: int, T: int) -> np.ndarray:
    return rng.integers(0, T, size=M, dtype=np.int64).astype(np.int32)


def prompt_tenant_ids(rng: np.random.Generator, M: int, T: int, prompts: int) -> np.ndarray:
    """Tenant id per row for M token rows that come as `prompts` consecutive
    prompts: lengths from prompts-1 distinct cut points drawn uniformly in
    (0, M), each prompt's tenant uniform over [0, T)."""
    cuts = np.sort(rng.choice(np.arange(1, M), size=prompts - 1, replace=False))
    lengths = np.diff(np.concatenate([[0], cuts, [M]]))
    tenants = rng.integers(0, T, size=prompts, dtype=np.int64)
    return np.repeat(tenants, lengths).astype(np.int32)


def make_problem(M: int, N: int, K: int, T: int = 1, *, seed: int = 0,
                 multi_tenant: bool = False, y_dtype: str = "bf16",
                 x_std: float = 1.0, w_std: float = 0.02,
                 signs_as_int8: bool = False, name: str = "custom",
                 dtype: str = "bf16") -> Problem:
    """Generic generator: x ~ N(0, x_std), W ~ N(0, w_std), Bernoulli signs.
    dtype picks the 16-bit type of x and W; y_dtype "half" means that type."""
    rng = np.random.default_rng(seed)
    normal = normal_f16 if dtype == "f16" else normal_bf16
    x = normal(rng, (M, K), x_std)
    w = normal(rng, (N, K), w_std)
    packed = signs = None
    if signs_as_int8:
        signs = random_signs_i8(rng, (T, N, K))
    else:
        packed = uniform_words(rng, (T, N, K // 32))
    a = alphas(rng, T)
    tid = tenant_draw(rng, M, T) if multi_tenant else None
    if y_dtype == "half":
        y_dtype = dtype
    return Problem(name, x, w, a, packed=packed, signs=signs, tenant_ids=tid,
                   y_dtype=y_dtype, dtype=dtype)


def tiny(seed: int = 0) -> Problem:
    return make_problem(4, 512, 256, 1, seed=seed, y_dtype="f32", signs_as_int8=True,
                        name="tiny 4x256 . 512x256, fp32 out")


def decode(M: int, seed: int = 0, dtype: str = "bf16") -> Problem:
    return make_problem(M, 4096, 4096, 1, seed=seed, name=f"decode M={M} 4096x4096 {dtype}",
                        dtype=dtype, y_dtype=dtype)


def mt_decode(seed: int = 0) -> Problem:
    return make_problem(32, 11008, 4096, 16, seed=seed, multi_tenant=True,
                        name="multi-tenant decode M=32 11008x4096 T=16")


def prefill(seed: int = 0, dtype: str = "bf16") -> Problem:
    return make_problem(4096, 4096, 4096, 1, seed=seed, name=f"prefill 4096^3 {dtype}",
                        dtype=dtype, y_dtype=dtype)


MT_PREFILL = {"M": 4096, "N": 4096, "K": 4096, "T": 8, "prompts": 16}


def mt_prefill(seed: int = 0) -> Problem:
    c = MT_PREFILL
    p = make_problem(c["M"], c["N"], c["K"], c["T"], seed=seed,
                     name="multi-tenant prefill 4096 rows (16 prompts, 8 tenants) x 4096x4096")
    p.tenant_ids = prompt_tenant_ids(np.random.default_rng([seed, 3]), c["M"], c["T"], c["prompts"])
    return p


def llama_shared_inputs(seed: int = 0):
    """x for K=4096 and K=11008 (64 rows each) and the 64 tenant ids."""
    rng = np.random.default_rng([seed, 1])
    x4096 = normal_bf16(rng, (LLAMA_ROWS, 4096), 1.0)
    x11008 = normal_bf16(rng, (LLAMA_ROWS, 11008), 1.0)
    tid = tenant_draw(rng, LLAMA_ROWS, LLAMA_TENANTS)
    return x4096, x11008, tid


def llama_matrix(layer: int, idx: int, shared=None, seed: int = 0) -> Problem:
    """One matrix of the sweep (W, signs, alpha), from its own seed sequence.

    Seed sequences are tagged ([seed, 1] for the shared inputs, [seed, 2, layer,
    idx] per matrix): numpy maps [s] and [s, 0] to the same stream, so untagged
    sub-seeds could replay x as W.
    """
    name, N, K = LLAMA_MATRICES[idx]
    if shared is None:
        shared = llama_shared_inputs(seed)
    x4096, x11008, tid = shared
    rng = np.random.default_rng([seed, 2, layer, idx])
    w = normal_bf16(rng, (N, K), 0.02)
    packed = uniform_words(rng, (LLAMA_TENANTS, N, K // 32))
    a = alphas(rng, LLAMA_TENANTS)
    x = x4096 if K == 4096 else x11008
    return Problem(f"llama L{layer}.{name} {N}x{K} T=8 M=64", x, w, a, packed=packed,
                   tenant_ids=tid, meta={"layer": layer, "matrix": name})


# ---- device-side generation for the benchmark (same recipe, torch RNG) ----

def device_problem(M: int, N: int, K: int, T: int, *, multi_tenant: bool, seed: int,
                   device="cuda", x_std: float = 1.0, w_std: float = 0.02, prompts: int = 0,
                   dtype: str = "bf16"):
    """Same distributions, drawn directly into device memory with torch's RNG.

    Returns a dict of torch tensors: x (bf16 or fp16 [M,K]), w (same, [N,K]),
    packed (int32 [T,N,K/32]), alpha (fp32 [T]), tenant_ids (int32 [M] or None).
    With prompts > 0 the tenant ids follow prompt_tenant_ids (drawn on the host).
    """
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    half = torch.float16 if dtype == "f16" else torch.bfloat16
    x = (torch.randn((M, K), generator=g, device=device, dtype=torch.float32) * x_std).to(half)
    w = (torch.randn((N, K), generator=g, device=device, dtype=torch.float32) * w_std).to(half)
    packed = torch.randint(0, 256, (T, N, K // 32, 4), generator=g, device=device,
                           dtype=torch.uint8).view(torch.int32).reshape(T, N, K // 32)
    alpha = (torch.rand((T,), generator=g, device=device, dtype=torch.float32)
             * 9e-4 + 1e-4)
    tid = None
    if multi_tenant and prompts > 0:
        ids = prompt_tenant_ids(np.random.default_rng([seed, 3]), M, T, prompts)
        tid = torch.from_numpy(ids).to(device)
    elif multi_tenant:
        tid = torch.randint(0, T, (M,), generator=g, device=device, dtype=torch.int32)
    return {"x": x, "w": w, "packed": packed, "alpha": alpha, "tenant_ids": tid}
