"""Seeded synthetic inputs for the LSA hot path.

This module only draws random numbers and stores them in the formats the method consumes:
bfloat16 bit patterns, OCP fp8 e4m3fn codes with one fp32 scale per token, fp32 head weights,
context lengths and page tables. It holds none of the method's arithmetic. Both the oracle
(through the tests and the benchmark's CPU leg) and the HIP library read exactly these arrays.

Distributions (stand-ins for the paper's workloads, which need model activations):
  * indexer queries and keys  ~ N(0, 1) / sqrt(d_I)
  * indexer head weights w    ~ U(0, 1); with signed weights (the head weights are a learned
    projection of either sign) ~ U(-1, 1), every fifth row with all weights <= 0
  * attention queries, latent KV, K, V ~ N(0, 1)
  * fp8 keys: per-token scale sigma = max|k| / 448 (1 for an all-zero key), code = e4m3fn(k / sigma)
    with round-to-nearest-even after clamping to the finite range +-448.

Host draws use numpy's PCG64 seeded by (seed, tensor id, chunk); large device-side tensors use
torch's Philox generator on the GPU seeded from the same triple.
"""
from __future__ import annotations

import numpy as np
import torch

# tensor ids: keep stable, they are part of the seed recipe
T_QI, T_KI, T_W = 1, 2, 3
T_Q, T_KV, T_V = 10, 20, 30          # + layer index
T_CTX, T_PERM = 40, 41
FP8_MAX = 448.0


def rng(seed: int, tensor_id: int, chunk: int = 0) -> np.random.Generator:
    return np.random.default_rng([seed, tensor_id, chunk])


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 array -> bfloat16 bit patterns (uint16), round-to-nearest-even (torch's cast)."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def quantize_fp8_per_token(k: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """float32 [n, d] -> (e4m3fn codes uint8 [n, d], scale float32 [n])."""
    k = np.asarray(k, dtype=np.float32)
    amax = np.abs(k).max(axis=1)
    scale = np.where(amax > 0, amax / np.float32(FP8_MAX), np.float32(1.0)).astype(np.float32)
    y = np.clip(k / scale[:, None], -FP8_MAX, FP8_MAX).astype(np.float32)
    codes = torch.from_numpy(y).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    return codes, scale


def indexer_inputs(seed: int, n_q: int, n_kv: int, n_heads: int, head_dim: int, fp8: bool,
                   signed_weights: bool = False):
    """Indexer query q_I [n_q, H, d] (bf16 bits), weights w [n_q, H] (fp32), key cache
    k_I [n_kv, d] (bf16 bits, or e4m3fn codes plus per-token scale [n_kv]). signed_weights: w ~
    U(-1, 1), and rows 0, 5, 10, ... get -|w| (all of their scores are then <= 0)."""
    s = np.float32(1.0 / np.sqrt(head_dim))
    q = to_bf16_bits(rng(seed, T_QI).standard_normal((n_q, n_heads, head_dim), dtype=np.float32) * s)
    k32 = rng(seed, T_KI).standard_normal((n_kv, head_dim), dtype=np.float32) * s
    w = rng(seed, T_W).random((n_q, n_heads), dtype=np.float32)
    if signed_weights:
        w = (np.float32(2.0) * w - np.float32(1.0)).astype(np.float32)
        w[::5] = -np.abs(w[::5])
    if fp8:
        k, k_scale = quantize_fp8_per_token(k32)
    else:
        k, k_scale = to_bf16_bits(k32), None
    return dict(q=q, w=w, k=k, k_scale=k_scale)


def attention_inputs(seed: int, layer: int, n_q: int, n_kv: int, n_heads: int, d_qk: int,
                     d_v: int, latent: bool):
    """Per-layer attention inputs ~ N(0,1) in bf16 bits: Q [n_q, H, d_qk] and either a shared
    latent KV [n_kv, d_qk] (V is its first d_v columns) or separate K [n_kv, d_qk], V [n_kv, d_v]."""
    q = to_bf16_bits(rng(seed, T_Q + layer).standard_normal((n_q, n_heads, d_qk), dtype=np.float32))
    kv = to_bf16_bits(rng(seed, T_KV + layer).standard_normal((n_kv, d_qk), dtype=np.float32))
    if latent:
        return dict(q=q, kv=kv, v=None)
    v = to_bf16_bits(rng(seed, T_V + layer).standard_normal((n_kv, d_v), dtype=np.float32))
    return dict(q=q, kv=kv, v=v)


def decode_layout(seed: int, batch: int, ctx_lo: int, ctx_hi: int, page_size: int):
    """Context lengths ~ U{ctx_lo..ctx_hi} and a random permutation of all physical pages
    dealt out to the sequences. Returns (ctx_len int32 [batch], page_table int32
    [batch, max_pages] padded with -1, n_phys)."""
    ctx = rng(seed, T_CTX).integers(ctx_lo, ctx_hi + 1, size=batch).astype(np.int32)
    n_pages = (ctx + page_size - 1) // page_size
    n_phys = int(n_pages.sum())
    perm = rng(seed, T_PERM).permutation(n_phys).astype(np.int32)
    max_pages = int(n_pages.max())
    table = np.full((batch, max_pages), -1, np.int32)
    off = 0
    for b in range(batch):
        table[b, :n_pages[b]] = perm[off:off + n_pages[b]]
        off += n_pages[b]
    return ctx, table, n_phys


# ----------------------------------------------------------------------------- device-side draws
def _philox_seed(seed: int, tensor_id: int, chunk: int) -> int:
    return int(np.random.default_rng([seed, tensor_id, chunk]).integers(0, 2**62))


def device_normal_bf16(shape, seed: int, tensor_id: int, device, scale: float = 1.0,
                       rows_per_chunk: int = 8192) -> torch.Tensor:
    """N(0,1)*scale in bf16 on the device, drawn chunk by chunk along dim 0 with torch's Philox
    generator, so a 100 GB input never exists in fp32. Reproducible for a fixed torch build."""
    out = torch.empty(shape, dtype=torch.bfloat16, device=device)
    g = torch.Generator(device=device)
    n = shape[0]
    for c, r0 in enumerate(range(0, n, rows_per_chunk)):
        r1 = min(n, r0 + rows_per_chunk)
        g.manual_seed(_philox_seed(seed, tensor_id, c))
        t = torch.randn((r1 - r0,) + tuple(shape[1:]), generator=g, device=device, dtype=torch.float32)
        if scale != 1.0:
            t.mul_(scale)
        out[r0:r1].copy_(t)
    return out


def device_uniform_f32(shape, seed: int, tensor_id: int, device) -> torch.Tensor:
    g = torch.Generator(device=device)
    g.manual_seed(_philox_seed(seed, tensor_id, 0))
    return torch.rand(shape, generator=g, device=device, dtype=torch.float32)


def device_fp8_keys(n_kv: int, head_dim: int, seed: int, device, rows_per_chunk: int = 65536):
    """Indexer keys ~ N(0,1)/sqrt(d) quantised per token to e4m3fn on the device.
    Returns (codes uint8 [n_kv, d], scale fp32 [n_kv])."""
    codes = torch.empty((n_kv, head_dim), dtype=torch.uint8, device=device)
    scale = torch.empty((n_kv,), dtype=torch.float32, device=device)
    g = torch.Generator(device=device)
    for c, r0 in enumerate(range(0, n_kv, rows_per_chunk)):
        r1 = min(n_kv, r0 + rows_per_chunk)
        g.manual_seed(_philox_seed(seed, T_KI, c))
        k = torch.randn((r1 - r0, head_dim), generator=g, device=device, dtype=torch.float32)
        k.mul_(1.0 / np.sqrt(head_dim))
        amax = k.abs().amax(dim=1)
        s = torch.where(amax > 0, amax / FP8_MAX, torch.ones_like(amax))
        y = (k / s[:, None]).clamp_(-FP8_MAX, FP8_MAX)
        codes[r0:r1] = y.to(torch.float8_e4m3fn).view(torch.uint8)
        scale[r0:r1] = s
    return codes, scale
