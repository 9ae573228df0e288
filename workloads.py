"""Seeded synthetic inputs shaped like the LoGra paper's workloads.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic, so both the HIP path's tests and the float64 oracle can
consume what it produces.  The paper's activations and gradients come from
Llama3-8B-Instruct / GPT-2 on OpenWebText (Sec. 4.2), which are not available
here; these Gaussian tensors of the same layer shapes stand in for them.

Host generation uses numpy's Philox counter-based generator; device
generation (for the multi-GB workloads) uses torch's seeded CUDA generator.
bf16 data on the host is carried as uint16 bit patterns, produced from fp32
by round-to-nearest-even.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

# --------------------------------------------------------------------------
# Layer shapes (n_in -> n_out) of the models the paper logs (Sec. 4.2).
# --------------------------------------------------------------------------
LLAMA3_8B_BLOCK = (
    ("q", 4096, 4096),
    ("k", 4096, 1024),
    ("v", 4096, 1024),
    ("o", 4096, 4096),
    ("gate", 4096, 14336),
    ("up", 4096, 14336),
    ("down", 14336, 4096),
)
GPT2_SMALL_BLOCK = (
    ("qkv", 768, 2304),
    ("out", 768, 768),
    ("fc", 768, 3072),
    ("proj", 3072, 768),
)


@dataclass(frozen=True)
class Workload:
    """A named synthetic workload: layer set, batch, precision and laws."""
    name: str
    layers: tuple              # ((name, n_in, n_out), ...) for one block
    blocks: int
    B: int                     # examples per batch
    T: int                     # padded tokens per example
    len_lo: int                # valid length ~ U{len_lo..len_hi} (right padding)
    len_hi: int
    k_in: int
    k_out: int
    x_std: float
    dy_std: float
    dtype: str                 # "f32" or "bf16"
    extra: dict = field(default_factory=dict)

    @property
    def n_layers(self) -> int:
        return len(self.layers) * self.blocks

    @property
    def D(self) -> int:
        return self.k_in * self.k_out


WORKLOADS = {
    # One 64->64 fp32 layer, 4 train + 2 test examples of 16 tokens, k = 8,
    # damping 1e-3 x mean eigenvalue, scores 2 x 4 and top-1 per query.
    "tiny_f32": Workload("tiny_f32", (("lin", 64, 64),), 1, 4, 16, 16, 16, 8, 8, 1.0, 1e-2,
                         "f32", {"Q": 2, "damp": 1e-3, "topk": 1}),
    # GPT-2-small logging: 12 blocks x 4 linears, B=32, T=512, lengths U{64..512}, k = 16.
    "gpt2_small_log": Workload("gpt2_small_log", GPT2_SMALL_BLOCK, 12, 32, 512, 64, 512, 16, 16,
                               1.0, 1e-3, "bf16"),
    # One Llama3-8B block, 7 linears, B=16, T=1024 all valid, k = 64.
    "llama3_8b_block": Workload("llama3_8b_block", LLAMA3_8B_BLOCK, 1, 16, 1024, 1024, 1024, 64, 64,
                                1.0, 1e-4, "bf16"),
    # Full 32-block Llama3-8B logging stream: 224 layers, B=8, lengths U{128..2048}, k = 16,
    # 65,536 examples, bf16 store of 57,344 dims per example.
    "llama3_8b_stream": Workload("llama3_8b_stream", LLAMA3_8B_BLOCK, 32, 8, 2048, 128, 2048, 16, 16,
                                 1.0, 1e-4, "bf16", {"examples": 65536}),
    # Influence scoring at scale: 500,000 stored x 1,024 test gradients of 57,344 dims
    # (224 blocks of 256), per-block scale factors U[0.1, 10], covariances from 4,096
    # gradients, damping 0.1 x mean eigenvalue, top-100 per query.
    "llama3_8b_scores": Workload("llama3_8b_scores", LLAMA3_8B_BLOCK, 32, 0, 0, 0, 0, 16, 16,
                                 1.0, 1.0, "bf16",
                                 {"N_train": 500_000, "Q": 1024, "N_cov": 4096, "damp": 0.1,
                                  "topk": 100, "scale_lo": 0.1, "scale_hi": 10.0}),
}


# --------------------------------------------------------------------------
# Host generation (numpy Philox)
# --------------------------------------------------------------------------
def rng(seed: int, *stream: int) -> np.random.Generator:
    """Counter-based generator keyed by (seed, stream ids)."""
    key = [int(seed)] + [int(s) for s in stream]
    return np.random.Generator(np.random.Philox(np.random.SeedSequence(key)))


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest, ties to even."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def normal(g: np.random.Generator, shape, std: float, dtype: str) -> np.ndarray:
    """N(0, std^2) samples in the requested storage type (float32 or bf16 bits)."""
    a = (g.standard_normal(size=shape, dtype=np.float32) * np.float32(std)).astype(np.float32)
    return a if dtype == "f32" else f32_to_bf16_bits(a)


def lengths(g: np.random.Generator, B: int, lo: int, hi: int) -> np.ndarray:
    """Valid lengths uniform on the integers lo..hi inclusive."""
    return g.integers(lo, hi + 1, size=B, dtype=np.int64)


def mask_from_lengths(lens: np.ndarray, T: int) -> np.ndarray:
    """Right padding: mask[b, t] = 1 iff t < len_b."""
    return (np.arange(T)[None, :] < np.asarray(lens)[:, None]).astype(np.uint8)


def projection(g: np.random.Generator, k: int, n: int, dtype: str) -> np.ndarray:
    """Random projection with i.i.d. N(0, 1/k) entries (Sec. 3.2 random init)."""
    return normal(g, (k, n), 1.0 / np.sqrt(k), dtype)


def layer_inputs(seed: int, layer: int, B: int, T: int, n_in: int, n_out: int, k_in: int,
                 k_out: int, x_std: float, dy_std: float, dtype: str,
                 lens: np.ndarray | None = None) -> dict:
    """x [B,T,n_in], dy [B,T,n_out], p_in [k_in,n_in], p_out [k_out,n_out], mask [B,T]."""
    gx = rng(seed, 1, layer)
    gp = rng(seed, 2, layer)
    out = {
        "x": normal(gx, (B, T, n_in), x_std, dtype),
        "dy": normal(gx, (B, T, n_out), dy_std, dtype),
        "p_in": projection(gp, k_in, n_in, dtype),
        "p_out": projection(gp, k_out, n_out, dtype),
    }
    out["mask"] = None if lens is None else mask_from_lengths(lens, T)
    return out


def block_scales(seed: int, n_blocks: int, lo: float, hi: float) -> np.ndarray:
    """One scale factor per layer block, uniform on [lo, hi]."""
    return rng(seed, 3).uniform(lo, hi, size=n_blocks).astype(np.float32)


def scaled_gradients(seed: int, stream: int, rows: int, block: int, scales: np.ndarray,
                     dtype: str = "bf16") -> np.ndarray:
    """rows x (len(scales) * block) gradients, N(0,1) scaled per block, host side."""
    g = rng(seed, 4, stream)
    a = g.standard_normal(size=(rows, len(scales), block), dtype=np.float32)
    a = (a * scales[None, :, None]).reshape(rows, -1)
    return a if dtype == "f32" else f32_to_bf16_bits(a)


# --------------------------------------------------------------------------
# Device generation (torch; multi-GB tensors are drawn on the GPU)
# --------------------------------------------------------------------------
def torch_generator(seed: int, *stream: int, device="cuda"):
    import torch
    s = int(np.random.SeedSequence([int(seed)] + [int(x) for x in stream]).generate_state(1)[0])
    g = torch.Generator(device=device)
    g.manual_seed(s)
    return g


def device_normal_(out, std: float, gen, chunk_elems: int = 1 << 28):
    """Fill a device tensor (bf16 or fp32) with N(0, std^2), drawn in fp32 and rounded RNE."""
    import torch
    flat = out.view(-1)
    n = flat.numel()
    for s in range(0, n, chunk_elems):
        e = min(n, s + chunk_elems)
        tmp = torch.randn(e - s, generator=gen, device=out.device, dtype=torch.float32)
        if std != 1.0:
            tmp.mul_(std)
        flat[s:e].copy_(tmp)
    return out


def device_scaled_rows_(out, scales, block: int, gen, rows_per_chunk: int = 4096):
    """Fill out [rows, n_blocks*block] (bf16) with N(0,1) * scales[block], drawn in fp32."""
    import torch
    rows, D = out.shape
    nb = D // block
    sc = torch.as_tensor(np.asarray(scales, dtype=np.float32), device=out.device)
    for r0 in range(0, rows, rows_per_chunk):
        r1 = min(rows, r0 + rows_per_chunk)
        tmp = torch.randn((r1 - r0, nb, block), generator=gen, device=out.device,
                          dtype=torch.float32)
        tmp.mul_(sc[None, :, None])
        out[r0:r1].copy_(tmp.view(r1 - r0, D))
    return out


def spd_matrix(seed: int, D: int, rank: int, scale: float = 1.0) -> np.ndarray:
    """A random symmetric PSD fp32 matrix with `rank` nonzero eigenvalues (log-uniform in
    [1e-2, 1] x scale) and uniformly random eigenvectors; exactly symmetric after rounding."""
    g = rng(seed, 5, D, rank)
    q, _ = np.linalg.qr(g.standard_normal((D, rank)))
    ev = scale * np.exp(g.uniform(np.log(1e-2), 0.0, size=rank))
    s = (q * ev) @ q.T
    s = np.triu(s.astype(np.float32))
    return s + np.triu(s, 1).T


def orthogonal(g: np.random.Generator, n: int) -> np.ndarray:
    """A uniformly random n x n orthogonal matrix (QR of a Gaussian, signs fixed), float64."""
    q, r = np.linalg.qr(g.standard_normal((n, n)))
    return q * np.sign(np.diag(r))


def spectral_matrix(seed: int, n: int, decay: float, scale: float = 1.0) -> np.ndarray:
    """Symmetric fp32 U diag(scale * decay^i) U^T with a random orthogonal U: a covariance
    whose top eigenvectors are well separated (ratio `decay` between neighbours); exactly
    symmetric after rounding."""
    u = orthogonal(rng(seed, 6, n), n)
    s = (u * (scale * decay ** np.arange(n))) @ u.T
    s = np.triu(s.astype(np.float32))
    return s + np.triu(s, 1).T


def structured_activations(g: np.random.Generator, B: int, T: int, n: int, decay: float, dtype: str):
    """Activations a_t = U (s * z_t), z ~ N(0, I), s_i = decay^(i / 2), U random orthogonal: the
    token covariance U diag(decay^i) U^T has a decaying spectrum, like the activations of a
    trained network (i.i.d. entries would give a flat one with no distinguished top-k)."""
    u = orthogonal(g, n)
    z = g.standard_normal((B, T, n)) * np.sqrt(decay ** np.arange(n))
    a = (z @ u.T).astype(np.float32)
    return f32_to_bf16_bits(a) if dtype == "bf16" else a


def integer_array(g: np.random.Generator, shape, lo: int, hi: int, dtype: str, density: float = 1.0):
    """Small integers in [lo, hi] (exact in bf16/fp32), zeroed with probability 1 - density."""
    a = g.integers(lo, hi + 1, size=shape).astype(np.float32)
    if density < 1.0:
        a *= (g.random(size=shape) < density)
    return a if dtype == "f32" else f32_to_bf16_bits(a)
