"""Seeded synthetic KV-cache workloads for GSRQ.

This module only draws inputs; it holds none of the quantiser's arithmetic.
It is shared by the tests, the oracle-based checks and the benchmark, and it
stands in for the paper's real LLaMA-3-8B KV activations, calibration sets and
gradient norms (Sec. 6.1, 6.2), none of which are available here.

Recipe (every draw from numpy's PCG64, one child SeedSequence per
(workload, layer), always in this order):
  1. key channel scales sigma_c ~ lognormal(0, key_sigma) for c < D;
  2. outlier channels: round(outlier_frac * D) channels chosen without
     replacement, their sigma multiplied by outlier_mult;
  3. keys = N(0, 1) * sigma_c, [N, D];
  4. values = N(0, 1), [N, D];
  5. w_K ~ lognormal(0, 1), [N];   6. w_V ~ lognormal(0, 1), [N];
  7. seed rows for GSKM initialisation: for K then V, for every stage m and
     subspace g, K distinct row indices drawn without replacement.
Data are drawn in float32 and rounded to the workload's storage dtype.
A row is one token's K (or V) vector with all heads concatenated
(D = heads * 128), so one weight per token is shared by every subspace.

Full-cache workloads (many layers of 131072 tokens) draw a layer's tokens on
the GPU (`make_kv_device`: torch's Philox generator seeded from the layer's
SeedSequence; keys N(0,1) * sigma_c, values N(0,1), lognormal weights) with
the channel scales of steps 1-2 above, and calibrate on a separate 4096-token
draw of the same layer (`make_calibration`, numpy, same recipe from step 3 on
with its own stream).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Tuple

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    N: int                  # tokens (rows)
    D: int                  # heads * head_dim
    d: int                  # subvector dimension
    K: int                  # codebook size
    M: int                  # residual stages
    T: int                  # GSKM iterations per stage
    dtype: str              # storage dtype of K/V: "float32" or "float16"
    layers: int = 1
    key_sigma: float = 1.0  # lognormal sigma of the per-channel key scale
    outlier_frac: float = 0.01
    outlier_mult: float = 10.0
    note: str = ""

    @property
    def G(self) -> int:
        return self.D // self.d


WORKLOADS = {
    # 4096 tokens x 1 head x 128, fp32; d=8, K=256, M=2, T=10
    "tiny": Workload("tiny", 4096, 128, 8, 256, 2, 10, "float32",
                     key_sigma=0.5, outlier_frac=0.0,
                     note="4096 tok x 1 head x 128 fp32, d=8 K=256 M=2 T=10"),
    # LLaMA-3-8B single layer: 32768 tokens x 8 KV heads x 128, fp16, 1 bit
    "llama3_8b_layer_1bit": Workload(
        "llama3_8b_layer_1bit", 32768, 1024, 8, 256, 1, 20, "float16",
        note="32768 tok x 8 heads x 128 fp16, d=8 K=256 M=1 (1 bit), weighted GSKM T=20"),
    # full-model cache: 32 layers x 131072 tokens, codebooks from 4096-token slices
    "llama3_8b_cache_1bit": Workload(
        "llama3_8b_cache_1bit", 131072, 1024, 8, 256, 1, 20, "float16", layers=32,
        note="32 layers x 131072 tok x 8 heads x 128 fp16, 1 bit"),
    # rate sweep at d=16: M in {1, 2, 4} -> 0.5 / 1 / 2 bit
    "rate_sweep_d16": Workload(
        "rate_sweep_d16", 65536, 1024, 16, 256, 4, 20, "float16",
        note="65536 tok x 8 heads x 128 fp16, d=16 K=256 M in {1,2,4}"),
    # the paper's own rate configuration: full-head subvectors, K = 256,
    # 32 stages (2 bits); its 12- and 16-stage prefixes are 0.75 and 1 bit
    "paper_rates_d128": Workload(
        "paper_rates_d128", 32768, 1024, 128, 256, 32, 20, "float16",
        note="32768 tok x 8 heads x 128 fp16, d=128 K=256 M=32 (2 bit; 12/16-stage prefixes "
             "are 0.75/1 bit)"),
    # the paper's lowest rate: subvectors of two heads (d = 256), K = 256,
    # 12 stages = 0.375 bit per element
    "paper_rates_d256": Workload(
        "paper_rates_d256", 32768, 1024, 256, 256, 12, 20, "float16",
        note="32768 tok x 8 heads x 128 fp16, d=256 K=256 M=12 (0.375 bit)"),
    # large codebook, full-head vectors
    "large_codebook_d128": Workload(
        "large_codebook_d128", 65536, 1024, 128, 4096, 8, 15, "float16",
        note="65536 tok x 8 heads x 128 fp16, d=128 K=4096 M=8 (0.75 bit)"),
}


def _children(seed: int, workload: str, layer: int) -> np.random.Generator:
    # one independent stream per (workload, layer); the workload name is
    # folded into the entropy so different workloads never share draws
    tag = [ord(c) for c in workload]
    ss = np.random.SeedSequence([seed, layer] + tag)
    return np.random.Generator(np.random.PCG64(ss))


@dataclass
class KVBatch:
    keys: np.ndarray
    values: np.ndarray
    w_keys: np.ndarray
    w_values: np.ndarray
    seeds_keys: np.ndarray     # [M, G, K] int64
    seeds_values: np.ndarray   # [M, G, K] int64
    key_scales: np.ndarray = field(repr=False, default=None)


def draw_seed_rows(rng: np.random.Generator, N: int, K: int, M: int, G: int) -> np.ndarray:
    out = np.empty((M, G, K), dtype=np.int64)
    for m in range(M):
        for g in range(G):
            out[m, g] = rng.choice(N, size=K, replace=False)
    return out


def make_kv(wl: Workload, layer: int = 0, seed: int = 0, N: int | None = None,
            M: int | None = None) -> KVBatch:
    """Draw one layer of keys/values, weights and seed rows for workload wl.

    N and M may be overridden (a shorter slice of the same distribution, or
    fewer stages); the draw order stays the one in the module docstring.
    """
    N = wl.N if N is None else int(N)
    M = wl.M if M is None else int(M)
    D, G, K = wl.D, wl.G, wl.K
    rng = _children(seed, wl.name, layer)
    scales = rng.lognormal(0.0, wl.key_sigma, size=D).astype(np.float32)
    n_out = int(round(wl.outlier_frac * D))
    if n_out > 0:
        ch = rng.choice(D, size=n_out, replace=False)
        scales[ch] *= np.float32(wl.outlier_mult)
    keys = rng.standard_normal((N, D), dtype=np.float32) * scales[None, :]
    values = rng.standard_normal((N, D), dtype=np.float32)
    w_k = rng.lognormal(0.0, 1.0, size=N).astype(np.float32)
    w_v = rng.lognormal(0.0, 1.0, size=N).astype(np.float32)
    sk = draw_seed_rows(rng, N, K, M, G)
    sv = draw_seed_rows(rng, N, K, M, G)
    dt = np.float16 if wl.dtype == "float16" else np.float32
    return KVBatch(keys.astype(dt), values.astype(dt), w_k, w_v, sk, sv, scales)


def small_case(N: int, D: int, d: int, K: int, M: int, seed: int = 0,
               dtype=np.float32, key_sigma: float = 0.5,
               weights: bool = True) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """A small generic case (X [N, D], w [N], seed rows [M, G, K]) for tests."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, N, D, d, K, M])))
    scales = rng.lognormal(0.0, key_sigma, size=D).astype(np.float32)
    X = (rng.standard_normal((N, D), dtype=np.float32) * scales[None, :]).astype(dtype)
    w = rng.lognormal(0.0, 1.0, size=N).astype(np.float32) if weights else np.ones(N, np.float32)
    seeds = draw_seed_rows(rng, N, K, M, D // d)
    return X, w, seeds


def layer_scales(wl: Workload, layer: int = 0, seed: int = 0) -> np.ndarray:
    """Key channel scales of a layer: steps 1-2 of the recipe, from the same
    stream as make_kv (so both see the same channels)."""
    rng = _children(seed, wl.name, layer)
    scales = rng.lognormal(0.0, wl.key_sigma, size=wl.D).astype(np.float32)
    n_out = int(round(wl.outlier_frac * wl.D))
    if n_out > 0:
        ch = rng.choice(wl.D, size=n_out, replace=False)
        scales[ch] *= np.float32(wl.outlier_mult)
    return scales


def make_calibration(wl: Workload, layer: int = 0, seed: int = 0, N: int = 4096,
                     M: int | None = None) -> KVBatch:
    """A calibration slice of a layer: N tokens drawn from their own stream
    (steps 3-7 of the recipe) with the layer's channel scales."""
    M = wl.M if M is None else int(M)
    scales = layer_scales(wl, layer, seed)
    rng = _children(seed, wl.name + "/calibration", layer)
    keys = rng.standard_normal((N, wl.D), dtype=np.float32) * scales[None, :]
    values = rng.standard_normal((N, wl.D), dtype=np.float32)
    w_k = rng.lognormal(0.0, 1.0, size=N).astype(np.float32)
    w_v = rng.lognormal(0.0, 1.0, size=N).astype(np.float32)
    sk = draw_seed_rows(rng, N, wl.K, M, wl.G)
    sv = draw_seed_rows(rng, N, wl.K, M, wl.G)
    dt = np.float16 if wl.dtype == "float16" else np.float32
    return KVBatch(keys.astype(dt), values.astype(dt), w_k, w_v, sk, sv, scales)


def make_kv_device(wl: Workload, layer: int = 0, seed: int = 0, device="cuda",
                   N: int | None = None):
    """(keys, values, w_keys, w_values) of one layer drawn on the device with
    torch's generator seeded from the layer's SeedSequence; keys use the
    layer's channel scales.  Storage dtype as the workload's."""
    import torch

    N = wl.N if N is None else int(N)
    scales = torch.from_numpy(layer_scales(wl, layer, seed)).to(device)
    ss = np.random.SeedSequence([seed, layer] + [ord(c) for c in wl.name + "/device"])
    gen = torch.Generator(device=device)
    gen.manual_seed(int(ss.generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1)))
    dt = torch.float16 if wl.dtype == "float16" else torch.float32
    keys = (torch.randn((N, wl.D), generator=gen, device=device) * scales[None, :]).to(dt)
    values = torch.randn((N, wl.D), generator=gen, device=device).to(dt)
    w_k = torch.empty(N, device=device).log_normal_(0.0, 1.0, generator=gen)
    w_v = torch.empty(N, device=device).log_normal_(0.0, 1.0, generator=gen)
    return keys, values, w_k, w_v


def gradient_rows(N: int, D: int, seed: int = 0, sigma: float = 1.5,
                  dtype=np.float16) -> np.ndarray:
    """Synthetic per-token gradient rows g_i = s_i z_i with z_i ~ N(0, I_D)
    and a heavy-tailed scale s_i ~ lognormal(0, sigma): stand-ins for the
    gradients of the loss with respect to the KV activations (Sec. 5.3),
    whose norms the paper reports as heavy-tailed (max/median > 400, and
    below 10 after the log smoothing, which with tau = 1 also bounds the raw
    ratio below 2^10 - 1).  sigma = 1.5 gives max/median ~ 700 at 32768
    rows."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, N, D, 77])))
    s = rng.lognormal(0.0, sigma, size=N).astype(np.float32)
    z = rng.standard_normal((N, D), dtype=np.float32)
    return (s[:, None] * z).astype(dtype)


def attn_case(B: int, cap: int, lens, Hkv: int, GQ: int, seed: int = 0, q_dtype="float32",
              q_scale: float = 1.0, hd: int = 128, K: int = 256, d: int = 8):
    """One decoding step over coded caches (1-bit cache: d = 8, K = 256,
    one stage): random codebooks and codes stand in for a calibrated layer's
    (any code is a valid input), queries N(0, q_scale^2).

    Draw order (PCG64 from SeedSequence([seed, B, cap, Hkv, GQ])): key gains
    sqrt(d) * lognormal(0, 0.25) [1, G, K], key shapes (unit rows of
    N(0, I_d)) [1, G, K, d], the same for values, key codes and value codes
    (uniform bytes, packed 4 per uint32 word, subspace g in byte g of a row)
    [B, cap, G / 4], queries [B, Hkv * GQ, hd].  lens gives seq_len."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, B, cap, Hkv, GQ])))
    G = Hkv * hd // d

    def codebook():
        gain = (np.sqrt(d) * rng.lognormal(0.0, 0.25, size=(1, G, K))).astype(np.float32)
        sh = rng.standard_normal((1, G, K, d))
        sh /= np.linalg.norm(sh, axis=-1, keepdims=True)
        return gain, sh.astype(np.float32)

    k_gain, k_shape = codebook()
    v_gain, v_shape = codebook()
    k_codes = rng.integers(0, K, size=(B, cap, G), dtype=np.uint8).view(np.uint32)
    v_codes = rng.integers(0, K, size=(B, cap, G), dtype=np.uint8).view(np.uint32)
    q = (q_scale * rng.standard_normal((B, Hkv * GQ, hd))).astype(q_dtype)
    return dict(k_codes=np.ascontiguousarray(k_codes), v_codes=np.ascontiguousarray(v_codes),
                lens=np.asarray(lens, np.int32), k_gain=k_gain, k_shape=k_shape,
                v_gain=v_gain, v_shape=v_shape, q=q, Hkv=Hkv, GQ=GQ)


def attn_case_rq(B: int, cap: int, lens, Hkv: int, GQ: int, M: int = 12, seed: int = 0,
                 q_dtype="float32", q_scale: float = 1.0, hd: int = 128, K: int = 256,
                 decay: float = 0.75):
    """One decoding step over residual-coded caches at the paper's sub-1-bit
    rates (one subspace per head, d = hd, K = 256, M stages; M = 12 is 0.75
    bit): random codebooks and codes stand in for a calibrated layer's.
    Stage m's gains are sqrt(hd) * decay^m * lognormal(0, 0.25), as the
    energy of a residual cascade falls stage by stage; shapes are unit rows
    of N(0, I_hd).

    Draw order (PCG64 from SeedSequence([seed, B, cap, Hkv, GQ, M, 7])): key
    gains [M, Hkv, K], key shapes [M, Hkv, K, hd], the same for values, key
    codes and value codes (uniform bytes [B, cap, M * Hkv], stage m of head
    h in byte m * Hkv + h of a row, rows padded with zero bytes to whole
    uint32 words), queries [B, Hkv * GQ, hd].  lens gives seq_len."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, B, cap, Hkv, GQ, M,
                                                                      7])))
    scale = (np.sqrt(hd) * decay ** np.arange(M))[:, None, None]

    def codebook():
        gain = (scale * rng.lognormal(0.0, 0.25, size=(M, Hkv, K))).astype(np.float32)
        sh = rng.standard_normal((M, Hkv, K, hd))
        sh /= np.linalg.norm(sh, axis=-1, keepdims=True)
        return gain, sh.astype(np.float32)

    k_gain, k_shape = codebook()
    v_gain, v_shape = codebook()
    W = (M * Hkv * 8 + 31) // 32
    codes = []
    for _ in range(2):
        c = np.zeros((B, cap, 4 * W), dtype=np.uint8)
        c[:, :, :M * Hkv] = rng.integers(0, K, size=(B, cap, M * Hkv), dtype=np.uint8)
        codes.append(np.ascontiguousarray(c).view(np.uint32))
    q = (q_scale * rng.standard_normal((B, Hkv * GQ, hd))).astype(q_dtype)
    return dict(k_codes=codes[0], v_codes=codes[1], lens=np.asarray(lens, np.int32),
                k_gain=k_gain, k_shape=k_shape, v_gain=v_gain, v_shape=v_shape, q=q, Hkv=Hkv,
                GQ=GQ, M=M)


def gaussian_case(N: int, D: int, K: int, seed: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """The random-normal inputs of Sec. 6.1: X [N, D] float32 with i.i.d.
    rows x ~ N(0, I_D), and K distinct seed row indices [K] drawn after X
    from the same stream (one stream per (seed, N, D, K))."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, N, D, K, 61])))
    X = rng.standard_normal((N, D), dtype=np.float32)
    seeds = rng.choice(N, size=K, replace=False).astype(np.int64)
    return X, seeds
