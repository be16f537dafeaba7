"""Seeded synthetic KV-cache inputs and the named workloads.

This module holds no codec arithmetic: it only draws random inputs (shaped like the KV
caches of the models the paper evaluates) and names the workloads.  Both the oracle side
and the GPU side of every test and of the benchmark take their inputs from here.

Recipe (per (tensor s, layer l, batch b, head h) slice, so that any slice can be
regenerated on its own):
  * values:  x ~ N(0, 1) per element;
  * keys:    x = N(0, 1) * c[l, h, channel], with c = exp(sigma * N(0, 1)) drawn once per
             (l, h, channel) and the first k channels of a seeded permutation of the
             channels multiplied by m (outlier channels);
  * bf16 caches round the float32 draws to bfloat16 with round-to-nearest-even;
  * decode-phase queries (attention over the cache): q ~ N(0, 1) per element, one vector per
    (layer, batch row, query head).
Streams are numpy Philox generators keyed through a SeedSequence of
(seed, purpose, s, l, b, h).
"""
from __future__ import annotations

import dataclasses
import os

import numpy as np

TAG_DATA, TAG_SCALE, TAG_NEW, TAG_QUERY = 1, 2, 3, 4


@dataclasses.dataclass(frozen=True)
class KeyDist:
    sigma: float = 0.7      # log-normal spread of the per-channel key scale
    outliers: int = 4       # outlier channels per (layer, head)
    mult: float = 20.0      # outlier channel multiplier


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    L: int
    B: int
    H: int
    T: int
    d: int
    dtype: str               # "bf16" or "f32"
    g: int
    backend: str             # "bu" or "kivi"
    bits: int
    block_c: int = 64
    key_tokens: int = 32
    val_channels: int = 64
    residual: int = 128
    keys: KeyDist = KeyDist()
    gauge: str = "haar"
    data_seed: int = 0xC0DEC0DE
    gauge_seed: int = 0x6A06E

    @property
    def n_elements(self) -> int:
        """N_KV = sum_l 2 B H T d (paper section 3)."""
        return 2 * self.L * self.B * self.H * self.T * self.d


WORKLOADS = {
    # one layer, 2 KV heads, head_dim 64, 256 tokens, fp32, g=16, BU 4-bit block 32
    "tiny": Workload("tiny", L=1, B=1, H=2, T=256, d=64, dtype="f32", g=16, backend="bu", bits=4, block_c=32,
                     keys=KeyDist(0.5, 2, 10.0), data_seed=0xC0DEC0DE + 0, gauge_seed=0x6A06E + 0),
    # Llama-3-8B-shaped KV: 32 layers, 8 KV heads, head_dim 128, batch 1, 8192 tokens, bf16, g=128, BU 4-bit n=64
    "llama8b": Workload("llama8b", L=32, B=1, H=8, T=8192, d=128, dtype="bf16", g=128, backend="bu", bits=4,
                        block_c=64, keys=KeyDist(0.7, 4, 20.0), data_seed=0xC0DEC0DE + 1,
                        gauge_seed=0x6A06E + 1),
    # KIVI-style on the same shape at batch 4, 32768 tokens, 3 bits, g=32
    "kivi": Workload("kivi", L=32, B=4, H=8, T=32768, d=128, dtype="bf16", g=32, backend="kivi", bits=3,
                     keys=KeyDist(0.7, 4, 20.0), data_seed=0xC0DEC0DE + 2, gauge_seed=0x6A06E + 2),
    # rolling decode: batch 32, 32k history, 6-bit BU block 64, g=128
    "rolling": Workload("rolling", L=32, B=32, H=8, T=32768, d=128, dtype="bf16", g=128, backend="bu", bits=6,
                        block_c=64, keys=KeyDist(0.7, 4, 20.0), data_seed=0xC0DEC0DE + 3,
                        gauge_seed=0x6A06E + 3),
    # 27B-shaped KV: 46 layers, 16 KV heads, head_dim 128, batch 2, 16384 tokens (g and bits swept)
    "gemma27b": Workload("gemma27b", L=46, B=2, H=16, T=16384, d=128, dtype="bf16", g=128, backend="bu", bits=4,
                         block_c=64, keys=KeyDist(0.7, 4, 20.0), data_seed=0xC0DEC0DE + 4,
                         gauge_seed=0x6A06E + 4),
}


def _rng(seed: int, tag: int, s: int, l: int, b: int, h: int) -> np.random.Generator:
    return np.random.Generator(np.random.Philox(np.random.SeedSequence([seed, tag, s, l, b, h])))


def key_channel_scale(seed: int, l: int, h: int, d: int, dist: KeyDist) -> np.ndarray:
    rng = _rng(seed, TAG_SCALE, 0, l, 0, h)
    c = np.exp(dist.sigma * rng.standard_normal(d))
    perm = rng.permutation(d)
    c[perm[: dist.outliers]] *= dist.mult
    return c.astype(np.float32)


def kv_slice(seed: int, s: int, l: int, b: int, h: int, T: int, d: int, dist: KeyDist, t_offset: int = 0,
             tag: int = TAG_DATA) -> np.ndarray:
    """float32 [T][d] draws of one slice (s = 0 keys, 1 values).

    Tokens are drawn in fixed chunks of 256 so that token t always receives the same value
    whatever T and t_offset are."""
    out = np.empty((T, d), dtype=np.float32)
    chunk = 256
    first, last = t_offset // chunk, (t_offset + T + chunk - 1) // chunk
    for c in range(first, last):
        rng = np.random.Generator(np.random.Philox(np.random.SeedSequence([seed, tag, s, l, b, h, c])))
        blk = rng.standard_normal((chunk, d), dtype=np.float32)
        lo = max(t_offset, c * chunk)
        hi = min(t_offset + T, (c + 1) * chunk)
        out[lo - t_offset:hi - t_offset] = blk[lo - c * chunk:hi - c * chunk]
    if s == 0:
        out *= key_channel_scale(seed, l, h, d, dist)[None, :]
    return out


def round_bf16_bits(a: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) of float32 data, round to nearest even (torch's cast)."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def kv_tensor(w: Workload, s: int, L: int | None = None, B: int | None = None, H: int | None = None,
              T: int | None = None, l0: int = 0, t_offset: int = 0) -> np.ndarray:
    """Host tensor [L][B][H][T][d] of workload w (uint16 bf16 bits, or float32), optionally a
    sub-range of layers / batch / heads / tokens with the same values as the full tensor."""
    L = w.L if L is None else L
    B = w.B if B is None else B
    H = w.H if H is None else H
    T = w.T if T is None else T
    f = np.empty((L, B, H, T, w.d), dtype=np.float32)

    def fill(idx):
        li, b, h = idx
        f[li, b, h] = kv_slice(w.data_seed, s, l0 + li, b, h, T, w.d, w.keys, t_offset)

    jobs = [(li, b, h) for li in range(L) for b in range(B) for h in range(H)]
    if len(jobs) * T * w.d >= (1 << 22):
        from concurrent.futures import ThreadPoolExecutor

        with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
            list(ex.map(fill, jobs))
    else:
        for j in jobs:
            fill(j)
    if w.dtype == "bf16":
        return round_bf16_bits(f)
    return f


def new_tokens(w: Workload, s: int, step: int, L: int | None = None, B: int | None = None,
               H: int | None = None) -> np.ndarray:
    """The K or V rows [L][B][H][d] a rolling step appends (same distribution as the history)."""
    L = w.L if L is None else L
    B = w.B if B is None else B
    H = w.H if H is None else H
    f = np.empty((L, B, H, w.d), dtype=np.float32)
    for li in range(L):
        for b in range(B):
            for h in range(H):
                f[li, b, h] = kv_slice(w.data_seed, s, li, b, h, 1, w.d, w.keys, t_offset=step, tag=TAG_NEW)[0]
    if w.dtype == "bf16":
        return round_bf16_bits(f)
    return f


def queries(w: Workload, Hq: int, L: int | None = None, B: int | None = None, step: int = 0) -> np.ndarray:
    """Decode-phase queries [L][B][Hq][d] (uint16 bf16 bits, or float32) of rolling step `step`."""
    L = w.L if L is None else L
    B = w.B if B is None else B
    f = np.empty((L, B, Hq, w.d), dtype=np.float32)
    for li in range(L):
        for b in range(B):
            f[li, b] = _rng(w.data_seed, TAG_QUERY, step, li, b, 0).standard_normal((Hq, w.d), dtype=np.float32)
    if w.dtype == "bf16":
        return round_bf16_bits(f)
    return f
