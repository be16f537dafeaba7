"""Python view of the CPU oracle (oracle.c) for the gauge-coded KV-cache codec.

TEST INFRASTRUCTURE ONLY: the test-suite, the smoke check and the CPU-baseline leg of the
benchmark use it; the product library never imports, links or runs it, and this package
imports nothing from the product package.

Every entry mirrors the codec-wrapper equations of the paper's section 3
(Z = G X, B_c = C(Z), Zhat = D(B_c), Xhat = G^T Zhat), the gauge parameterisation of
section 4.1 (G = exp(A - A^T), G^-1 = G^T) and the block-uniform / KIVI-style backends of
section 4.3.  The arithmetic itself lives in oracle.c; this file only marshals numpy arrays
and states the byte layouts the codec writes (a library contract the oracle mirrors).
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import os

import numpy as np

from . import build as _build

PASSTHROUGH, BLOCK_UNIFORM, KIVI, ZFP = 0, 1, 2, 3
GAUGE_IDENTITY, GAUGE_HAAR, GAUGE_DCT2, GAUGE_HADAMARD, GAUGE_EXPM, GAUGE_USER = range(6)
FLAG_NONFINITE, FLAG_SIDE_OVERFLOW = 1, 2

_lib = None


def lib():
    global _lib
    if _lib is None:
        path = _build.LIB
        if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_build.SRC):
            _build.build()
        L = C.CDLL(path)
        vp, i, u64 = C.c_void_p, C.c_int, C.c_uint64
        L.orc_philox4x32_10.argtypes = [vp, vp, vp]
        L.orc_gaussian.argtypes = [u64, u64, u64]
        L.orc_gaussian.restype = C.c_double
        L.orc_f16_round_dir.argtypes = [C.c_double, i]
        L.orc_f16_round_dir.restype = C.c_double
        L.orc_f16_bits.argtypes = [C.c_double]
        L.orc_f16_bits.restype = C.c_uint16
        L.orc_f16_value.argtypes = [C.c_uint16]
        L.orc_f16_value.restype = C.c_double
        L.orc_bf16_to_f32.argtypes = [C.c_uint16]
        L.orc_bf16_to_f32.restype = C.c_float
        L.orc_f32_to_bf16.argtypes = [C.c_float]
        L.orc_f32_to_bf16.restype = C.c_uint16
        L.orc_orthogonality_error.argtypes = [i, vp]
        L.orc_orthogonality_error.restype = C.c_double
        L.orc_gauge_make.argtypes = [i, i, i, i, i, u64, vp, vp]
        L.orc_gauge_apply.argtypes = [i, i, vp, vp, vp]
        L.orc_gauge_inverse.argtypes = [i, i, vp, vp, vp]
        L.orc_quantize_block.argtypes = [vp, i, i, vp, vp, vp]
        L.orc_dequantize_block.argtypes = [vp, i, C.c_uint16, C.c_uint16, vp]
        L.orc_pack_codes.argtypes = [vp, i, i, vp]
        L.orc_unpack_codes.argtypes = [vp, i, i, vp]
        L.orc_kv_encode.argtypes = [i] * 14 + [i, vp, vp, i, vp, vp, vp, i]
        L.orc_kv_decode.argtypes = [i] * 13 + [vp, i, vp, vp, vp, vp, i, i, i, vp]
        L.orc_kv_append.argtypes = [i] * 13 + [i, vp, vp, i, vp, vp, vp, vp]
        L.orc_zfp_order.argtypes = [vp]
        L.orc_zfp_fwd4.argtypes = [vp, i]
        L.orc_zfp_inv4.argtypes = [vp, i]
        L.orc_negabinary.argtypes = [C.c_int32]
        L.orc_negabinary.restype = C.c_uint32
        L.orc_from_negabinary.argtypes = [C.c_uint32]
        L.orc_from_negabinary.restype = C.c_int32
        L.orc_zfp_encode_block.argtypes = [vp, i, vp]
        L.orc_zfp_decode_block.argtypes = [vp, i, vp]
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


# ------------------------------------------------------------------------------------------
# number formats and the counter-based generator
# ------------------------------------------------------------------------------------------

def philox4x32_10(ctr, key):
    c = np.asarray(ctr, dtype=np.uint32).copy()
    k = np.asarray(key, dtype=np.uint32).copy()
    out = np.zeros(4, dtype=np.uint32)
    lib().orc_philox4x32_10(_p(c), _p(k), _p(out))
    return out


def gaussian(seed: int, index: int, k: int) -> float:
    return lib().orc_gaussian(seed, index, k)


def f16_round_dir(v: float, direction: int) -> float:
    return lib().orc_f16_round_dir(float(v), int(direction))


def f16_bits(v: float) -> int:
    return int(lib().orc_f16_bits(float(v)))


def f16_value(bits: int) -> float:
    return lib().orc_f16_value(int(bits))


def bf16_to_f32(bits: int) -> float:
    return lib().orc_bf16_to_f32(int(bits))


def f32_to_bf16(v: float) -> int:
    return int(lib().orc_f32_to_bf16(float(v)))


# ------------------------------------------------------------------------------------------
# gauges (section 3 Table 1; section 4.1; section 4.3 controls)
# ------------------------------------------------------------------------------------------

def gauge_make(kind: int, L: int, H: int, d: int, g: int, seed: int = 0, params=None) -> np.ndarray:
    """Every gauge of a cache as float32 [L][2][H][R][g][g], R = d / g."""
    R = d // g
    G = np.zeros((L, 2, H, R, g, g), dtype=np.float32)
    par = None if params is None else np.ascontiguousarray(params, dtype=np.float32)
    rc = lib().orc_gauge_make(kind, L, H, d, g, seed, _p(par), _p(G))
    if rc != 0:
        raise ValueError(f"orc_gauge_make failed with {rc}")
    return G


def orthogonality_error(Gblock: np.ndarray) -> float:
    Gb = np.ascontiguousarray(Gblock, dtype=np.float32)
    return lib().orc_orthogonality_error(Gb.shape[-1], _p(Gb))


def gauge_apply(Gs: np.ndarray, x: np.ndarray) -> np.ndarray:
    """z = G x for one vector; Gs holds the R gauges [R][g][g] of its (l, s, h)."""
    Gs = np.ascontiguousarray(Gs, dtype=np.float32)
    x = np.ascontiguousarray(x, dtype=np.float32)
    z = np.zeros_like(x)
    lib().orc_gauge_apply(x.shape[0], Gs.shape[-1], _p(Gs), _p(x), _p(z))
    return z


def gauge_inverse(Gs: np.ndarray, z: np.ndarray) -> np.ndarray:
    Gs = np.ascontiguousarray(Gs, dtype=np.float32)
    z = np.ascontiguousarray(z, dtype=np.float32)
    x = np.zeros_like(z)
    lib().orc_gauge_inverse(z.shape[0], Gs.shape[-1], _p(Gs), _p(z), _p(x))
    return x


# ------------------------------------------------------------------------------------------
# quantiser and packing (section 4.3)
# ------------------------------------------------------------------------------------------

def quantize_block(z: np.ndarray, bits: int):
    z = np.ascontiguousarray(z, dtype=np.float32)
    q = np.zeros(z.shape[0], dtype=np.uint8)
    mn = np.zeros(1, dtype=np.uint16)
    sc = np.zeros(1, dtype=np.uint16)
    flags = lib().orc_quantize_block(_p(z), z.shape[0], bits, _p(q), _p(mn), _p(sc))
    return q, int(mn[0]), int(sc[0]), flags


def dequantize_block(q: np.ndarray, mn_bits: int, sc_bits: int) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.uint8)
    out = np.zeros(q.shape[0], dtype=np.float32)
    lib().orc_dequantize_block(_p(q), q.shape[0], mn_bits, sc_bits, _p(out))
    return out


def pack_codes(q: np.ndarray, bits: int) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.uint8)
    out = np.zeros((q.shape[0] * bits + 7) // 8, dtype=np.uint8)
    lib().orc_pack_codes(_p(q), q.shape[0], bits, _p(out))
    return out


def unpack_codes(packed: np.ndarray, n: int, bits: int) -> np.ndarray:
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    q = np.zeros(n, dtype=np.uint8)
    lib().orc_unpack_codes(_p(packed), n, bits, _p(q))
    return q


# ------------------------------------------------------------------------------------------
# zfp-style fixed-rate block codec (the paper's zfp backend, from zfp's published algorithm)
# ------------------------------------------------------------------------------------------

def zfp_order() -> np.ndarray:
    """Sequency order: position k of the coded coefficients holds block entry 4 j + i."""
    out = np.zeros(16, dtype=np.int32)
    lib().orc_zfp_order(_p(out))
    return out


def zfp_fwd4(v) -> np.ndarray:
    a = np.ascontiguousarray(v, dtype=np.int32).copy()
    lib().orc_zfp_fwd4(_p(a), 1)
    return a


def zfp_inv4(v) -> np.ndarray:
    a = np.ascontiguousarray(v, dtype=np.int32).copy()
    lib().orc_zfp_inv4(_p(a), 1)
    return a


def negabinary(i: int) -> int:
    return int(lib().orc_negabinary(int(i)))


def from_negabinary(u: int) -> int:
    return int(lib().orc_from_negabinary(int(u)))


def zfp_encode_block(v, rate: int):
    """v: 16 float32 values, entry 4 j + i = channel i of token j.  Returns (2 rate bytes, flags)."""
    a = np.ascontiguousarray(v, dtype=np.float32)
    out = np.zeros(2 * rate, dtype=np.uint8)
    flags = lib().orc_zfp_encode_block(_p(a), rate, _p(out))
    return out, flags


def zfp_decode_block(code, rate: int) -> np.ndarray:
    c = np.ascontiguousarray(code, dtype=np.uint8)
    out = np.zeros(16, dtype=np.float32)
    lib().orc_zfp_decode_block(_p(c), rate, _p(out))
    return out


# ------------------------------------------------------------------------------------------
# whole-cache codec over the library's byte layouts
# ------------------------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Codec:
    backend: int = BLOCK_UNIFORM
    bits: int = 4
    block_c: int = 64          # block-uniform channel block n
    key_tokens: int = 32       # KIVI key token group
    val_channels: int = 64     # KIVI value channel group
    residual: int = 128        # KIVI full-precision window
    block_t: int = 1           # block-uniform tile tokens Tb (1: one token per block)

    def args(self):
        return [self.backend, self.bits, self.block_c, self.key_tokens, self.val_channels, self.residual,
                self.block_t]


def cache_layout(codec: Codec, s: int, L: int, B: int, H: int, T_cap: int, d: int) -> dict:
    """Shapes and dtypes of the (codes, side, residual) buffers of one K or V cache."""
    b = codec.bits
    if codec.backend == ZFP:
        # one 4 x 4 block (4 tokens x 4 channels) of 16 b bits per 4 tokens and 4 channels
        return {"codes": ((L, B, H, T_cap // 4, d // 4, 2 * b), np.uint8), "side": None, "residual": None}
    if codec.backend == PASSTHROUGH:
        return {"codes": ((L, B, H, T_cap, d), np.float32), "side": None, "residual": None}
    if codec.backend == BLOCK_UNIFORM:
        n, bt = codec.block_c, codec.block_t
        staging = ((L, B, H, bt, d), np.uint16) if bt > 1 else None
        return {"codes": ((L, B, H, T_cap, d * b // 8), np.uint8),
                "side": ((L, B, H, T_cap // bt, d // n, 2), np.uint16), "residual": staging}
    kg, kvc, win = codec.key_tokens, codec.val_channels, codec.residual
    ring = ((L, B, H, win + kg, d), np.uint16)
    if s == 0:
        return {"codes": ((L, B, H, T_cap // kg, d, kg * b // 8), np.uint8),
                "side": ((L, B, H, T_cap // kg, d, 2), np.uint16), "residual": ring}
    return {"codes": ((L, B, H, T_cap, d * b // 8), np.uint8),
            "side": ((L, B, H, T_cap, d // kvc, 2), np.uint16), "residual": ring}


def empty_cache(codec: Codec, s: int, L: int, B: int, H: int, T_cap: int, d: int) -> dict:
    lay = cache_layout(codec, s, L, B, H, T_cap, d)
    return {k: (None if v is None else np.zeros(v[0], dtype=v[1])) for k, v in lay.items()}


def tile_tq(T: int, codec: Codec) -> int:
    """Tokens quantised when a block-uniform cache of Tb-token tiles holds T tokens."""
    return (T // codec.block_t) * codec.block_t


def kivi_tq(T: int, codec: Codec) -> int:
    """Tokens quantised when a KIVI cache holds T tokens."""
    if T < codec.residual:
        return 0
    return ((T - codec.residual) // codec.key_tokens) * codec.key_tokens


def kv_encode(codec: Codec, s: int, X: np.ndarray, G: np.ndarray, T_cap: int, cache: dict | None = None,
              t0: int = 0):
    """Encode X[L][B][H][T][d] (uint16 bf16 bits or float32) at positions [t0, t0+T)."""
    L_, B, H, T, d = X.shape
    g = G.shape[-1]
    x_bf16 = 1 if X.dtype == np.uint16 else 0
    X = np.ascontiguousarray(X)
    Gc = np.ascontiguousarray(G, dtype=np.float32)
    if cache is None:
        cache = empty_cache(codec, s, L_, B, H, T_cap, d)
    flags = lib().orc_kv_encode(*codec.args(), s, L_, B, H, T, d, g, x_bf16, _p(X), _p(Gc), T_cap,
                                _p(cache["codes"]), _p(cache["side"]), _p(cache["residual"]), t0)
    if flags < 0:
        raise ValueError(f"orc_kv_encode rejected its arguments ({flags})")
    return cache, flags


def kv_decode(codec: Codec, s: int, G: np.ndarray, cache: dict, t0: int, Tout: int, lens=None,
              out_bf16: bool = True) -> np.ndarray:
    """Decode tokens [t0, t0+Tout) into Xhat[L][B][H][Tout][d] (uint16 bf16 bits or float32)."""
    L_, B, H = cache["codes"].shape[:3]
    d = G.shape[-3] * G.shape[-1]
    g = G.shape[-1]
    if codec.backend == KIVI and s == 0:
        T_cap = cache["codes"].shape[3] * codec.key_tokens
    elif codec.backend == ZFP:
        T_cap = cache["codes"].shape[3] * 4
    else:
        T_cap = cache["codes"].shape[3]
    Gc = np.ascontiguousarray(G, dtype=np.float32)
    out = np.zeros((L_, B, H, Tout, d), dtype=np.uint16 if out_bf16 else np.float32)
    ln = None if lens is None else np.ascontiguousarray(lens, dtype=np.int32)
    rc = lib().orc_kv_decode(*codec.args(), s, L_, B, H, d, g, _p(Gc), T_cap, _p(cache["codes"]),
                             _p(cache["side"]), _p(cache["residual"]), _p(ln), t0, Tout, 1 if out_bf16 else 0,
                             _p(out))
    if rc < 0:
        raise ValueError(f"orc_kv_decode rejected its arguments ({rc})")
    return out


def kv_append(codec: Codec, s: int, Xnew: np.ndarray, G: np.ndarray, cache: dict, pos) -> int:
    """Rolling append of Xnew[L][B][H][d] at pos[b]; returns the flags."""
    L_, B, H, d = Xnew.shape
    g = G.shape[-1]
    x_bf16 = 1 if Xnew.dtype == np.uint16 else 0
    if codec.backend == KIVI and s == 0:
        T_cap = cache["codes"].shape[3] * codec.key_tokens
    else:
        T_cap = cache["codes"].shape[3]
    Xn = np.ascontiguousarray(Xnew)
    Gc = np.ascontiguousarray(G, dtype=np.float32)
    ps = np.ascontiguousarray(pos, dtype=np.int32)
    flags = lib().orc_kv_append(*codec.args(), s, L_, B, H, d, g, x_bf16, _p(Xn), _p(Gc), T_cap,
                                _p(cache["codes"]), _p(cache["side"]), _p(cache["residual"]), _p(ps))
    if flags < 0:
        raise ValueError(f"orc_kv_append rejected its arguments ({flags})")
    return flags


# ------------------------------------------------------------------------------------------
# cache metrics (section 4.4 and the metric-definition table of the appendix)
# ------------------------------------------------------------------------------------------

def nrmse(ref: np.ndarray, got: np.ndarray) -> float:
    """sqrt(sum SSE / sum reference SSE) over all elements, in binary64."""
    r = np.asarray(ref, dtype=np.float64)
    e = np.asarray(got, dtype=np.float64) - r
    return float(np.sqrt(np.sum(e * e) / np.sum(r * r)))


def live_bytes(codec: Codec, s: int, T: int, d: int) -> int:
    """Bytes one (l, b, h) slice of a K or V cache holding T tokens occupies: codes, side info
    and the full-precision window (the gauge itself is a per-checkpoint object, not counted)."""
    b = codec.bits
    if codec.backend == PASSTHROUGH:
        return T * d * 4
    if codec.backend == BLOCK_UNIFORM:
        tq = tile_tq(T, codec)
        return tq * d * b // 8 + (tq // codec.block_t) * (d // codec.block_c) * 4 + (T - tq) * d * 2
    tq = kivi_tq(T, codec)
    win = (T - tq) * d * 2
    if s == 0:
        return tq * d * b // 8 + (tq // codec.key_tokens) * d * 4 + win
    return tq * (d * b // 8 + (d // codec.val_channels) * 4) + win


def bits_per_value(codec: Codec, T: int, d: int) -> float:
    """Measured bits per represented K/V value for one (l, b, h) slice pair."""
    tot = live_bytes(codec, 0, T, d) + live_bytes(codec, 1, T, d)
    return 8.0 * tot / (2.0 * T * d)


# ------------------------------------------------------------------------------------------
# codec-facing spectral statistics (section 4.2, gauge training objective)
# ------------------------------------------------------------------------------------------

def dct2_matrix(N: int) -> np.ndarray:
    """Orthonormal DCT-II as a matrix, row k the k-th frequency (binary64):
    C[k][n] = sqrt((1 if k == 0 else 2) / N) cos(pi (2n + 1) k / (2N))."""
    k = np.arange(N, dtype=np.float64)[:, None]
    n = np.arange(N, dtype=np.float64)[None, :]
    C = np.cos(np.pi * (2.0 * n + 1.0) * k / (2.0 * N)) * np.sqrt(2.0 / N)
    C[0, :] = np.sqrt(1.0 / N)
    return C


def spectral_radius(Tb: int, d: int) -> np.ndarray:
    """rho(u, v) = sqrt((u / (Tb - 1))^2 + (v / (d - 1))^2) / sqrt(2), the normalised radius of
    coefficient (u, v) of a Tb x d token-channel block (section 4.2)."""
    u = np.arange(Tb, dtype=np.float64)[:, None] / (Tb - 1)
    v = np.arange(d, dtype=np.float64)[None, :] / (d - 1)
    return np.sqrt(u * u + v * v) / np.sqrt(2.0)


def spectral_stats(X: np.ndarray, G: np.ndarray, s: int, Tb: int = 16, tau: float = 0.04, eps: float = 1e-12):
    """Spectral statistics of the gauge-transformed cache X' = G X of type s (section 4.2), per
    layer, in binary64.  The token axis is cut into blocks of Tb tokens (tokens past the last
    whole block are ignored); each Tb x d block of X' goes through the orthonormal 2-D DCT-II,
    U = C_Tb Z C_d^T.  With E = U^2 summed over the layer's blocks (every batch row, head and
    token block), returns (stats [L][4], energy [L][Tb][d]) where
        stats[l] = (L_freq, L_rate, 1 - L_freq, sum E),
        L_freq = sum E rho / (sum E + eps),
        L_rate = mean over the layer's coefficients of log(1 + |U| / tau)."""
    L_, B, H, T, d = X.shape
    R, g = G.shape[-3], G.shape[-1]
    if X.dtype == np.uint16:
        x = (X.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    else:
        x = X.astype(np.float64)
    nblk = T // Tb
    Ct, Cd = dct2_matrix(Tb), dct2_matrix(d)
    rho = spectral_radius(Tb, d)
    stats = np.zeros((L_, 4))
    energy = np.zeros((L_, Tb, d))
    for l in range(L_):
        lsum, count = 0.0, 0
        for h in range(H):
            Gd = np.zeros((d, d))
            for r in range(R):
                Gd[r * g:(r + 1) * g, r * g:(r + 1) * g] = G[l, s, h, r].astype(np.float64)
            for b in range(B):
                Z = x[l, b, h, :nblk * Tb] @ Gd.T                     # z_t = G x_t, [T][d]
                for k in range(nblk):
                    U = Ct @ Z[k * Tb:(k + 1) * Tb] @ Cd.T
                    energy[l] += U * U
                    lsum += float(np.log1p(np.abs(U) / tau).sum())
                    count += U.size
        tot = float(energy[l].sum())
        lf = float((energy[l] * rho).sum()) / (tot + eps)
        stats[l] = (lf, lsum / max(count, 1), 1.0 - lf, tot)
    return stats, energy


# ------------------------------------------------------------------------------------------
# gradient of the training objective with respect to the gauge parameters (sections 4.1-4.2)
# ------------------------------------------------------------------------------------------

def expm64(W: np.ndarray) -> np.ndarray:
    """exp(W) of a square matrix in binary64 from the power series exp(W) = sum_k W^k / k!:
    W is halved s times until its 1-norm is at most 1/2, the series of W / 2^s is summed until a
    term no longer changes the sum, and the sum is squared s times."""
    W = np.asarray(W, dtype=np.float64)
    n1 = float(np.abs(W).sum(axis=0).max()) if W.size else 0.0
    s = 0
    while n1 > 0.5:
        n1 *= 0.5
        s += 1
    Ws = W / 2.0 ** s
    term = np.eye(W.shape[0])
    total = term.copy()
    for k in range(1, 80):
        term = term @ Ws / k
        nxt = total + term
        if np.array_equal(nxt, total):
            break
        total = nxt
    for _ in range(s):
        total = total @ total
    return total


def expm_frechet64(M: np.ndarray, E: np.ndarray) -> np.ndarray:
    """Frechet derivative of the matrix exponential at M in the direction E,
    L(M, E) = d/dh exp(M + h E) at h = 0: the top-right block of exp([[M, E], [0, M]])."""
    n = M.shape[0]
    W = np.zeros((2 * n, 2 * n))
    W[:n, :n] = M
    W[:n, n:] = E
    W[n:, n:] = M
    return expm64(W)[:n, n:]


def gauge_from_params(A: np.ndarray) -> np.ndarray:
    """G = exp(A - A^T) per block (section 4.1) in binary64: A [..][g][g] -> G [..][g][g]."""
    A = np.asarray(A, dtype=np.float64)
    G = np.zeros_like(A)
    for idx in np.ndindex(*A.shape[:-2]):
        G[idx] = expm64(A[idx] - A[idx].T)
    return G


def spectral_train_loss(X: np.ndarray, A: np.ndarray, s: int, Tb: int = 16, tau: float = 0.04,
                        lam_f: float = 1.0, lam_r: float = 0.02, eps: float = 1e-12) -> np.ndarray:
    """L_train = lam_f L_freq + lam_r L_rate per layer (section 4.2) of X' = G X with
    G = exp(A - A^T) (section 4.1) taken in binary64 from the generators A [L][2][H][R][g][g]."""
    stats, _ = spectral_stats(X, gauge_from_params(A), s, Tb, tau, eps)
    return lam_f * stats[:, 0] + lam_r * stats[:, 1]


def spectral_train_grad(X: np.ndarray, A: np.ndarray, s: int, Tb: int = 16, tau: float = 0.04,
                        lam_f: float = 1.0, lam_r: float = 0.02, eps: float = 1e-12) -> np.ndarray:
    """dL_train(l) / dA[l][s][h][r] as [L][H][R][g][g] (binary64), by the chain rule through the
    objective of section 4.2 and the parameterisation of section 4.1, per layer l:
      1. U = C_Tb Z C_d^T per block with Z = x G^T (the block's rows z_t = G x_t), and per layer
         D = sum E + eps, L_freq = sum E rho / D, N = the layer's coefficient count;
      2. dL/dU = lam_f 2 U (rho - L_freq) / D + lam_r sign(U) / (N (tau + |U|));
      3. dL/dZ = C_Tb^T (dL/dU) C_d (both DCTs orthonormal);
      4. dL/dG = sum over blocks of (dL/dZ)^T x, restricted to the gauge's diagonal blocks;
      5. with S = A - A^T and G = exp(S): dL/dS = L(S^T, dL/dG), the adjoint of the Frechet
         derivative of exp at S (for the trace inner product, <Y, L(S, E)> = <L(S^T, Y), E>);
      6. dL/dA = dL/dS - (dL/dS)^T.
    The -L_freq part of step 2 multiplies the gradient of the total energy sum E, which G and
    the DCTs leave unchanged, so it contributes nothing for an exactly orthogonal G; it is kept
    as the literal derivative of the quotient."""
    L_, B, H, T, d = X.shape
    R, g = A.shape[3], A.shape[-1]
    Aa = np.asarray(A, dtype=np.float64)
    G = gauge_from_params(Aa)
    stats, energy = spectral_stats(X, G, s, Tb, tau, eps)
    if X.dtype == np.uint16:
        x = (X.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    else:
        x = X.astype(np.float64)
    nblk = T // Tb
    Ct, Cd = dct2_matrix(Tb), dct2_matrix(d)
    rho = spectral_radius(Tb, d)
    grad = np.zeros((L_, H, R, g, g))
    for l in range(L_):
        D = float(energy[l].sum()) + eps
        lf = float(stats[l, 0])
        count = B * H * nblk * Tb * d
        for h in range(H):
            Gd = np.zeros((d, d))
            for r in range(R):
                Gd[r * g:(r + 1) * g, r * g:(r + 1) * g] = G[l, s, h, r]
            dGd = np.zeros((d, d))
            for b in range(B):
                for k in range(nblk):
                    xb = x[l, b, h, k * Tb:(k + 1) * Tb]
                    U = Ct @ (xb @ Gd.T) @ Cd.T
                    dU = lam_f * 2.0 * U * (rho - lf) / D + lam_r * np.sign(U) / (count * (tau + np.abs(U)))
                    dZ = Ct.T @ dU @ Cd
                    dGd += dZ.T @ xb
            for r in range(R):
                S = Aa[l, s, h, r] - Aa[l, s, h, r].T
                dS = expm_frechet64(S.T, dGd[r * g:(r + 1) * g, r * g:(r + 1) * g])
                grad[l, h, r] = dS - dS.T
    return grad


# ------------------------------------------------------------------------------------------
# decode-phase attention over a compressed cache (the consumer of the decoded history)
# ------------------------------------------------------------------------------------------

def attend(codec: Codec, G: np.ndarray, kcache: dict, vcache: dict, q: np.ndarray, lens, scale: float) -> np.ndarray:
    """Single-query attention of every query head over the decoded K / V caches, binary64:
    q [L][B][Hq][d] (Hq a multiple of the H cached heads, query head j reading KV head
    j // (Hq / H)); batch row b attends to positions [0, lens[b]).  The caches decode with
    kv_decode (binary32 X_hat = G^T Z_hat), then o = softmax(scale q K_hat^T) V_hat.  A row
    with no positions (lens[b] = 0) has an empty softmax; its output is taken as zero."""
    if not np.issubdtype(q.dtype, np.floating):
        raise TypeError("attend takes query values (a floating-point array), not bf16 bit patterns")
    L_, B, Hq, d = q.shape
    H = kcache["codes"].shape[2]
    grp = Hq // H
    Tmax = int(max(lens))
    if Tmax == 0:
        return np.zeros((L_, B, Hq, d))
    Kh = kv_decode(codec, 0, G, kcache, 0, Tmax, lens=lens, out_bf16=False).astype(np.float64)
    Vh = kv_decode(codec, 1, G, vcache, 0, Tmax, lens=lens, out_bf16=False).astype(np.float64)
    out = np.zeros((L_, B, Hq, d))
    for l in range(L_):
        for b in range(B):
            n = int(lens[b])
            if n == 0:
                continue
            for j in range(Hq):
                h = j // grp
                s = scale * (Kh[l, b, h, :n] @ q[l, b, j].astype(np.float64))
                p = np.exp(s - s.max())
                out[l, b, j] = (p / p.sum()) @ Vh[l, b, h, :n]
    return out
