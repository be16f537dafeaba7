"""Helpers of the GPU parity tests: moving caches between the oracle's numpy layout and the
library's device buffers, unpacking codes, and the comparison criteria.

Criteria (all against the CPU oracle on the same seeded inputs):
  * gauge stage (passthrough backend): per group ||dz||_2 <= 1e-5 ||x||_2;
  * quantise-only (identity gauge on binary32 input, so z = x exactly): codes, side
    information and packed bytes bit-exact;
  * fused encoder: side-info values within one binary16 ulp; at most 1e-4 of the codes
    differ, each by exactly one step, and only where the oracle's z quantised with the GPU's
    side information lies within 1e-3 of a rounding tie;
  * decoder fed the oracle's cache: binary32 out per group ||dx||_2 <= 1e-5 ||x||_2, bf16 out
    within one bf16 ulp of the oracle's binary32 value plus 1e-5 of the group norm (the
    binary32 gauge tolerance, which dominates for elements tiny against their group).
"""
from __future__ import annotations

import numpy as np
import torch

import oracle as O
from paper_2607_20538_amd import codec as cg

GAUGE_TOL = 1e-5
CODE_FRAC = 1e-4
TIE_EPS = 1e-3


def bf16_dev(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def x_dev(X: np.ndarray) -> torch.Tensor:
    return bf16_dev(X) if X.dtype == np.uint16 else torch.from_numpy(np.ascontiguousarray(X)).cuda()


def x_f64(X: np.ndarray) -> np.ndarray:
    if X.dtype == np.uint16:
        return (X.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return X.astype(np.float64)


def out_host(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def to_cg(oc: O.Codec) -> cg.Codec:
    return cg.Codec(oc.backend, oc.bits, oc.block_c, oc.key_tokens, oc.val_channels, oc.residual, oc.block_t)


def cache_to_host(dev: cg.Cache, oc: O.Codec, s: int) -> dict:
    lay = O.cache_layout(oc, s, dev.L, dev.B, dev.H, dev.T_cap, dev.d)
    out = {}
    for key, buf in (("codes", dev.codes), ("side", dev.side), ("residual", dev.residual)):
        if lay[key] is None:
            out[key] = None
            continue
        shp, dt = lay[key]
        nbytes = int(np.prod(shp)) * np.dtype(dt).itemsize
        out[key] = buf[:nbytes].cpu().numpy().view(dt).reshape(shp)
    return out


def cache_to_dev(host: dict, oc: O.Codec, s: int, L: int, B: int, H: int, T_cap: int, d: int, len_: int = 0):
    dev = cg.Cache(to_cg(oc), s, L, B, H, T_cap, d)
    for key in ("codes", "side", "residual"):
        if host.get(key) is not None:
            raw = torch.from_numpy(np.ascontiguousarray(host[key]).view(np.uint8).reshape(-1))
            getattr(dev, key)[: raw.numel()].copy_(raw.cuda())
    dev.len = len_
    return dev


def unpack_rows(codes: np.ndarray, count: int, bits: int) -> np.ndarray:
    """LSB-first streams [..., count*bits/8] -> codes [..., count] (numpy's bit unpacking)."""
    bitsarr = np.unpackbits(codes, axis=-1, bitorder="little").reshape(*codes.shape[:-1], count, bits)
    return (bitsarr.astype(np.uint32) << np.arange(bits, dtype=np.uint32)).sum(axis=-1)


def token_codes(cache: dict, oc: O.Codec, s: int, d: int) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Per-element codes [L][B][H][T][d] with the (min, scale) bits of their block."""
    b = oc.bits
    if oc.backend == O.KIVI and s == 0:
        q = unpack_rows(cache["codes"], oc.key_tokens, b)           # [L,B,H,G,d,kg]
        q = np.moveaxis(q, -1, -2)                                  # [L,B,H,G,kg,d]
        q = q.reshape(*q.shape[:3], -1, d)
        side = np.repeat(cache["side"], oc.key_tokens, axis=3)      # [L,B,H,G*kg,d,2]
        return q, side[..., 0], side[..., 1]
    n = oc.block_c if oc.backend == O.BLOCK_UNIFORM else oc.val_channels
    q = unpack_rows(cache["codes"], d, b)
    side = np.repeat(cache["side"], n, axis=-2)
    if oc.backend == O.BLOCK_UNIFORM and oc.block_t > 1:               # one side row per tile
        side = np.repeat(side, oc.block_t, axis=3)
    return q, side[..., 0], side[..., 1]


def f16(bits: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(bits).astype(np.uint16).view(np.float16).astype(np.float32)


def block_max(z: np.ndarray, oc: O.Codec, s: int, d: int) -> np.ndarray:
    """Per element, the maximum of z over the element's quantisation block ([..., T, d], T a
    whole number of blocks along tokens)."""
    z = z.astype(np.float32)
    if oc.backend == O.KIVI and s == 0:
        kg = oc.key_tokens
        m = z.reshape(*z.shape[:-2], -1, kg, d).max(axis=-2, keepdims=True)
        return np.broadcast_to(m, m.shape[:-2] + (kg, d)).reshape(z.shape)
    n = oc.block_c if oc.backend == O.BLOCK_UNIFORM else oc.val_channels
    bt = oc.block_t if oc.backend == O.BLOCK_UNIFORM else 1
    m = z.reshape(*z.shape[:-2], -1, bt, d // n, n).max(axis=(-3, -1), keepdims=True)
    return np.broadcast_to(m, m.shape[:-3] + (bt, d // n, n)).reshape(z.shape)


def f16_up_bits(v: np.ndarray) -> np.ndarray:
    """binary16 bits of binary32 v rounded toward +inf (-0 returned as +0)."""
    v = np.asarray(v, dtype=np.float32)
    h = v.astype(np.float16)
    up = h.astype(np.float32) < v
    h = np.where(up, np.nextafter(h, np.float16(np.inf)), h)
    bits = h.view(np.uint16)
    return np.where(bits == 0x8000, np.uint16(0), bits)


def check_fused_codes(gpu: dict, orc: dict, z_orc: np.ndarray, oc: O.Codec, s: int, d: int, T: int) -> dict:
    qg, mng, scg = token_codes(gpu, oc, s, d)
    qo, mno, sco = token_codes(orc, oc, s, d)
    qg, mng, scg, qo, mno, sco = (a[:, :, :, :T] for a in (qg, mng, scg, qo, mno, sco))
    qmax = (1 << oc.bits) - 1
    side_diff = (mng != mno) | (scg != sco)
    if side_diff.any():
        # the minimum rounds toward -inf from the block's z, so a z within the gauge tolerance moves
        # it by at most one binary16 ulp; the scale is rounded up from (max - mn_h) / (2^b - 1) with
        # the block's own rounded minimum, so it is checked against that formula evaluated with the
        # GPU's minimum (a one-ulp move of a minimum far from zero shifts the scale by more than an
        # ulp of the scale), within the one ulp the maximum's gauge error can move it
        dmn = np.abs(mng[side_diff].astype(np.int32) - mno[side_diff].astype(np.int32))
        assert dmn.max() <= 1, "block minimum differs by more than one binary16 ulp"
        mx = block_max(z_orc[:, :, :, :T], oc, s, d)[side_diff]
        rng = (mx - f16(mng[side_diff])).astype(np.float32)
        sc_from_mn = f16_up_bits((rng / np.float32(qmax)).astype(np.float32)).astype(np.int32)
        g_sc = scg[side_diff].astype(np.int32)
        ok = (np.abs(g_sc - sco[side_diff].astype(np.int32)) <= 1) | (np.abs(g_sc - sc_from_mn) <= 1)
        assert ok.all(), "block scale differs from the oracle's by more than its minimum explains"
    diff = qg != qo
    frac = float(diff.mean())
    assert frac <= CODE_FRAC, f"{frac:.2e} of codes differ"
    if diff.any():
        assert np.abs(qg[diff].astype(np.int64) - qo[diff]).max() == 1
        mn, sc = f16(mng[diff]), f16(scg[diff])
        inv = np.where(sc == 0, np.float32(0), np.float32(1) / np.where(sc == 0, np.float32(1), sc))
        t = ((z_orc[:, :, :, :T][diff].astype(np.float32) - mn) * inv).astype(np.float32)
        same = np.clip(np.rint(t), 0, qmax) == qg[diff]
        near_tie = np.abs(np.abs(t - np.floor(t)) - 0.5) <= TIE_EPS
        assert np.all(same | near_tie), "a differing code is not at a rounding tie"
    return {"code_frac": frac, "side_blocks": int(side_diff.sum())}


def group_rel_err(ref: np.ndarray, got: np.ndarray, g: int) -> float:
    if ref.size == 0:
        return 0.0
    r = ref.reshape(*ref.shape[:-1], -1, g).astype(np.float64)
    e = got.reshape(*got.shape[:-1], -1, g).astype(np.float64) - r
    num = np.sqrt((e * e).sum(-1))
    den = np.sqrt((r * r).sum(-1))
    return float((num / np.maximum(den, 1e-30)).max())


def check_bf16_within_ulp(ref_f32: np.ndarray, got_bits: np.ndarray, g: int):
    """bf16 output within one bf16 ulp of the oracle's binary32 value, widened by the binary32
    gauge tolerance (1e-5 of the group norm) for elements small against their group."""
    if ref_f32.size == 0:
        return
    got = (got_bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    ref = ref_f32.astype(np.float64)
    a = np.abs(ref_f32).astype(np.float32)
    e = np.floor(np.log2(np.maximum(a, np.float32(1e-38))))
    ulp = np.exp2(e - 7)
    r = ref.reshape(*ref.shape[:-1], -1, g)
    gnorm = np.repeat(np.sqrt((r * r).sum(-1)), g, axis=-1).reshape(ref.shape)
    tol = ulp * (1 + 1e-6) + GAUGE_TOL * gnorm + 1e-38
    bad = np.abs(got - ref) > tol
    assert not bad.any(), (int(bad.sum()), float(np.abs(got - ref)[bad].max()))


def cache_slice(dev: cg.Cache, oc: O.Codec, s: int, l: int, b: int, h: int) -> dict:
    """Slice (l, b, h) of a device cache as a one-slice ([1][1][1]...) cache in the oracle's layout
    (every buffer is [L][B][H][...] with contiguous slices)."""
    lay = O.cache_layout(oc, s, dev.L, dev.B, dev.H, dev.T_cap, dev.d)
    idx = (l * dev.B + b) * dev.H + h
    out = {}
    for key in ("codes", "side", "residual"):
        if lay[key] is None:
            out[key] = None
            continue
        shp, dt = lay[key]
        per = int(np.prod(shp[3:])) * np.dtype(dt).itemsize
        raw = getattr(dev, key)[idx * per:(idx + 1) * per].cpu().numpy()
        out[key] = np.ascontiguousarray(raw.view(dt).reshape((1, 1, 1) + tuple(shp[3:])))
    return out


def bf16_slice_host(x: np.ndarray) -> np.ndarray:
    """float32 draws -> bf16 bit patterns (round to nearest even), as synth does."""
    from paper_2607_20538_amd import synth

    return synth.round_bf16_bits(x)
