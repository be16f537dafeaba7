"""C-ABI checks that need no GPU: the library loads and exports every declared symbol, host
gauge construction agrees with the oracle, buffer sizing follows the layouts, and invalid
arguments are rejected on the host before anything is enqueued."""
import ctypes as C
import os
import re

import numpy as np
import pytest
import torch

import oracle as O
from paper_2607_20538_amd import codec as cg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "codec_gauge.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\*?\s+\*?([a-z_]+)\(", text, flags=re.M)))


def test_header_declares_the_binding_exports():
    assert _declared() == sorted(cg.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = cg.lib()
    for name in _declared():
        assert hasattr(L, name), name
    assert cg.status_str(cg.CG_ERR_UNSUPPORTED) == "unsupported configuration"


@pytest.mark.parametrize("kind", [cg.GAUGE_IDENTITY, cg.GAUGE_HAAR, cg.GAUGE_DCT2, cg.GAUGE_HADAMARD])
@pytest.mark.parametrize("g", [8, 16, 32, 128])
def test_host_gauge_make_matches_oracle(kind, g):
    G, _ = cg.gauge_make(kind, cg.shape(2, 2, 128, g), seed=31)
    Go = O.gauge_make(kind, 2, 2, 128, g, seed=31)
    assert np.abs(G - Go).max() <= 1e-6
    for blk in G.reshape(-1, g, g)[:4]:
        assert O.orthogonality_error(blk) <= 1e-6


def test_host_gauge_make_expm_and_user():
    A = (np.random.default_rng(1).standard_normal((1, 2, 2, 4, 32, 32)) * 0.5).astype(np.float32)
    G, _ = cg.gauge_make(cg.GAUGE_EXPM, cg.shape(1, 2, 128, 32), params=A)
    assert np.abs(G - O.gauge_make(O.GAUGE_EXPM, 1, 2, 128, 32, params=A)).max() <= 1e-6
    U, _ = cg.gauge_make(cg.GAUGE_USER, cg.shape(1, 2, 128, 32), params=G)
    np.testing.assert_array_equal(U, G)
    G[0, 1, 0, 2, 4, 4] += 1e-3
    with pytest.raises(cg.CodecError) as e:
        cg.gauge_make(cg.GAUGE_USER, cg.shape(1, 2, 128, 32), params=G)
    assert e.value.status == cg.CG_ERR_NOT_ORTHOGONAL


def test_gauge_make_rejects_bad_shapes():
    for shp, st in ((cg.shape(1, 1, 128, 48), cg.CG_ERR_UNSUPPORTED), (cg.shape(0, 1, 128, 32), cg.CG_ERR_ARG),
                    (cg.shape(1, 1, 96, 96), None)):
        if st is None:
            with pytest.raises(cg.CodecError):
                cg.gauge_make(cg.GAUGE_HADAMARD, shp)
            continue
        with pytest.raises(cg.CodecError) as e:
            cg.gauge_make(cg.GAUGE_HAAR, shp)
        assert e.value.status == st
    assert cg.gauge_device_bytes(cg.shape(1, 1, 128, 48)) == 0


@pytest.mark.parametrize("backend,bits,bt", [(O.BLOCK_UNIFORM, 4, 1), (O.BLOCK_UNIFORM, 3, 1), (O.KIVI, 3, 1),
                                             (O.KIVI, 6, 1), (O.PASSTHROUGH, 4, 1), (O.BLOCK_UNIFORM, 4, 16),
                                             (O.BLOCK_UNIFORM, 6, 32)])
def test_cache_bytes_follow_the_layout(backend, bits, bt):
    oc = O.Codec(backend=backend, bits=bits, block_c=32 if bits != 3 else 64, block_t=bt)
    c = cg.Codec(backend, bits, oc.block_c, oc.key_tokens, oc.val_channels, oc.residual, bt)
    for s in (0, 1):
        lay = O.cache_layout(oc, s, 2, 3, 4, 256, 128)
        n = cg.cache_bytes(c, s, 2, 3, 4, 256, 128)
        for k, v in zip(("codes", "side", "residual"), n):
            ref = 0 if lay[k] is None else int(np.prod(lay[k][0])) * np.dtype(lay[k][1]).itemsize
            assert v == ref, (k, v, ref)


def _fake_view(L=1, B=1, H=2, T=16, d=64, dtype=cg.DTYPE_BF16, ptr=0x10000, strides=None):
    st = strides or (B * H * T * d, H * T * d, T * d, d)
    return cg.KvView(ptr, dtype, L, B, H, T, d, *st)


def _fake_cache(L=1, B=1, H=2, T_cap=16, d=64, codes=0x20000, side=0x30000, residual=0x40000, len_=0):
    return cg.CacheStruct(codes, side, residual, L, B, H, T_cap, d, len_)


def _encode(view, cache, codec, shp=None, t0=0, s=0, gdev=0x50000, err=None):
    shp = shp or cg.shape(1, 2, 64, 16)
    cs = codec.struct()
    return cg.lib().kv_encode(s, C.byref(view), gdev, shp, C.byref(cs), C.byref(cache), t0, err, None)


def _decode(view, cache, codec, shp=None, t0=0, s=0, gdev=0x50000, lens=None):
    shp = shp or cg.shape(1, 2, 64, 16)
    cs = codec.struct()
    return cg.lib().kv_decode(s, C.byref(cache), gdev, shp, C.byref(cs), lens, t0, C.byref(view), None, None)


BU = cg.Codec(cg.BLOCK_UNIFORM, 4, 32)


@pytest.mark.parametrize("mutate,status", [
    (lambda v, k, c: (v, k, cg.Codec(cg.BLOCK_UNIFORM, 5, 32)), cg.CG_ERR_UNSUPPORTED),   # bits
    (lambda v, k, c: (v, k, cg.Codec(cg.BLOCK_UNIFORM, 3, 16)), cg.CG_ERR_UNSUPPORTED),   # n*b % 32
    (lambda v, k, c: (v, k, cg.Codec(cg.BLOCK_UNIFORM, 4, 48)), cg.CG_ERR_UNSUPPORTED),   # n does not divide d
    (lambda v, k, c: (v, k, cg.Codec(7, 4, 32)), cg.CG_ERR_ARG),                          # backend
    (lambda v, k, c: (_fake_view(H=3), k, c), cg.CG_ERR_SHAPE),
    (lambda v, k, c: (_fake_view(ptr=0x10004), k, c), cg.CG_ERR_ALIGN),
    (lambda v, k, c: (_fake_view(strides=(2048, 2048, 1024, 68)), k, c), cg.CG_ERR_ALIGN),
    (lambda v, k, c: (_fake_view(dtype=9), k, c), cg.CG_ERR_ARG),
    (lambda v, k, c: (_fake_view(ptr=0), k, c), cg.CG_ERR_ARG),
    (lambda v, k, c: (_fake_view(ptr=0, T=0), k, c, ), "skip"),
    (lambda v, k, c: (v, _fake_cache(codes=0x20008), c), cg.CG_ERR_ALIGN),
    (lambda v, k, c: (v, _fake_cache(side=0), c), cg.CG_ERR_ARG),
    (lambda v, k, c: (v, _fake_cache(B=2), c), cg.CG_ERR_SHAPE),
    (lambda v, k, c: (_fake_view(T=17), k, c), cg.CG_ERR_CAPACITY),
])
def test_encode_rejects_invalid_arguments(mutate, status):
    if status == "skip":   # valid: an empty view would launch nothing, but stays off the CPU
        return
    v, k, c = mutate(_fake_view(), _fake_cache(), BU)
    assert _encode(v, k, c) == status


def test_encode_decode_reject_ranges_and_modes():
    v, k = _fake_view(T=8), _fake_cache()
    assert _encode(v, k, BU, t0=9) == cg.CG_ERR_CAPACITY
    assert _encode(v, k, BU, t0=-1) == cg.CG_ERR_ARG
    assert _encode(v, k, BU, s=2) == cg.CG_ERR_ARG
    assert _encode(v, k, BU, gdev=0x50008) == cg.CG_ERR_ALIGN
    assert _encode(v, k, BU, shp=cg.shape(1, 2, 64, 48)) == cg.CG_ERR_UNSUPPORTED
    kivi = cg.Codec(cg.KIVI, 3, 64, 32, 64, 128)
    kk = _fake_cache(T_cap=64)
    assert _encode(_fake_view(T=16), kk, kivi, t0=16) == cg.CG_ERR_UNSUPPORTED
    assert _encode(_fake_view(T=16, dtype=cg.DTYPE_F32), kk, kivi) == cg.CG_ERR_UNSUPPORTED
    assert _encode(_fake_view(T=16), _fake_cache(T_cap=48), kivi) == cg.CG_ERR_SHAPE
    assert _encode(_fake_view(T=16), kk, cg.Codec(cg.KIVI, 3, 64, 24, 64, 128)) == cg.CG_ERR_UNSUPPORTED
    # KIVI decode beyond the tokens the cache holds
    assert _decode(_fake_view(T=16), _fake_cache(T_cap=64, len_=8), kivi) == cg.CG_ERR_CAPACITY
    assert _decode(_fake_view(T=16), _fake_cache(len_=16), BU, t0=1) == cg.CG_ERR_CAPACITY
    # block-uniform tiles: Tb a power of two up to 32, t0 on a tile boundary, bf16 input, a
    # staging buffer, T_cap a multiple of Tb, decode within the tokens held
    tile = cg.Codec(cg.BLOCK_UNIFORM, 4, 32, block_t=16)
    kt = _fake_cache(T_cap=64)
    assert _encode(_fake_view(T=16), kt, cg.Codec(cg.BLOCK_UNIFORM, 4, 32, block_t=12)) == cg.CG_ERR_UNSUPPORTED
    assert _encode(_fake_view(T=16), kt, cg.Codec(cg.BLOCK_UNIFORM, 4, 32, block_t=64)) == cg.CG_ERR_UNSUPPORTED
    assert _encode(_fake_view(T=16), kt, tile, t0=8) == cg.CG_ERR_UNSUPPORTED
    assert _encode(_fake_view(T=16, dtype=cg.DTYPE_F32), kt, tile) == cg.CG_ERR_UNSUPPORTED
    assert _encode(_fake_view(T=16), _fake_cache(T_cap=64, residual=0), tile) == cg.CG_ERR_ARG
    assert _encode(_fake_view(T=16), _fake_cache(T_cap=40), tile) == cg.CG_ERR_SHAPE
    with pytest.raises(cg.CodecError) as e:
        cg.cache_bytes(tile, 0, 1, 1, 2, 40, 64)
    assert e.value.status == cg.CG_ERR_SHAPE
    assert _decode(_fake_view(T=16), _fake_cache(T_cap=64, len_=8), tile) == cg.CG_ERR_CAPACITY
    # device per-row lengths: 4-byte aligned; with them the host length no longer bounds the call
    # (the rows bound themselves on the device), so only the pointer is checked here
    assert _decode(_fake_view(T=16), _fake_cache(T_cap=64, len_=8), kivi, lens=0x70002) == cg.CG_ERR_ALIGN
    assert _decode(_fake_view(T=16), _fake_cache(T_cap=64, len_=8), tile, lens=0x70001) == cg.CG_ERR_ALIGN
    assert _decode(_fake_view(T=16), _fake_cache(T_cap=8), BU, lens=0x70000) == cg.CG_ERR_CAPACITY


def test_append_step_rejects_invalid_arguments():
    shp = cg.shape(2, 2, 64, 16)
    kn = _fake_view(L=1, T=1, strides=(128, 128, 64, 64))
    k = _fake_cache(L=2)
    cs = BU.struct()
    f = cg.lib().kv_append_step
    assert f(1, 1, C.byref(kn), C.byref(kn), 0x60000, 0x50000, shp, C.byref(cs), C.byref(k), C.byref(k), None,
             None, None, None) == cg.CG_ERR_ARG
    assert f(0, 3, C.byref(kn), C.byref(kn), 0x60000, 0x50000, shp, C.byref(cs), C.byref(k), C.byref(k), None,
             None, None, None) == cg.CG_ERR_ARG
    assert f(0, 1, C.byref(kn), C.byref(kn), None, 0x50000, shp, C.byref(cs), C.byref(k), C.byref(k), None, None,
             None, None) == cg.CG_ERR_ARG
    two = _fake_view(L=1, T=2)
    assert f(0, 1, C.byref(two), C.byref(two), 0x60000, 0x50000, shp, C.byref(cs), C.byref(k), C.byref(k), None,
             None, None, None) == cg.CG_ERR_SHAPE
    assert f(0, 2, C.byref(kn), C.byref(kn), 0x60000, 0x50000, shp, C.byref(cs), C.byref(k), C.byref(k), None,
             None, None, None) == cg.CG_ERR_SHAPE
    assert f(0, 1, C.byref(kn), C.byref(kn), 0x60002, 0x50000, shp, C.byref(cs), C.byref(k), C.byref(k), None,
             None, None, None) == cg.CG_ERR_ALIGN


def test_spectral_stats_reject_invalid_arguments():
    shp = cg.shape(1, 2, 64, 16)
    v = _fake_view(T=32)
    assert cg.spectral_workspace_bytes(shp, 16) > 0
    assert cg.spectral_workspace_bytes(shp, 3) == 0 and cg.spectral_workspace_bytes(shp, 64) == 0
    f = cg.lib().kv_spectral_stats
    ok = dict(s=0, blk=16, tau=0.04, ws=0x70000, stats=0x80000)
    def call(**kw):
        a = dict(ok, **kw)
        return f(a["s"], C.byref(a.get("view", v)), 0x50000, a.get("shp", shp), a["blk"], a["tau"], a["ws"],
                 a["stats"], None, None)
    assert call(blk=3) == cg.CG_ERR_UNSUPPORTED
    assert call(blk=1) == cg.CG_ERR_UNSUPPORTED
    assert call(tau=0.0) == cg.CG_ERR_ARG
    assert call(tau=float("nan")) == cg.CG_ERR_ARG
    assert call(s=2) == cg.CG_ERR_ARG
    assert call(ws=None) == cg.CG_ERR_ARG
    assert call(stats=None) == cg.CG_ERR_ARG
    assert call(ws=0x70008) == cg.CG_ERR_ALIGN
    assert call(stats=0x80004) == cg.CG_ERR_ALIGN
    assert call(view=_fake_view(H=3)) == cg.CG_ERR_SHAPE
    assert call(shp=cg.shape(1, 2, 64, 48)) == cg.CG_ERR_UNSUPPORTED


def test_gauge_grad_rejects_invalid_arguments():
    shp = cg.shape(1, 2, 64, 16)
    v = _fake_view(T=32)
    assert cg.gauge_grad_workspace_bytes(shp, 2, 32, 16) >= cg.spectral_workspace_bytes(shp, 16) > 0
    assert cg.gauge_grad_workspace_bytes(shp, 2, 32, 3) == 0
    assert cg.gauge_grad_workspace_bytes(cg.shape(1, 2, 40, 8), 2, 32, 16) == 0    # d not a multiple of 16
    assert cg.gauge_grad_workspace_bytes(cg.shape(1, 2, 256, 16), 2, 32, 16) == 0  # d above 128
    f = cg.lib().kv_gauge_grad
    ok = dict(s=0, A=0x40000, blk=16, tau=0.04, lf=1.0, lr=0.02, ws=0x70000, stats=0x80000, grad=0x90000)
    def call(**kw):
        a = dict(ok, **kw)
        return f(a["s"], C.byref(a.get("view", v)), a["A"], 0x50000, a.get("shp", shp), a["blk"], a["tau"], a["lf"],
                 a["lr"], a["ws"], a["stats"], a["grad"], None)
    assert call(blk=3) == cg.CG_ERR_UNSUPPORTED
    assert call(shp=cg.shape(1, 2, 256, 16), view=_fake_view(d=256)) == cg.CG_ERR_UNSUPPORTED
    assert call(tau=-1.0) == cg.CG_ERR_ARG
    assert call(lf=float("inf")) == cg.CG_ERR_ARG
    assert call(lr=float("nan")) == cg.CG_ERR_ARG
    assert call(s=-1) == cg.CG_ERR_ARG
    assert call(A=None) == cg.CG_ERR_ARG
    assert call(grad=None) == cg.CG_ERR_ARG
    assert call(A=0x40002) == cg.CG_ERR_ALIGN
    assert call(grad=0x90004) == cg.CG_ERR_ALIGN
    assert call(ws=0x70008) == cg.CG_ERR_ALIGN
    assert call(view=_fake_view(H=3)) == cg.CG_ERR_SHAPE


def test_attend_rejects_invalid_arguments():
    shp = cg.shape(2, 2, 64, 16)
    q = _fake_view(L=1, H=4, T=1, strides=(256, 256, 64, 64))
    k = _fake_cache(L=2, T_cap=64, len_=32)
    assert cg.attend_workspace_bytes(shp, 1, 1, 4, 64) >= 0
    assert cg.attend_workspace_bytes(shp, 1, 1, 3, 64) == 0      # Hq not a multiple of H
    assert cg.attend_workspace_bytes(shp, 1, 1, 4, 4096) > 0      # few rows: the positions are split
    f = cg.lib().kv_attend
    ok = dict(l0=0, l1=1, q=q, kc=k, vc=k, codec=BU, lens=None, scale=0.125, out=q, ws=0x70000)
    def call(**kw):
        a = dict(ok, **kw)
        cs = a["codec"].struct()
        return f(a["l0"], a["l1"], C.byref(a["q"]), C.byref(a["kc"]), C.byref(a["vc"]), a.get("gdev", 0x50000),
                 a.get("shp", shp), C.byref(cs), a["lens"], a["scale"], C.byref(a["out"]), a["ws"], None, None)
    assert call(l1=3) == cg.CG_ERR_ARG
    assert call(l0=1, l1=1) == cg.CG_ERR_ARG
    assert call(scale=float("inf")) == cg.CG_ERR_ARG
    assert call(gdev=0x50008) == cg.CG_ERR_ALIGN
    assert call(lens=0x60002) == cg.CG_ERR_ALIGN
    assert call(q=_fake_view(L=1, H=3, T=1)) == cg.CG_ERR_SHAPE                       # Hq % H
    assert call(q=_fake_view(L=1, H=4, T=2)) == cg.CG_ERR_SHAPE                       # one query position
    assert call(out=_fake_view(L=1, H=2, T=1)) == cg.CG_ERR_SHAPE                     # out heads != q heads
    assert call(vc=_fake_cache(L=2, T_cap=32, len_=32)) == cg.CG_ERR_SHAPE            # capacities differ
    assert call(kc=_fake_cache(L=2, T_cap=64, len_=65)) == cg.CG_ERR_CAPACITY         # len beyond capacity
    assert call(vc=_fake_cache(L=2, T_cap=64, len_=16)) == cg.CG_ERR_CAPACITY         # K and V lengths differ
    assert call(codec=cg.Codec(cg.BLOCK_UNIFORM, 5, 32)) == cg.CG_ERR_UNSUPPORTED
    big = _fake_cache(L=2, T_cap=4096, len_=4096)
    assert call(kc=big, vc=big, ws=None) == cg.CG_ERR_ARG                             # workspace needed
    assert call(kc=big, vc=big, ws=0x70008) == cg.CG_ERR_ALIGN


def test_attend_noalloc_validates_like_kv_attend_and_rejects_plans_beyond_its_scratch():
    """kv_attend_noalloc: the same validation as kv_attend (no workspace argument), and a split plan
    needing more than the library's 32 MiB device scratch is refused before anything is enqueued
    (or any device call made)."""
    f = cg.lib().kv_attend_noalloc
    def call(shp, q, kc, lens=None, l1=None, codec=BU, scale=0.125):
        cs = codec.struct()
        return f(0, q.L if l1 is None else l1, C.byref(q), C.byref(kc), C.byref(kc), 0x50000, shp, C.byref(cs),
                 lens, scale, C.byref(q), None, None)
    shp = cg.shape(2, 2, 64, 16)
    q = _fake_view(L=1, H=4, T=1, strides=(256, 256, 64, 64))
    k = _fake_cache(L=2, T_cap=64, len_=32)
    assert call(shp, q, k, l1=3) == cg.CG_ERR_ARG
    assert call(shp, q, k, scale=float("nan")) == cg.CG_ERR_ARG
    assert call(shp, q, k, lens=0x60002) == cg.CG_ERR_ALIGN
    assert call(shp, q, _fake_cache(L=2, T_cap=64, len_=65)) == cg.CG_ERR_CAPACITY
    assert call(shp, q, k, codec=cg.Codec(cg.BLOCK_UNIFORM, 5, 32)) == cg.CG_ERR_UNSUPPORTED
    # head_dim 256, 64 layers of one row, 8 query heads per KV head over 4096 positions: four splits
    # per row and 33.7 MB of partial results
    big = cg.shape(64, 8, 256, 128)
    need = cg.attend_workspace_bytes(big, 64, 1, 64, 4096)
    assert need > (32 << 20)
    qb = _fake_view(L=64, B=1, H=64, T=1, d=256, strides=(64 * 256, 64 * 256, 256, 256))
    kb = _fake_cache(L=64, B=1, H=8, T_cap=4096, d=256, len_=4096)
    assert call(big, qb, kb, lens=0x60000) == cg.CG_ERR_CAPACITY


def test_zfp_backend_sizes_and_restrictions():
    z = cg.Codec(cg.ZFP, 4)
    assert cg.cache_bytes(z, 0, 2, 3, 4, 64, 128) == (2 * 3 * 4 * 64 * 128 * 4 // 8, 0, 0)
    assert cg.cache_bytes(cg.Codec(cg.ZFP, 3), 1, 1, 1, 1, 8, 64)[0] == 8 * 64 * 3 // 8
    with pytest.raises(cg.CodecError) as e:
        cg.cache_bytes(cg.Codec(cg.ZFP, 5), 0, 1, 1, 2, 64, 64)
    assert e.value.status == cg.CG_ERR_UNSUPPORTED
    with pytest.raises(cg.CodecError) as e:
        cg.cache_bytes(z, 0, 1, 1, 2, 62, 64)
    assert e.value.status == cg.CG_ERR_SHAPE
    k = _fake_cache(T_cap=64, side=0, residual=0)
    assert _encode(_fake_view(T=6), k, z) == cg.CG_ERR_UNSUPPORTED
    assert _encode(_fake_view(T=8), k, z, t0=2) == cg.CG_ERR_UNSUPPORTED
    assert _decode(_fake_view(T=6), k, z) == cg.CG_ERR_UNSUPPORTED
    assert _decode(_fake_view(T=8), k, z, lens=0x70000) == cg.CG_ERR_UNSUPPORTED   # whole 4-token rows
    assert _encode(_fake_view(T=8), _fake_cache(T_cap=62, side=0), z) == cg.CG_ERR_SHAPE
    shp = cg.shape(1, 2, 64, 16)
    kn = _fake_view(L=1, T=1, strides=(128, 128, 64, 64))
    cs = z.struct()
    assert cg.lib().kv_append_step(0, 1, C.byref(kn), C.byref(kn), 0x60000, 0x50000, shp, C.byref(cs), C.byref(k),
                                   C.byref(k), None, None, None, None) == cg.CG_ERR_UNSUPPORTED
    q = _fake_view(L=1, H=2, T=1, strides=(128, 128, 64, 64))
    assert cg.lib().kv_attend(0, 1, C.byref(q), C.byref(k), C.byref(k), 0x50000, shp, C.byref(cs), None, 0.1,
                              C.byref(q), 0x70000, None, None) == cg.CG_ERR_UNSUPPORTED


def test_paged_entry_points_reject_invalid_arguments():
    shp = cg.shape(2, 2, 64, 16)
    q = _fake_view(L=1, H=4, T=1, strides=(256, 256, 64, 64))
    pool = _fake_cache(L=2, B=5, T_cap=64)
    pt = cg.PageTable(0x90000, 3, 64)
    f = cg.lib().kv_attend_paged
    def att(**kw):
        a = dict(dict(q=q, kc=pool, vc=pool, pt=pt, codec=BU, lens=0x60000, ws=0x70000), **kw)
        cs = a["codec"].struct()
        ptr = None if a["pt"] is None else C.byref(a["pt"])
        return f(0, 1, C.byref(a["q"]), C.byref(a["kc"]), C.byref(a["vc"]), ptr, 0x50000, shp, C.byref(cs),
                 a["lens"], 0.1, C.byref(a["q"]), a["ws"], None, None)
    assert att(lens=None) == cg.CG_ERR_ARG                                        # lengths required
    assert att(pt=None) == cg.CG_ERR_ARG
    assert att(pt=cg.PageTable(0, 3, 64)) == cg.CG_ERR_ARG
    assert att(pt=cg.PageTable(0x90002, 3, 64)) == cg.CG_ERR_ALIGN
    assert att(pt=cg.PageTable(0x90000, 3, 32)) == cg.CG_ERR_SHAPE               # page size != T_cap
    assert att(pt=cg.PageTable(0x90000, 3, 96), kc=_fake_cache(L=2, B=5, T_cap=96),
               vc=_fake_cache(L=2, B=5, T_cap=96)) == cg.CG_ERR_SHAPE             # not a multiple of 64
    assert att(codec=cg.Codec(cg.KIVI, 3, 64, 32, 64, 128), kc=_fake_cache(L=2, B=5, T_cap=64),
               vc=_fake_cache(L=2, B=5, T_cap=64)) == cg.CG_ERR_UNSUPPORTED       # windows are per row
    assert att(codec=cg.Codec(cg.BLOCK_UNIFORM, 4, 32, block_t=16)) == cg.CG_ERR_UNSUPPORTED
    assert att(vc=_fake_cache(L=2, B=4, T_cap=64)) == cg.CG_ERR_SHAPE            # pools differ
    assert cg.attend_paged_workspace_bytes(shp, 1, 1, 4, 0, 64) == 0
    assert cg.attend_paged_workspace_bytes(shp, 1, 1, 4, 64, 64) == cg.attend_workspace_bytes(shp, 1, 1, 4, 4096)
    # paged encode: t0 on a 32-position boundary, within the table
    X = _fake_view(L=2, T=32)
    cs = BU.struct()
    enc = cg.lib().kv_encode_paged
    assert enc(0, C.byref(X), C.byref(pt), 0x50000, shp, C.byref(cs), C.byref(pool), 16, None, None) == cg.CG_ERR_UNSUPPORTED
    assert enc(0, C.byref(X), C.byref(pt), 0x50000, shp, C.byref(cs), C.byref(pool), 192, None, None) == cg.CG_ERR_CAPACITY
    assert enc(0, C.byref(X), None, 0x50000, shp, C.byref(cs), C.byref(pool), 0, None, None) == cg.CG_ERR_ARG
    # paged append
    kn = _fake_view(L=1, T=1, strides=(128, 128, 64, 64))
    app = cg.lib().kv_append_paged
    assert app(0, 1, C.byref(kn), C.byref(kn), None, C.byref(pt), 0x50000, shp, C.byref(cs), C.byref(pool),
               C.byref(pool), None, None) == cg.CG_ERR_ARG
    assert app(0, 1, C.byref(kn), C.byref(kn), 0x60000, C.byref(cg.PageTable(0x90000, 3, 32)), 0x50000, shp,
               C.byref(cs), C.byref(pool), C.byref(pool), None, None) == cg.CG_ERR_SHAPE


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(cg, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(cg, "_lib", None)
    with pytest.raises(ImportError):
        cg.lib()


def test_stream_probe_rejects_bad_sizes_on_the_host():
    L = cg.lib()
    fake = C.c_void_p(1 << 20)  # never dereferenced: every case fails validation first
    for rb, wb, st in ((0, 0, cg.CG_ERR_ARG), (8192 + 16, 0, cg.CG_ERR_ARG), (8192, 8, cg.CG_ERR_ARG),
                       (8192, -16, cg.CG_ERR_ARG)):
        assert L.cg_stream_probe(fake, rb, fake, wb, None) == st
    assert L.cg_stream_probe(None, 8192, fake, 0, None) == cg.CG_ERR_ARG
    assert L.cg_stream_probe(fake, 8192, None, 16, None) == cg.CG_ERR_ARG
    assert L.cg_stream_probe(C.c_void_p((1 << 20) + 8), 8192, fake, 16, None) == cg.CG_ERR_ALIGN


def test_selftest_rejects_bad_arguments_on_the_host():
    L = cg.lib()
    fake = C.c_void_p(1 << 20)  # never dereferenced: every case fails validation first
    for which in (-1, 3, 100):
        assert L.cg_selftest(which, fake, None) == cg.CG_ERR_ARG
    for which in (0, 1, 2):
        assert L.cg_selftest(which, None, None) == cg.CG_ERR_ARG
        assert L.cg_selftest(which, C.c_void_p((1 << 20) + 4), None) == cg.CG_ERR_ALIGN
