"""Launch geometries: the matrix-core pipelines in the multi-tile form the benchmarks run.

At test sizes the resident grid gives every workgroup one 32-token tile, so the steady state
of the software pipelines (LDS ring wrap-around, prefetch of later tiles, the overlapped flush
of the previous tile, the decoders' exact counts of younger memory operations) only runs on
full-size inputs.  CG_TILES_PER_WG=k fixes k tiles per workgroup; every case here runs with
k = 7 and k = 16 on 17 tiles per slice (a ragged last tile), at least kStages + 2 = 7 tiles for
the encoder's ring and DS + 2 = 10 for the decoders', and is compared

  * bit for bit with the resident (one tile per workgroup) geometry: codes, side information,
    windows and decoded rows (the two geometries run the same arithmetic on every tile), and
  * with the CPU oracle under the criteria of tests/_parity.py.

The templates are the ones the workloads time: block-uniform g = 128 at 3 / 4 / 6 bits (the
Llama-3-8B headline, the rolling history and the 27B sweep), g = 32 and g = 8 at 3 / 4 / 6 bits
(the 27B sweep's centred decoder), KIVI with g = 32 at 3 bits (key encoder, key decoder, value
rows, window), 16-token tiles, the zfp-style coder and the error-free backend."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2607_20538_amd import codec as cg
from paper_2607_20538_amd import synth

from _parity import (bf16_dev, cache_to_dev, cache_to_host, check_bf16_within_ulp, check_fused_codes,
                     group_rel_err, out_host, to_cg, x_dev, GAUGE_TOL)

pytestmark = pytest.mark.gpu

GEOMETRIES = [None, 7, 16]          # None: the resident grid
NT = 17                             # tiles per slice
T_BU = 32 * (NT - 1) + 13           # 525 tokens: 16 whole tiles and a ragged one


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cg.lib()


def _set_geometry(monkeypatch, k):
    monkeypatch.delenv("CG_KERNELS", raising=False)
    if k is None:
        monkeypatch.delenv("CG_TILES_PER_WG", raising=False)
    else:
        monkeypatch.setenv("CG_TILES_PER_WG", str(k))


def _workload(T, L=1, B=1, H=2, seed=0x6E0):
    return synth.Workload("geometry", L=L, B=B, H=H, T=T, d=128, dtype="bf16", g=0, backend="bu", bits=4,
                          data_seed=seed)


def _gauge(kind, L, H, g, seed=23):
    G = O.gauge_make(kind, L, H, 128, g, seed=seed)
    shp = cg.shape(L, H, 128, g)
    Gd = cg.alloc_gauge(shp)
    cg.gauge_make(cg.GAUGE_USER, shp, params=G, G_host=None, G_dev=Gd)
    return G, Gd, shp


def _host(dev: cg.Cache) -> dict:
    return {k: (None if getattr(dev, k) is None else getattr(dev, k).cpu().numpy().copy())
            for k in ("codes", "side", "residual")}


def _same_bytes(a: dict, b: dict):
    for k in a:
        if a[k] is None:
            assert b[k] is None
        else:
            np.testing.assert_array_equal(a[k], b[k], err_msg=k)


CASES = [
    # (name, backend, g, bits, n, block_t)
    ("bu-g128-b4", O.BLOCK_UNIFORM, 128, 4, 64, 1),
    ("bu-g128-b6", O.BLOCK_UNIFORM, 128, 6, 64, 1),
    ("bu-g128-b3", O.BLOCK_UNIFORM, 128, 3, 64, 1),
    ("bu-g32-b3", O.BLOCK_UNIFORM, 32, 3, 64, 1),
    ("bu-g32-b4", O.BLOCK_UNIFORM, 32, 4, 64, 1),
    ("bu-g32-b6", O.BLOCK_UNIFORM, 32, 6, 64, 1),
    ("bu-g8-b3", O.BLOCK_UNIFORM, 8, 3, 64, 1),
    ("bu-g8-b6", O.BLOCK_UNIFORM, 8, 6, 64, 1),
    ("bu-g64-b4-n32", O.BLOCK_UNIFORM, 64, 4, 32, 1),
    ("kivi-g32-b3", O.KIVI, 32, 3, 64, 1),
    ("kivi-g128-b4", O.KIVI, 128, 4, 64, 1),
    ("tile-g128-b4", O.BLOCK_UNIFORM, 128, 4, 128, 16),
    ("tile-g32-b3", O.BLOCK_UNIFORM, 32, 3, 64, 16),
    ("tile-g64-b4-n128", O.BLOCK_UNIFORM, 64, 4, 128, 16),
    ("zfp-g128-r4", O.ZFP, 128, 4, 64, 1),
    ("pass-g128", O.PASSTHROUGH, 128, 8, 64, 1),
]


@pytest.mark.parametrize("name,backend,g,bits,n,bt", CASES, ids=[c[0] for c in CASES])
def test_multi_tile_pipelines_match_one_tile_and_oracle(name, backend, g, bits, n, bt, monkeypatch):
    kivi = backend == O.KIVI
    # KIVI: T_q = floor((T - 128) / 32) * 32 quantised positions in 17 key groups, the rest in
    # the window; zfp: whole 4-token rows
    T = 32 * NT + 128 + 5 if kivi else (T_BU - 1 if backend == O.ZFP else T_BU)
    T_cap = ((T + 31) // 32) * 32 + (32 if kivi else 0)
    w = _workload(T)
    # zfp-style: the identity gauge makes z = x exact on the matrix cores, so the coder's blocks and
    # decoded rows must equal the oracle's bit for bit
    G, Gd, shp = _gauge(O.GAUGE_IDENTITY if backend == O.ZFP else O.GAUGE_HAAR, 1, 2, g)
    oc = O.Codec(backend=backend, bits=bits, block_c=n, key_tokens=32, val_channels=64, residual=128, block_t=bt)
    tq = O.kivi_tq(T, oc) if kivi else (O.tile_tq(T, oc) if bt > 1 else T)
    lens = [T] * w.B
    for s in (0, 1):
        X = synth.kv_tensor(w, s)
        orc, flags = O.kv_encode(oc, s, X, G, T_cap=T_cap)
        assert flags == 0
        zo, _ = O.kv_encode(O.Codec(backend=O.PASSTHROUGH), s, X, G, T_cap=T_cap)
        ref32 = O.kv_decode(oc, s, G, orc, 0, T, lens=lens, out_bf16=False)
        ddev = cache_to_dev(orc, oc, s, w.L, w.B, w.H, T_cap, 128, len_=T)
        enc, dec32, dec16 = {}, {}, {}
        for k in GEOMETRIES:
            _set_geometry(monkeypatch, k)
            err = torch.zeros(1, dtype=torch.int32, device="cuda")
            dev = cg.Cache(to_cg(oc), s, w.L, w.B, w.H, T_cap, 128)
            for key in ("codes", "side", "residual"):
                if getattr(dev, key) is not None:
                    getattr(dev, key).fill_(0x5A)        # untouched bytes compare equal across runs
            cg.kv_encode(s, x_dev(X), Gd, shp, to_cg(oc), dev, err_flag=err)
            outs = []
            for dt in (torch.float32, torch.bfloat16):
                Y = torch.full((w.L, w.B, w.H, T, 128), 3.0, dtype=dt, device="cuda")
                cg.kv_decode(s, ddev, Gd, shp, to_cg(oc), 0, Y, err_flag=err)
                outs.append(Y)
            torch.cuda.synchronize()
            assert int(err.item()) == 0, (k, int(err.item()))
            enc[k], dec32[k], dec16[k] = _host(dev), out_host(outs[0]), out_host(outs[1])
        base = GEOMETRIES[0]
        for k in GEOMETRIES[1:]:
            _same_bytes(enc[base], enc[k])
            np.testing.assert_array_equal(dec32[base], dec32[k])
            np.testing.assert_array_equal(dec16[base], dec16[k])
        got = cache_to_host_np(enc[16], oc, s, w, T_cap)
        if backend == O.PASSTHROUGH:
            assert group_rel_err(orc["codes"][:, :, :, :T], got["codes"][:, :, :, :T], g) <= GAUGE_TOL
        elif backend == O.ZFP:
            np.testing.assert_array_equal(got["codes"][:, :, :, :T // 4], orc["codes"][:, :, :, :T // 4])
            np.testing.assert_array_equal(dec32[16], ref32)
        else:
            check_fused_codes(got, orc, zo["codes"], oc, s, 128, tq)
            if kivi:   # the window slots the encode writes: positions [T_q, T), slot = position mod 160
                slots = [t % (oc.residual + oc.key_tokens) for t in range(tq, T)]
                np.testing.assert_array_equal(got["residual"][:, :, :, slots], orc["residual"][:, :, :, slots])
        assert group_rel_err(ref32[:, :, :, :tq], dec32[16][:, :, :, :tq], g) <= GAUGE_TOL
        check_bf16_within_ulp(ref32[:, :, :, :tq], dec16[16][:, :, :, :tq], g)
        if tq < T:   # window / staged rows come back bit for bit
            np.testing.assert_array_equal(dec16[16][:, :, :, tq:], X[:, :, :, tq:])


def cache_to_host_np(raw: dict, oc: O.Codec, s: int, w, T_cap: int) -> dict:
    """Raw device bytes (as copied by _host) in the oracle's layout."""
    lay = O.cache_layout(oc, s, w.L, w.B, w.H, T_cap, 128)
    out = {}
    for key in ("codes", "side", "residual"):
        if lay[key] is None:
            out[key] = None
            continue
        shp, dt = lay[key]
        nbytes = int(np.prod(shp)) * np.dtype(dt).itemsize
        out[key] = raw[key][:nbytes].view(dt).reshape(shp)
    return out


# ------------------------------------------------------------------------------------------
# rolling step in the multi-tile form: per-row positions, 6-bit g = 128 (the rolling workload's
# templates) and KIVI g = 32 3-bit (flushes of the window during the steps)
# ------------------------------------------------------------------------------------------
@pytest.mark.parametrize("backend,g,bits", [(O.BLOCK_UNIFORM, 128, 6), (O.KIVI, 32, 3), (O.BLOCK_UNIFORM, 32, 4)])
def test_append_step_multi_tile_history(backend, g, bits, monkeypatch):
    L, B, H, d = 2, 2, 2, 128
    T0, steps = 540, 24
    T_cap = 576
    w = _workload(T_cap, L=L, B=B, H=H, seed=0xA11)
    G, Gd, shp = _gauge(O.GAUGE_HAAR, L, H, g, seed=31)
    oc = O.Codec(backend=backend, bits=bits, block_c=64, key_tokens=32, val_channels=64, residual=128)
    Xk, Xv = synth.kv_tensor(w, 0), synth.kv_tensor(w, 1)
    start = np.array([T0, T0 + 7])   # row 1 runs 7 positions ahead (its slots [T0, T0 + 7) stay empty)
    hists = {}
    caches = {}
    for k in GEOMETRIES:
        _set_geometry(monkeypatch, k)
        ok, _ = O.kv_encode(oc, 0, np.ascontiguousarray(Xk[:, :, :, :T0]), G, T_cap=T_cap)
        ov, _ = O.kv_encode(oc, 1, np.ascontiguousarray(Xv[:, :, :, :T0]), G, T_cap=T_cap)
        kc = cache_to_dev(ok, oc, 0, L, B, H, T_cap, d)
        vc = cache_to_dev(ov, oc, 1, L, B, H, T_cap, d)
        khist = torch.full((L, B, H, T_cap, d), 5.0, dtype=torch.bfloat16, device="cuda")
        vhist = torch.full_like(khist, 5.0)
        err = torch.zeros(1, dtype=torch.int32, device="cuda")
        for i in range(steps):
            pos = start + i
            kn = np.ascontiguousarray(Xk[:, np.arange(B), :, pos].transpose(1, 0, 2, 3))
            vn = np.ascontiguousarray(Xv[:, np.arange(B), :, pos].transpose(1, 0, 2, 3))
            if k == GEOMETRIES[-1]:
                O.kv_append(oc, 0, kn, G, ok, pos)
                O.kv_append(oc, 1, vn, G, ov, pos)
            pos_d = torch.tensor(pos, dtype=torch.int32, device="cuda")
            cg.kv_append_step(0, L, bf16_dev(kn[:, :, :, None, :]), bf16_dev(vn[:, :, :, None, :]), pos_d, Gd, shp,
                              to_cg(oc), kc, vc, khist, vhist, err_flag=err)
        torch.cuda.synchronize()
        assert int(err.item()) == 0
        hists[k] = (out_host(khist), out_host(vhist))
        caches[k] = (cache_to_host(kc, oc, 0), cache_to_host(vc, oc, 1), kc, vc)
    for k in GEOMETRIES[1:]:
        for i in range(2):
            np.testing.assert_array_equal(hists[GEOMETRIES[0]][i], hists[k][i])
    final = start + steps - 1
    kc_h, vc_h, kc, vc = caches[GEOMETRIES[-1]]
    lens = torch.tensor(final + 1, dtype=torch.int32, device="cuda")
    for s, orc, got, dc in ((0, ok, kc_h, kc), (1, ov, vc_h, vc)):
        X = Xk if s == 0 else Xv
        zo, _ = O.kv_encode(O.Codec(backend=O.PASSTHROUGH), s, X, G, T_cap=T_cap)
        held = int(final.min()) + 1
        tq = O.kivi_tq(held, oc) if backend == O.KIVI else held
        check_fused_codes(got, orc, zo["codes"], oc, s, d, tq)
        # the history rows: against the oracle decoding the GPU's own cache, and against
        # kv_decode of the same cache with the rows' lengths on the device
        ref = O.kv_decode(oc, s, G, got, 0, T_cap, lens=final + 1, out_bf16=False)
        ref16 = O.kv_decode(oc, s, G, got, 0, T_cap, lens=final + 1, out_bf16=True)
        Y = torch.full((L, B, H, T_cap, d), 5.0, dtype=torch.bfloat16, device="cuda")
        cg.kv_decode(s, dc, Gd, shp, to_cg(oc), 0, Y, lens=lens)
        torch.cuda.synchronize()
        h = hists[GEOMETRIES[-1]][s]
        np.testing.assert_array_equal(out_host(Y), h)
        for b in range(B):
            n = int(final[b]) + 1
            tqb = O.kivi_tq(n, oc) if backend == O.KIVI else n
            check_bf16_within_ulp(ref[:, b:b + 1, :, :tqb], h[:, b:b + 1, :, :tqb], g)
            # window rows: the cache's raw bf16 (row 1's never-written slots hold zeros on both sides)
            np.testing.assert_array_equal(h[:, b, :, tqb:n], ref16[:, b, :, tqb:n])
            assert (h[:, b, :, n:] == 0x40A0).all()      # bf16 5.0: rows past the position untouched
