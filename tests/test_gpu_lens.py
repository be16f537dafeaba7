"""kv_decode with per-row device lengths (a layer's [B x H x T x d] cache whose batch rows hold
different numbers of tokens, paper section 3), against the oracle's decode with the same lengths.

Each batch row's cache is what encoding only that row's first lens[b] tokens gives (the oracle
encodes the rows one by one), so a KIVI row quantises T_q(lens[b]) positions and keeps the rest
in its window, and a tile row stages its unfinished tile.  Rows write only their positions
[t0, min(t0 + T, lens[b])); the rest of the view keeps its previous contents; a length outside
[0, T_cap] flags CG_FLAG_POS_RANGE and writes nothing."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2607_20538_amd import codec as cg
from paper_2607_20538_amd import synth

from _parity import cache_to_dev, check_bf16_within_ulp, group_rel_err, out_host, to_cg, GAUGE_TOL

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cg.lib()


@pytest.fixture(params=["mfma", "mfma-multi", "generic"])
def kernels(request, monkeypatch):
    monkeypatch.delenv("CG_KERNELS", raising=False)
    monkeypatch.delenv("CG_TILES_PER_WG", raising=False)
    if request.param == "generic":
        monkeypatch.setenv("CG_KERNELS", "generic")
    elif request.param == "mfma-multi":
        monkeypatch.setenv("CG_TILES_PER_WG", "7")
    return request.param


CASES = [(O.BLOCK_UNIFORM, 128, 4, 64, 1), (O.BLOCK_UNIFORM, 32, 6, 64, 1), (O.KIVI, 32, 3, 64, 1),
         (O.KIVI, 8, 4, 64, 1), (O.BLOCK_UNIFORM, 128, 4, 128, 16), (O.PASSTHROUGH, 128, 8, 64, 1)]


def _row_caches(oc, s, X, G, lens, T_cap):
    """The cache of every batch row b encoded from its first lens[b] tokens alone."""
    L_, B, H, _, d = X.shape
    full = O.empty_cache(oc, s, L_, B, H, T_cap, d)
    for b, n in enumerate(lens):
        if n == 0:
            continue
        part, flags = O.kv_encode(oc, s, np.ascontiguousarray(X[:, b:b + 1, :, :n]), G, T_cap=T_cap)
        assert flags == 0
        for key in full:
            if full[key] is not None:
                full[key][:, b:b + 1] = part[key]
    return full


@pytest.mark.parametrize("backend,g,bits,n,bt", CASES)
def test_ragged_rows_match_oracle(backend, g, bits, n, bt, kernels):
    L, B, H, d = 2, 4, 2, 128
    T_cap = 480
    lens = [T_cap - 7, 301, 0, 171]            # ragged; row 2 holds nothing
    w = synth.Workload("lens", L=L, B=B, H=H, T=T_cap, d=d, dtype="bf16", g=g, backend="bu", bits=bits,
                       data_seed=0x1E45)
    G = O.gauge_make(O.GAUGE_HAAR, L, H, d, g, seed=41)
    shp = cg.shape(L, H, d, g)
    Gd = cg.alloc_gauge(shp)
    cg.gauge_make(cg.GAUGE_USER, shp, params=G, G_host=None, G_dev=Gd)
    oc = O.Codec(backend=backend, bits=bits, block_c=n, key_tokens=32, val_channels=64, residual=128, block_t=bt)
    lens_d = torch.tensor(lens, dtype=torch.int32, device="cuda")
    for s in (0, 1):
        X = synth.kv_tensor(w, s)
        orc = _row_caches(oc, s, X, G, lens, T_cap)
        dev = cache_to_dev(orc, oc, s, L, B, H, T_cap, d, len_=0)   # the host length is not used
        for t0, T in ((0, T_cap), (37, 300)):
            ref = O.kv_decode(oc, s, G, orc, t0, T, lens=lens, out_bf16=False)
            for dt in (torch.float32, torch.bfloat16):
                Y = torch.full((L, B, H, T, d), 9.0, dtype=dt, device="cuda")
                err = torch.zeros(1, dtype=torch.int32, device="cuda")
                cg.kv_decode(s, dev, Gd, shp, to_cg(oc), t0, Y, err_flag=err, lens=lens_d)
                torch.cuda.synchronize()
                assert int(err.item()) == 0
                got = out_host(Y)
                for b, nb in enumerate(lens):
                    m = max(0, min(T, nb - t0))               # view rows the row writes
                    if backend == O.KIVI:
                        q = max(0, min(m, O.kivi_tq(nb, oc) - t0))
                    elif bt > 1:
                        q = max(0, min(m, O.tile_tq(nb, oc) - t0))
                    else:
                        q = m
                    rb, gb = ref[:, b:b + 1], got[:, b:b + 1]
                    if dt == torch.float32:
                        assert group_rel_err(rb[:, :, :, :q], gb[:, :, :, :q], g) <= GAUGE_TOL
                        np.testing.assert_array_equal(gb[:, :, :, q:m], rb[:, :, :, q:m])
                        assert (gb[:, :, :, m:] == 9.0).all()
                    else:
                        check_bf16_within_ulp(rb[:, :, :, :q], gb[:, :, :, :q], g)
                        np.testing.assert_array_equal(gb[:, :, :, q:m], X[:, b:b + 1, :, t0 + q:t0 + m])
                        assert (gb[:, :, :, m:] == 0x4110).all()  # bf16 9.0


def test_lengths_outside_the_cache_are_flagged(kernels):
    L, B, H, d, g = 1, 3, 2, 128, 128
    T_cap = 96
    shp = cg.shape(L, H, d, g)
    Gd = cg.alloc_gauge(shp)
    cg.gauge_make(cg.GAUGE_HAAR, shp, seed=3, G_host=None, G_dev=Gd)
    codec = cg.Codec(cg.KIVI, 3, 64, 32, 64, 64)
    cache = cg.Cache(codec, 0, L, B, H, T_cap, d)
    for buf in (cache.codes, cache.side, cache.residual):
        buf.zero_()
    Y = torch.full((L, B, H, T_cap, d), 9.0, dtype=torch.bfloat16, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    lens = torch.tensor([T_cap + 1, -2, 40], dtype=torch.int32, device="cuda")
    cg.kv_decode(0, cache, Gd, shp, codec, 0, Y, err_flag=err, lens=lens)
    torch.cuda.synchronize()
    assert int(err.item()) & cg.CG_FLAG_POS_RANGE
    assert bool((Y[:, :2].float() == 9.0).all())          # flagged rows write nothing
    assert bool((Y[:, 2, :, :40].float() == 0.0).all())    # row 2: 40 window tokens (all zero)
    assert bool((Y[:, 2, :, 40:].float() == 9.0).all())
