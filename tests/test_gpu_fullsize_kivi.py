"""Full-size parity of the KIVI-style workload: L = 32, B = 4, H = 8, T = 32768, head_dim 128,
bf16, Haar gauge g = 32, 3 bits, keys per channel over 32-token groups, values per token over
64 channels, a 128-token window (section 4.3), encoded and decoded as bench.py runs it (each
whole K / V tensor in one call, so every workgroup runs the multi-tile pipelines).

Inputs: synth's first two layers repeated over the 32 (materialised: the input views span more
than 2^32 bytes, so addressing is exercised at full size).  The oracle takes whole (layer,
batch, head) slices at the start, the middle and the end of the tensor: its own encode of the
same slice input with its own Haar gauge under the fused-encoder criteria (codes, side words,
and the window bit for bit), and its decode of the GPU's cache rows against the GPU's decoded
rows (bf16 within an ulp; window rows bit for bit)."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2607_20538_amd import codec as cg
from paper_2607_20538_amd import synth

from _parity import bf16_slice_host, cache_slice, check_bf16_within_ulp, check_fused_codes

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS["kivi"]
ND = 2                                          # distinct layers, repeated over W.L
SLICES = [(0, 0, 0), (13, 2, 5), (31, 3, 7)]    # (layer, batch, head)


@pytest.fixture(scope="module")
def gauges():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    shp = cg.shape(W.L, W.H, W.d, W.g)
    Gd = cg.alloc_gauge(shp)
    cg.gauge_make(cg.GAUGE_HAAR, shp, seed=W.gauge_seed, G_host=None, G_dev=Gd)
    G_orc = O.gauge_make(O.GAUGE_HAAR, W.L, W.H, W.d, W.g, seed=W.gauge_seed)
    return shp, Gd, G_orc


def _input(s):
    xs = synth.kv_tensor(W, s, L=ND)
    xs = torch.from_numpy(xs.view(np.int16)).view(torch.bfloat16).cuda()
    X = torch.empty((W.L, W.B, W.H, W.T, W.d), dtype=torch.bfloat16, device="cuda")
    for l in range(W.L):
        X[l] = xs[l % ND]
    del xs
    return X


@pytest.mark.parametrize("s", [0, 1])
def test_kivi_full_size_matches_oracle(gauges, s):
    shp, Gd, G_orc = gauges
    codec = cg.Codec(cg.KIVI, W.bits, 64, W.key_tokens, W.val_channels, W.residual)
    oc = O.Codec(backend=O.KIVI, bits=W.bits, key_tokens=W.key_tokens, val_channels=W.val_channels,
                 residual=W.residual)
    tq = O.kivi_tq(W.T, oc)
    X = _input(s)
    cache = cg.Cache(codec, s, W.L, W.B, W.H, W.T, W.d)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    cg.kv_encode(s, X, Gd, shp, codec, cache, err_flag=err)
    del X
    cache.len = W.T
    Y = torch.empty((W.L, W.B, W.H, W.T, W.d), dtype=torch.bfloat16, device="cuda")
    cg.kv_decode(s, cache, Gd, shp, codec, 0, Y, err_flag=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for l, b, h in SLICES:
        xs = bf16_slice_host(synth.kv_slice(W.data_seed, s, l % ND, b, h, W.T, W.d, W.keys))[None, None, None]
        Gs = np.ascontiguousarray(G_orc[l:l + 1, :, h:h + 1])
        orc, flags = O.kv_encode(oc, s, xs, Gs, T_cap=W.T)
        assert flags == 0
        zo, _ = O.kv_encode(O.Codec(backend=O.PASSTHROUGH), s, xs, Gs, T_cap=W.T)
        got = cache_slice(cache, oc, s, l, b, h)
        check_fused_codes(got, orc, zo["codes"], oc, s, W.d, tq)
        np.testing.assert_array_equal(got["residual"], orc["residual"])
        ref = O.kv_decode(oc, s, Gs, got, 0, W.T, lens=[W.T], out_bf16=False)
        y = Y[l, b, h].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)[None, None, None]
        check_bf16_within_ulp(ref[:, :, :, :tq], y[:, :, :, :tq], W.g)
        np.testing.assert_array_equal(y[:, :, :, tq:], xs[:, :, :, tq:])
    del Y, cache
    torch.cuda.empty_cache()
