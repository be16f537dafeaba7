"""Full-size parity of the 27B-shaped sweep: L = 46, B = 2, H = 16, T = 16384, head_dim 128, bf16,
block-uniform with 64-channel blocks, Haar gauges g in {8, 32, 128} x b in {3, 4, 6}, each whole
K / V tensor encoded and decoded in one call as bench.py times it (every workgroup runs the
multi-tile pipelines; the input views span more than 2^32 bytes).

Inputs: synth's first two layers repeated over the 46.  The oracle checks whole (layer, batch,
head) slices at the start and the end of the tensor: its own encode of the slice with its own
Haar gauge under the fused-encoder criteria, and its decode of the GPU's cache rows against the
GPU's decoded rows (bf16 within an ulp)."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2607_20538_amd import codec as cg
from paper_2607_20538_amd import synth

from _parity import bf16_slice_host, cache_slice, check_bf16_within_ulp, check_fused_codes

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS["gemma27b"]
ND = 2
SLICES = [(0, 0, 0), (45, 1, 15)]
SWEEP = [(g, b) for g in (8, 32, 128) for b in (3, 4, 6)]


@pytest.fixture(scope="module")
def inputs():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    out = {}
    for s in (0, 1):
        xs = synth.kv_tensor(W, s, L=ND)
        xs = torch.from_numpy(xs.view(np.int16)).view(torch.bfloat16).cuda()
        X = torch.empty((W.L, W.B, W.H, W.T, W.d), dtype=torch.bfloat16, device="cuda")
        for l in range(W.L):
            X[l] = xs[l % ND]
        out[s] = X
        del xs
    yield out
    out.clear()
    torch.cuda.empty_cache()


_GAUGES = {}


def _oracle_gauge(g):
    """The oracle's own Haar gauge of the workload (all layers: the sampled slices include the last)."""
    if g not in _GAUGES:
        _GAUGES[g] = O.gauge_make(O.GAUGE_HAAR, W.L, W.H, W.d, g, seed=W.gauge_seed)
    return _GAUGES[g]


@pytest.mark.parametrize("g,bits", SWEEP)
def test_27b_sweep_full_size_matches_oracle(inputs, g, bits):
    shp = cg.shape(W.L, W.H, W.d, g)
    Gd = cg.alloc_gauge(shp)
    cg.gauge_make(cg.GAUGE_HAAR, shp, seed=W.gauge_seed, G_host=None, G_dev=Gd)
    codec = cg.Codec(cg.BLOCK_UNIFORM, bits, W.block_c)
    oc = O.Codec(backend=O.BLOCK_UNIFORM, bits=bits, block_c=W.block_c)
    G_orc = _oracle_gauge(g)
    for s in (0, 1):
        cache = cg.Cache(codec, s, W.L, W.B, W.H, W.T, W.d)
        err = torch.zeros(1, dtype=torch.int32, device="cuda")
        cg.kv_encode(s, inputs[s], Gd, shp, codec, cache, err_flag=err)
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
            check_fused_codes(got, orc, zo["codes"], oc, s, W.d, W.T)
            ref = O.kv_decode(oc, s, Gs, got, 0, W.T, out_bf16=False)
            y = Y[l, b, h].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)[None, None, None]
            check_bf16_within_ulp(ref, y, g)
        del Y, cache
    del Gd
    torch.cuda.empty_cache()
