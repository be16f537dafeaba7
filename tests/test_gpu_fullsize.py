"""Full-size parity: the Llama-3-8B-shaped workload (32 layers, 8 KV heads, head_dim 128,
8192 tokens, bf16; Haar gauge g = 128; block-uniform 4-bit, block 64) encoded and decoded in
the same launch configuration as bench.py (whole K / V tensors in one call each).

The oracle cannot redo 2 x 268M elements in seconds, so it checks sampled outputs it can
compute on their own: token windows at the start, middle and end of several (layer, head)
slices of K and V, encoded by the oracle from the same inputs with its own Haar gauge and
compared under the fused-encoder criteria; and the GPU decoder's rows against the oracle
decoding the GPU's own cache rows.  Every element is checked by a property that holds at any
size: per token and group, ||x - xhat||_2 stays within the quantiser bound sqrt(sum_k n (sc_k /
2)^2) of the side information stored for it (the gauge is orthogonal), widened by the bf16
output rounding and the binary32 gauge tolerance."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2607_20538_amd import codec as cg
from paper_2607_20538_amd import synth

from _parity import check_bf16_within_ulp, check_fused_codes, to_cg

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS["llama8b"]
SLICES = [(0, 0), (13, 5), (31, 7)]           # (layer, head)
WINDOWS = [(0, 160), (4000, 4160), (W.T - 160, W.T)]


@pytest.fixture(scope="module")
def full():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    shp = cg.shape(W.L, W.H, W.d, W.g)
    codec = cg.Codec(cg.BLOCK_UNIFORM, W.bits, W.block_c)
    Gd = cg.alloc_gauge(shp)
    cg.gauge_make(cg.GAUGE_HAAR, shp, seed=W.gauge_seed, G_host=None, G_dev=Gd)
    G_orc = O.gauge_make(O.GAUGE_HAAR, W.L, W.H, W.d, W.g, seed=W.gauge_seed)
    out = {}
    for s in (0, 1):
        Xh = synth.kv_tensor(W, s)
        X = torch.from_numpy(Xh.view(np.int16)).view(torch.bfloat16).cuda()
        cache = cg.Cache(codec, s, W.L, W.B, W.H, W.T, W.d)
        err = torch.zeros(1, dtype=torch.int32, device="cuda")
        cg.kv_encode(s, X, Gd, shp, codec, cache, err_flag=err)
        Y = torch.empty_like(X)
        cg.kv_decode(s, cache, Gd, shp, codec, 0, Y, err_flag=err)
        torch.cuda.synchronize()
        assert int(err.item()) == 0
        out[s] = (Xh, X, cache, Y)
    return shp, codec, G_orc, out


def _rows(cache: cg.Cache, oc: O.Codec, s: int, l: int, h: int, t0: int, t1: int) -> dict:
    """The cache rows [t0, t1) of slice (l, 0, h) as a one-slice oracle-layout cache."""
    nc = W.d * W.bits // 8
    nbk = W.d // W.block_c
    slice_ = (l * W.B + 0) * W.H + h
    codes = cache.codes[: W.L * W.B * W.H * W.T * nc].view(W.L * W.B * W.H, W.T, nc)
    side = cache.side[: W.L * W.B * W.H * W.T * nbk * 4].view(torch.int16).view(W.L * W.B * W.H, W.T, nbk, 2)
    c = codes[slice_, t0:t1].cpu().numpy().reshape(1, 1, 1, t1 - t0, nc)
    sd = side[slice_, t0:t1].cpu().numpy().view(np.uint16).reshape(1, 1, 1, t1 - t0, nbk, 2)
    return {"codes": np.ascontiguousarray(c), "side": np.ascontiguousarray(sd), "residual": None}


@pytest.mark.parametrize("s", [0, 1])
def test_sampled_codes_match_oracle(full, s):
    _, _, G_orc, out = full
    Xh, _, cache, _ = out[s]
    oc = O.Codec(backend=O.BLOCK_UNIFORM, bits=W.bits, block_c=W.block_c)
    for l, h in SLICES:
        Gs = np.ascontiguousarray(G_orc[l:l + 1, :, h:h + 1])
        for t0, t1 in WINDOWS:
            Xs = np.ascontiguousarray(Xh[l:l + 1, :, h:h + 1, t0:t1])
            orc, flags = O.kv_encode(oc, s, Xs, Gs, T_cap=t1 - t0)
            assert flags == 0
            zo, _ = O.kv_encode(O.Codec(backend=O.PASSTHROUGH), s, Xs, Gs, T_cap=t1 - t0)
            check_fused_codes(_rows(cache, oc, s, l, h, t0, t1), orc, zo["codes"], oc, s, W.d, t1 - t0)


@pytest.mark.parametrize("s", [0, 1])
def test_sampled_decoder_rows_match_oracle(full, s):
    _, _, G_orc, out = full
    _, _, cache, Y = out[s]
    oc = O.Codec(backend=O.BLOCK_UNIFORM, bits=W.bits, block_c=W.block_c)
    for l, h in SLICES:
        Gs = np.ascontiguousarray(G_orc[l:l + 1, :, h:h + 1])
        for t0, t1 in WINDOWS:
            rows = _rows(cache, oc, s, l, h, t0, t1)
            ref = O.kv_decode(oc, s, Gs, rows, 0, t1 - t0, out_bf16=False)
            got = Y[l:l + 1, :, h:h + 1, t0:t1].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
            check_bf16_within_ulp(ref, got, W.g)


@pytest.mark.parametrize("s", [0, 1])
def test_every_vector_within_quantiser_bound(full, s):
    _, _, _, out = full
    _, X, cache, Y = out[s]
    nbk = W.d // W.block_c
    side = cache.side[: W.L * W.B * W.H * W.T * nbk * 4].view(torch.float16).view(W.L, W.B, W.H, W.T, nbk, 2)
    for l in range(W.L):
        x = X[l].float()
        y = Y[l].float()
        sc = side[l, ..., 1].float()                                  # [B][H][T][nbk]
        err2 = ((x - y) ** 2).view(*x.shape[:-1], W.d // W.g, W.g).sum(-1)        # per group
        bound2 = (W.block_c * (sc / 2) ** 2).view(*sc.shape[:-1], W.d // W.g, -1).sum(-1)
        xn2 = (x * x).view(*x.shape[:-1], W.d // W.g, W.g).sum(-1)
        yn2 = (y * y).view(*y.shape[:-1], W.d // W.g, W.g).sum(-1)
        # bf16 rounding of xhat (half an ulp: 2^-9 relative) and the gauge tolerance
        slack = (torch.sqrt(bound2) * (1 + 1e-4) + 2.0 ** -9 * torch.sqrt(yn2) + 1e-5 * torch.sqrt(xn2)) ** 2
        bad = err2 > slack
        assert not bool(bad.any()), f"layer {l}: {int(bad.sum())} token groups exceed the quantiser bound"
