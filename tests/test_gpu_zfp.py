"""GPU parity of the zfp-style fixed-rate backend (general kernels, through the C ABI) against
the oracle.

  * coder alone (identity gauge, binary32 input, so z = x exactly): the GPU's blocks equal the
    oracle's byte for byte, and the GPU decoder returns the oracle's decoded values bit for bit;
  * with a Haar gauge: the decoder fed the oracle's cache meets the decoder criteria of the other
    backends (per group 1e-5 in binary32, one bf16 ulp plus 1e-5 of the group in bf16); the
    fused encoder's z differs from the oracle's by the binary32 gauge rounding, so a block's
    code may differ where a coded bit sits on that rounding: at most 2% of the blocks differ,
    and a differing block decodes within twice the oracle's own error on that block (plus 2^-20
    of its largest value)."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2607_20538_amd import codec as cg
from paper_2607_20538_amd import synth

from _parity import cache_to_dev, cache_to_host, check_bf16_within_ulp, group_rel_err, to_cg, x_dev, GAUGE_TOL

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cg.lib()


def _gauge(kind, L, H, d, g, seed=17):
    G = O.gauge_make(kind, L, H, d, g, seed=seed)
    shp = cg.shape(L, H, d, g)
    Gd = cg.alloc_gauge(shp)
    cg.gauge_make(cg.GAUGE_USER, shp, params=G, G_host=None, G_dev=Gd)
    return G, Gd, shp


def _encode_gpu(X, s, Gd, shp, oc, T_cap, t0=0, err=None):
    L_, B, H, T, d = X.shape
    dev = cg.Cache(to_cg(oc), s, L_, B, H, T_cap, d)
    cg.kv_encode(s, x_dev(X), Gd, shp, to_cg(oc), dev, t0=t0, err_flag=err)
    torch.cuda.synchronize()
    return dev


def _decode_gpu(dev, s, Gd, shp, oc, t0, T, dtype=torch.bfloat16):
    Y = torch.zeros((dev.L, dev.B, dev.H, T, dev.d), dtype=dtype, device="cuda")
    cg.kv_decode(s, dev, Gd, shp, to_cg(oc), t0, Y)
    torch.cuda.synchronize()
    if dtype == torch.bfloat16:
        return Y.view(torch.int16).cpu().numpy().view(np.uint16)
    return Y.cpu().numpy()


@pytest.mark.parametrize("rate", [2, 3, 4, 6, 8])
@pytest.mark.parametrize("d", [128, 64])
def test_coder_alone_is_bit_exact(rate, d):
    T = 36
    w = synth.Workload("z", L=1, B=2, H=2, T=T, d=d, dtype="f32", g=16, backend="bu", bits=4, data_seed=0x2F9)
    G, Gd, shp = _gauge(O.GAUGE_IDENTITY, 1, 2, d, 16)
    oc = O.Codec(backend=O.ZFP, bits=rate)
    for s in (0, 1):
        X = synth.kv_tensor(w, s)
        orc, flags = O.kv_encode(oc, s, X, G, T_cap=T)
        assert flags == 0
        dev = _encode_gpu(X, s, Gd, shp, oc, T)
        np.testing.assert_array_equal(cache_to_host(dev, oc, s)["codes"], orc["codes"])
        ref = O.kv_decode(oc, s, G, orc, 0, T, out_bf16=False)
        np.testing.assert_array_equal(_decode_gpu(dev, s, Gd, shp, oc, 0, T, torch.float32), ref)
        # a sub-range starting on a block row
        np.testing.assert_array_equal(_decode_gpu(dev, s, Gd, shp, oc, 8, 24, torch.float32), ref[:, :, :, 8:32])


@pytest.mark.parametrize("rate", [3, 4, 8])
@pytest.mark.parametrize("g", [32, 128])
def test_fused_with_gauge(rate, g):
    T = 132
    w = synth.Workload("z", L=2, B=1, H=2, T=T, d=128, dtype="bf16", g=g, backend="bu", bits=4, data_seed=0x2FA)
    G, Gd, shp = _gauge(O.GAUGE_HAAR, 2, 2, 128, g)
    I = O.gauge_make(O.GAUGE_IDENTITY, 2, 2, 128, g)
    oc = O.Codec(backend=O.ZFP, bits=rate)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    for s in (0, 1):
        X = synth.kv_tensor(w, s)
        orc, flags = O.kv_encode(oc, s, X, G, T_cap=T)
        assert flags == 0
        dev = _encode_gpu(X, s, Gd, shp, oc, T, err=err)
        got = cache_to_host(dev, oc, s)
        # blocks: 4 tokens x 4 channels, 2 rate bytes each
        diff = (got["codes"] != orc["codes"]).any(axis=-1)
        assert diff.mean() <= 0.02, diff.mean()
        z = O.kv_encode(O.Codec(backend=O.PASSTHROUGH), s, X, G, T_cap=T)[0]["codes"]
        zo = O.kv_decode(oc, s, I, orc, 0, T, out_bf16=False)      # identity: zhat itself
        zg = O.kv_decode(oc, s, I, got, 0, T, out_bf16=False)
        blk = lambda a: a.reshape(2, 1, 2, T // 4, 4, 32, 4).transpose(0, 1, 2, 3, 5, 4, 6).reshape(2, 1, 2, T // 4, 32, 16)
        e_orc = np.abs(blk(zo) - blk(z)).max(-1)
        d_gpu = np.abs(blk(zg) - blk(zo)).max(-1)
        scale = np.abs(blk(z)).max(-1)
        assert (d_gpu <= 2 * e_orc + scale * 2.0 ** -20).all()
        # decoder on the oracle's cache
        ddev = cache_to_dev(orc, oc, s, 2, 1, 2, T, 128)
        ref = O.kv_decode(oc, s, G, orc, 0, T, out_bf16=False)
        assert group_rel_err(ref, _decode_gpu(ddev, s, Gd, shp, oc, 0, T, torch.float32), g) <= GAUGE_TOL
        check_bf16_within_ulp(ref, _decode_gpu(ddev, s, Gd, shp, oc, 0, T), g)
    assert int(err.item()) == 0


def test_nonfinite_input_flags_and_codes_a_zero_block():
    T = 8
    w = synth.Workload("z", L=1, B=1, H=1, T=T, d=64, dtype="f32", g=16, backend="bu", bits=4, data_seed=3)
    G, Gd, shp = _gauge(O.GAUGE_IDENTITY, 1, 1, 64, 16)
    oc = O.Codec(backend=O.ZFP, bits=4)
    X = synth.kv_tensor(w, 0)
    X[0, 0, 0, 5, 9] = np.nan
    orc, flags = O.kv_encode(oc, 0, X, G, T_cap=T)
    assert flags == O.FLAG_NONFINITE
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    dev = _encode_gpu(X, 0, Gd, shp, oc, T, err=err)
    assert int(err.item()) & cg.CG_FLAG_NONFINITE
    np.testing.assert_array_equal(cache_to_host(dev, oc, 0)["codes"], orc["codes"])


def test_full_size_sampled():
    """Llama-3-8B-shaped K at rate 4 (32 layers, 8 heads, 8192 tokens, bf16, Haar g = 128) in one
    kv_encode call, as bench.py --workload zfp times it: sampled 64-token windows of several
    (layer, head) slices against the oracle under the fused criterion above, and every decoded
    value finite."""
    W = synth.WORKLOADS["llama8b"]
    shp = cg.shape(W.L, W.H, W.d, W.g)
    Gd = cg.alloc_gauge(shp)
    cg.gauge_make(cg.GAUGE_HAAR, shp, seed=W.gauge_seed, G_host=None, G_dev=Gd)
    G = O.gauge_make(O.GAUGE_HAAR, W.L, W.H, W.d, W.g, seed=W.gauge_seed)
    I = O.gauge_make(O.GAUGE_IDENTITY, 1, 1, W.d, W.g)
    oc = O.Codec(backend=O.ZFP, bits=4)
    Xh = synth.kv_tensor(W, 0)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    dev = _encode_gpu(Xh, 0, Gd, shp, oc, W.T, err=err)
    assert int(err.item()) == 0
    Y = torch.empty((W.L, W.B, W.H, W.T, W.d), dtype=torch.bfloat16, device="cuda")
    cg.kv_decode(0, dev, Gd, shp, to_cg(oc), 0, Y)
    torch.cuda.synchronize()
    assert torch.isfinite(Y.float()).all()
    nblk = W.d // 4
    codes = dev.codes[: W.L * W.B * W.H * (W.T // 4) * nblk * 8].view(W.L * W.B * W.H, W.T // 4, nblk, 8)
    for l, h in ((0, 0), (13, 5), (31, 7)):
        for t0 in (0, 4096, W.T - 64):
            Xs = np.ascontiguousarray(Xh[l:l + 1, :, h:h + 1, t0:t0 + 64])
            Gs = np.ascontiguousarray(G[l:l + 1, :, h:h + 1])
            orc, _ = O.kv_encode(oc, 0, Xs, Gs, T_cap=64)
            got = {"codes": codes[(l * W.B) * W.H + h, t0 // 4:(t0 + 64) // 4].cpu().numpy().reshape(1, 1, 1, 16, nblk, 8),
                   "side": None, "residual": None}
            assert (got["codes"] != orc["codes"]).any(axis=-1).mean() <= 0.02
            z = O.kv_encode(O.Codec(backend=O.PASSTHROUGH), 0, Xs, Gs, T_cap=64)[0]["codes"]
            zo = O.kv_decode(oc, 0, I, orc, 0, 64, out_bf16=False)
            zg = O.kv_decode(oc, 0, I, got, 0, 64, out_bf16=False)
            blk = lambda a: a.reshape(16, 4, nblk, 4).transpose(0, 2, 1, 3).reshape(16, nblk, 16)
            e_orc = np.abs(blk(zo) - blk(z)).max(-1)
            d_gpu = np.abs(blk(zg) - blk(zo)).max(-1)
            assert (d_gpu <= 2 * e_orc + np.abs(blk(z)).max(-1) * 2.0 ** -20).all()
