"""GPU parity of the zfp-style fixed-rate backend (through the C ABI) against the oracle.

  * coder alone (identity gauge, binary32 input, so z = x exactly): the GPU's blocks equal the
    oracle's byte for byte, and the GPU decoder returns the oracle's decoded values bit for bit;
  * with a Haar gauge: the decoder fed the oracle's cache meets the decoder criteria of the other
    backends (per group 1e-5 in binary32, one bf16 ulp plus 1e-5 of the group in bf16).  The
    fused encoder splits into its two stages: its z (read back through the error-free backend,
    which runs the same matrix-core chain) is within the gauge tolerance of the oracle's z, and
    its blocks equal, byte for byte, the oracle's coder applied to that z.  The coder is a
    deterministic function of z (section 4.3: the backend codes Z), so no block may differ."""
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


def _gpu_z(X, s, Gd, shp, T_cap):
    """The GPU's z of X through the error-free backend: binary32 [L][B][H][T][d]."""
    L_, B, H, T, d = X.shape
    oc = O.Codec(backend=O.PASSTHROUGH)
    dev = _encode_gpu(X, s, Gd, shp, oc, T_cap)
    return cache_to_host(dev, oc, s)["codes"][:, :, :, :T].copy()


def _check_fused_blocks(got_codes, X, s, G, z_gpu, oc, g):
    """Fused-encoder criterion: z within the gauge tolerance of the oracle's, blocks equal to the
    oracle's coder applied to the GPU's z (identity gauge on binary32 input)."""
    L_, B, H, T, d = X.shape
    z_orc = O.kv_encode(O.Codec(backend=O.PASSTHROUGH), s, X, G, T_cap=T)[0]["codes"][:, :, :, :T]
    assert group_rel_err(z_orc, z_gpu, g) <= GAUGE_TOL
    I = O.gauge_make(O.GAUGE_IDENTITY, L_, H, d, g)
    ref, flags = O.kv_encode(oc, s, np.ascontiguousarray(z_gpu, dtype=np.float32), I, T_cap=T)
    assert flags == 0
    np.testing.assert_array_equal(got_codes, ref["codes"])


@pytest.mark.parametrize("rate", [2, 3, 4, 6, 8])
@pytest.mark.parametrize("g", [32, 128])
def test_fused_with_gauge(rate, g):
    T = 132
    w = synth.Workload("z", L=2, B=1, H=2, T=T, d=128, dtype="bf16", g=g, backend="bu", bits=4, data_seed=0x2FA)
    G, Gd, shp = _gauge(O.GAUGE_HAAR, 2, 2, 128, g)
    oc = O.Codec(backend=O.ZFP, bits=rate)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    for s in (0, 1):
        X = synth.kv_tensor(w, s)
        orc, flags = O.kv_encode(oc, s, X, G, T_cap=T)
        assert flags == 0
        dev = _encode_gpu(X, s, Gd, shp, oc, T, err=err)
        _check_fused_blocks(cache_to_host(dev, oc, s)["codes"], X, s, G, _gpu_z(X, s, Gd, shp, T), oc, g)
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
    (layer, head) slices under the fused criterion above (the GPU's z from the error-free backend
    over the whole tensor), the decoder on those windows of the GPU's cache against the oracle's
    decode of the same blocks, and every decoded value finite."""
    W = synth.WORKLOADS["llama8b"]
    shp = cg.shape(W.L, W.H, W.d, W.g)
    Gd = cg.alloc_gauge(shp)
    cg.gauge_make(cg.GAUGE_HAAR, shp, seed=W.gauge_seed, G_host=None, G_dev=Gd)
    G = O.gauge_make(O.GAUGE_HAAR, W.L, W.H, W.d, W.g, seed=W.gauge_seed)
    oc = O.Codec(backend=O.ZFP, bits=4)
    Xh = synth.kv_tensor(W, 0)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    dev = _encode_gpu(Xh, 0, Gd, shp, oc, W.T, err=err)
    assert int(err.item()) == 0
    Y = torch.empty((W.L, W.B, W.H, W.T, W.d), dtype=torch.bfloat16, device="cuda")
    cg.kv_decode(0, dev, Gd, shp, to_cg(oc), 0, Y)
    torch.cuda.synchronize()
    assert torch.isfinite(Y.float()).all()
    pdev = cg.Cache(cg.Codec(cg.PASSTHROUGH), 0, W.L, W.B, W.H, W.T, W.d)
    cg.kv_encode(0, x_dev(Xh), Gd, shp, cg.Codec(cg.PASSTHROUGH), pdev)
    torch.cuda.synchronize()
    nz = W.L * W.B * W.H * W.T * W.d
    zall = pdev.codes[: 4 * nz].view(torch.float32).view(W.L, W.B, W.H, W.T, W.d)
    nblk = W.d // 4
    codes = dev.codes[: W.L * W.B * W.H * (W.T // 4) * nblk * 8].view(W.L * W.B * W.H, W.T // 4, nblk, 8)
    for l, h in ((0, 0), (13, 5), (31, 7)):
        for t0 in (0, 4096, W.T - 64):
            Xs = np.ascontiguousarray(Xh[l:l + 1, :, h:h + 1, t0:t0 + 64])
            Gs = np.ascontiguousarray(G[l:l + 1, :, h:h + 1])
            zs = zall[l:l + 1, :, h:h + 1, t0:t0 + 64].cpu().numpy()
            got = codes[(l * W.B) * W.H + h, t0 // 4:(t0 + 64) // 4].cpu().numpy().reshape(1, 1, 1, 16, nblk, 8)
            _check_fused_blocks(got, Xs, 0, Gs, zs, oc, W.g)
            ref = O.kv_decode(oc, 0, Gs, {"codes": got, "side": None, "residual": None}, 0, 64, out_bf16=False)
            check_bf16_within_ulp(ref, Y[l:l + 1, :, h:h + 1, t0:t0 + 64].view(torch.int16).cpu().numpy().view(np.uint16), W.g)
