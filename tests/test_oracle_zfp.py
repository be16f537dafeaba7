"""Pins of the oracle's zfp-style fixed-rate codec (the paper's zfp backend, section 4.3, written
from zfp's published algorithm) against what the algorithm's definition and the mathematics fix:
the published 4-point transform matrix, negabinary digits, the sequency order, the exact fixed
rate (4.000 bits/value at rate 4, section 4.4's zfp-4 row), the embedded (prefix) property of
the bit-plane stream, exactness at full precision and monotone error in the rate."""
import numpy as np
import pytest

import oracle as O
from paper_2607_20538_amd import synth

A = np.array([[4, 4, 4, 4], [5, 1, -1, -5], [-4, 4, 4, -4], [-2, 6, -6, 2]]) / 16.0


def test_transform_is_the_published_matrix():
    """The lifting computes A v up to the rounding of its halvings (a few units), and the
    inverse lifting returns v from A v up to the same order."""
    rng = np.random.default_rng(1)
    for _ in range(2000):
        v = rng.integers(-(1 << 29), 1 << 29, 4)
        f = O.zfp_fwd4(v)
        assert np.abs(f - A @ v).max() <= 2.0
        back = O.zfp_inv4(f)
        assert np.abs(back - v).max() <= 8
    # basis vectors of a large scale recover the matrix columns
    for k in range(4):
        e = np.zeros(4, dtype=np.int64)
        e[k] = 1 << 20
        np.testing.assert_allclose(O.zfp_fwd4(e) / (1 << 20), A[:, k], atol=4.0 / (1 << 20))


def test_negabinary_digits():
    """u's bits are the base -2 digits of i: i = sum_k bit_k(u) (-2)^k."""
    rng = np.random.default_rng(2)
    for i in list(range(-40, 41)) + list(rng.integers(-(1 << 30), 1 << 30, 200)):
        u = O.negabinary(int(i))
        assert sum(((u >> k) & 1) * (-2) ** k for k in range(32)) == i
        assert O.from_negabinary(u) == i


def test_sequency_order():
    order = O.zfp_order()
    assert sorted(order.tolist()) == list(range(16))
    deg = [(k % 4) + (k // 4) for k in order]
    assert deg == sorted(deg) and order[0] == 0 and order[-1] == 15


@pytest.mark.parametrize("rate", [2, 3, 4, 6, 8])
def test_fixed_rate_is_exact(rate):
    """Every block is 16 rate bits, so a cache holds exactly rate bits per value (the paper's
    zfp-4 row: 4.000 bits/value at rate 4)."""
    codec = O.Codec(backend=O.ZFP, bits=rate)
    lay = O.cache_layout(codec, 0, 2, 3, 4, 64, 128)
    nbytes = int(np.prod(lay["codes"][0]))
    assert lay["side"] is None and lay["residual"] is None
    assert nbytes * 8 / (2 * 3 * 4 * 64 * 128) == rate
    v = np.random.default_rng(3).standard_normal(16).astype(np.float32)
    code, flags = O.zfp_encode_block(v, rate)
    assert code.size == 2 * rate and flags == 0


def test_stream_is_embedded():
    """A rate-r block is the first 16 r bits of the rate-8 block: the stream can be cut anywhere
    (embedded coding), so fixed-rate truncation keeps the most significant information."""
    rng = np.random.default_rng(4)
    for _ in range(200):
        v = (rng.standard_normal(16) * rng.choice([1e-3, 1.0, 50.0], 16)).astype(np.float32)
        full, _ = O.zfp_encode_block(v, 8)
        for r in (2, 3, 4, 6):
            part, _ = O.zfp_encode_block(v, r)
            np.testing.assert_array_equal(part, full[: 2 * r])


def test_error_falls_with_rate_and_vanishes_at_full_precision():
    rng = np.random.default_rng(5)
    V = (rng.standard_normal((300, 16)) * np.exp(rng.standard_normal((300, 1)))).astype(np.float32)
    errs = []
    for r in (2, 3, 4, 6, 8, 16):
        e = max(np.abs(O.zfp_decode_block(O.zfp_encode_block(v, r)[0], r) - v).max() / np.abs(v).max() for v in V)
        errs.append(e)
    assert all(a >= b for a, b in zip(errs, errs[1:])), errs
    # the transform decorrelates: a block that is linear in channel and token has three nonzero
    # coefficients, so rate 4 codes it to about 2^-11 of its largest value and rate 6 to 2^-19
    i = np.arange(4)
    for a, b, c in rng.standard_normal((100, 3)):
        v = (a + b * i[None, :] + c * i[:, None]).astype(np.float32).reshape(16)
        for r, bound in ((4, 1e-3), (6, 1e-5)):
            out = O.zfp_decode_block(O.zfp_encode_block(v, r)[0], r)
            assert np.abs(out - v).max() <= bound * np.abs(v).max()
    # rate 32 codes every plane: the error is that of the 30-bit fixed point and the transform's
    # halvings (a few units of 2^(e - 30)), far below binary32 rounding of the largest value
    for v in V[:50]:
        e = np.frexp(np.abs(v).max())[1]
        out = O.zfp_decode_block(O.zfp_encode_block(v, 32)[0], 32)
        assert np.abs(out - v).max() <= 16 * 2.0 ** (e - 30) + np.abs(v).max() * 2.0 ** -24


def test_special_blocks():
    # all zero: one 0 bit, decoded as zeros
    code, _ = O.zfp_encode_block(np.zeros(16, np.float32), 4)
    assert not code.any()
    assert not O.zfp_decode_block(code, 4).any()
    # a constant block has only the mean coefficient: at rate 8 every plane fits, exact
    for c in (1.0, -3.25, 1e-30, 6.5e4):
        v = np.full(16, c, np.float32)
        np.testing.assert_array_equal(O.zfp_decode_block(O.zfp_encode_block(v, 8)[0], 8), v)
    # non-finite values flag and code a zero block
    v = np.ones(16, np.float32)
    v[3] = np.inf
    code, flags = O.zfp_encode_block(v, 4)
    assert flags == O.FLAG_NONFINITE and not code.any()


def test_cache_round_trip_with_gauge():
    """Whole-cache encode / decode: the zfp-style cache decodes within the block error of the
    same data coded without the gauge (identity gauge: the codec alone), and an orthogonal gauge
    keeps the per-token error norm of z (the decode applies G^T)."""
    w = synth.Workload("t", L=1, B=1, H=2, T=64, d=64, dtype="f32", g=16, backend="bu", bits=4, data_seed=7)
    X = synth.kv_tensor(w, 1)
    for kind in (O.GAUGE_IDENTITY, O.GAUGE_HAAR):
        G = O.gauge_make(kind, 1, 2, 64, 16, seed=8)
        codec = O.Codec(backend=O.ZFP, bits=8)
        cache, flags = O.kv_encode(codec, 1, X, G, T_cap=64)
        assert flags == 0
        Xh = O.kv_decode(codec, 1, G, cache, 0, 64, out_bf16=False)
        rel = np.linalg.norm(Xh - X) / np.linalg.norm(X)
        assert rel < 2e-2, (kind, rel)
    # t0 and token counts must be multiples of 4
    with pytest.raises(ValueError):
        O.kv_encode(O.Codec(backend=O.ZFP, bits=4), 1, X[:, :, :, :6], G, T_cap=64)
