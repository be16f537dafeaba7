"""Pins of the oracle's quantisation backends (paper section 4.3: block-uniform ranges and
KIVI-style per-channel key / per-token value ranges, same bit settings) and of the rolling
compressed-history path (section 4.4), against bounds, brute force, numpy's bit unpacking,
structural equivalences between the backends and closed-form byte counts."""
import itertools

import numpy as np
import pytest

import oracle as O
from paper_2607_20538_amd import synth

BITS = [2, 3, 4, 6, 8]


def _f16(bits):
    return O.f16_value(bits)


def _blocks(rng, n, count):
    out = []
    for k in range(count):
        kind = k % 6
        if kind == 0:
            z = rng.standard_normal(n)
        elif kind == 1:
            z = rng.standard_normal(n) * 20.0 + 5.0
        elif kind == 2:
            z = rng.standard_normal(n) * 1e-3
        elif kind == 3:
            z = np.where(rng.random(n) < 0.1, 40.0, 1.0) * rng.standard_normal(n)
        elif kind == 4:
            z = rng.uniform(100.0, 101.0, n)
        else:
            z = -np.abs(rng.standard_normal(n)) * 300.0
        out.append(z.astype(np.float32))
    return out


@pytest.mark.parametrize("bits", BITS)
@pytest.mark.parametrize("n", [16, 32, 64])
def test_quantiser_error_bound_and_side_info(bits, n):
    """|z - zhat| <= sc_h / 2 (up to binary32 rounding of the reconstruction), codes in range,
    mn_h is the largest binary16 <= min and the grid covers [min, max]."""
    rng = np.random.default_rng(bits * 100 + n)
    qmax = (1 << bits) - 1
    for z in _blocks(rng, n, 60):
        q, mnb, scb, flags = O.quantize_block(z, bits)
        assert flags == 0
        assert q.max() <= qmax
        mn, sc = _f16(mnb), _f16(scb)
        assert mn <= z.min()
        assert np.float16(mn) == mn and np.float16(sc) == sc
        nxt = float(np.nextafter(np.float16(mn), np.float16(np.inf), dtype=np.float16))
        assert nxt > z.min()
        assert sc >= 0 and not (mn == 0 and np.signbit(mn))
        zh = O.dequantize_block(q, mnb, scb)
        bound = sc / 2 * (1 + 2.0 ** -20) + 2.0 ** -22 * np.abs(z).max()
        assert np.abs(z.astype(np.float64) - zh).max() <= bound


@pytest.mark.parametrize("bits", BITS)
def test_constant_block(bits):
    for v in (0.0, 1.5, -3.25, 1000.0, 0.1):
        z = np.full(32, v, np.float32)
        q, mnb, scb, _ = O.quantize_block(z, bits)
        assert np.all(q == q[0])
        zh = O.dequantize_block(q, mnb, scb)
        if float(np.float16(v)) == v:   # min representable in binary16: code 0, exact
            assert np.all(q == 0)
            assert _f16(scb) == 0.0
            np.testing.assert_array_equal(zh, z)
        else:
            assert np.abs(zh - z).max() <= _f16(scb) / 2 * (1 + 2.0 ** -20)


@pytest.mark.parametrize("n,bits", list(itertools.product([2, 4, 8], [2, 3])))
def test_quantiser_brute_force_nearest_code(n, bits):
    """Each code is the nearest grid point mn_h + q sc_h over all 2^b codes, except inside
    a rounding tie where both neighbours are equally near."""
    rng = np.random.default_rng(n * 7 + bits)
    for z in _blocks(rng, n, 300):
        q, mnb, scb, _ = O.quantize_block(z, bits)
        mn, sc = np.float32(_f16(mnb)), np.float32(_f16(scb))
        grid = mn.astype(np.float64) + np.arange(1 << bits) * sc.astype(np.float64)
        for i in range(n):
            dist = np.abs(grid - z[i])
            best = dist.min()
            if dist[q[i]] != best:
                t = (np.float32(z[i] - mn) * (np.float32(1.0) / sc)) if sc else 0.0
                assert abs(abs(t - np.floor(t)) - 0.5) < 1e-5, (z, i, q[i], dist)


def test_quantiser_grid_aligned_block_is_idempotent():
    for bits in BITS:
        qmax = (1 << bits) - 1
        mn, sc = np.float32(-2.0), np.float32(0.125)
        q0 = np.arange(qmax + 1) % (qmax + 1)
        z = (mn + q0.astype(np.float32) * sc).astype(np.float32)
        q, mnb, scb, _ = O.quantize_block(z, bits)
        np.testing.assert_array_equal(q, q0)
        np.testing.assert_array_equal(O.dequantize_block(q, mnb, scb), z)


def test_quantiser_flags_nonfinite_and_overflow():
    z = np.ones(16, np.float32)
    z[3] = np.inf
    assert O.quantize_block(z, 4)[3] & O.FLAG_NONFINITE
    z = np.array([-70000.0] + [0.0] * 15, np.float32)
    assert O.quantize_block(z, 4)[3] & O.FLAG_SIDE_OVERFLOW
    z = np.array([0.0] * 15 + [2e6], np.float32)
    assert O.quantize_block(z, 4)[3] & O.FLAG_SIDE_OVERFLOW
    assert O.quantize_block(np.array([0.0] * 15 + [6e4], np.float32), 4)[3] == 0


@pytest.mark.parametrize("bits", BITS)
def test_pack_order_matches_numpy_little_endian_bits(bits):
    rng = np.random.default_rng(bits)
    patterns = [rng.integers(0, 1 << bits, 64), np.zeros(64, int), np.full(64, (1 << bits) - 1),
                np.arange(64) % 2 * ((1 << bits) - 1)]
    for codes in patterns:
        codes = codes.astype(np.uint8)
        packed = O.pack_codes(codes, bits)
        assert packed.size == 64 * bits // 8
        stream = np.unpackbits(packed, bitorder="little")
        rebuilt = np.array([sum(int(stream[i * bits + k]) << k for k in range(bits)) for i in range(64)])
        np.testing.assert_array_equal(rebuilt, codes)
        np.testing.assert_array_equal(O.unpack_codes(packed, 64, bits), codes)


def _tensor(T, d=128, L=1, B=2, H=2, seed=0xABC, dtype="bf16"):
    w = synth.Workload("t", L=L, B=B, H=H, T=T, d=d, dtype=dtype, g=32, backend="bu", bits=4, data_seed=seed)
    return w, synth.kv_tensor(w, 0), synth.kv_tensor(w, 1)


def test_block_uniform_row_layout():
    """A BU code row holds the d/n blocks of one token in channel order, each its own
    LSB-first stream; side rows hold (min, scale) per block."""
    w, K, _ = _tensor(8, d=128)
    G = O.gauge_make(O.GAUGE_HAAR, 1, 2, 128, 32, seed=1)
    codec = O.Codec(backend=O.BLOCK_UNIFORM, bits=3, block_c=32)
    cache, flags = O.kv_encode(codec, 0, K, G, T_cap=8)
    assert flags == 0
    for (b, h, t) in [(0, 0, 0), (1, 1, 7), (0, 1, 3)]:
        x = np.array([O.bf16_to_f32(v) for v in K[0, b, h, t]], np.float32)
        z = O.gauge_apply(G[0, 0, h], x)
        for k in range(4):
            q, mnb, scb, _ = O.quantize_block(z[32 * k:32 * k + 32], 3)
            np.testing.assert_array_equal(cache["codes"][0, b, h, t, 12 * k:12 * k + 12], O.pack_codes(q, 3))
            assert tuple(cache["side"][0, b, h, t, k]) == (mnb, scb)


def test_kivi_values_equal_block_uniform_with_value_group():
    w, K, V = _tensor(256 + 40)
    T = V.shape[3]
    G = O.gauge_make(O.GAUGE_HAAR, 1, 2, 128, 32, seed=4)
    kivi = O.Codec(backend=O.KIVI, bits=3, key_tokens=32, val_channels=64, residual=128)
    bu = O.Codec(backend=O.BLOCK_UNIFORM, bits=3, block_c=64)
    ck, _ = O.kv_encode(kivi, 1, V, G, T_cap=320)
    cb, _ = O.kv_encode(bu, 1, V, G, T_cap=320)
    tq = O.kivi_tq(T, kivi)
    assert tq == 160
    np.testing.assert_array_equal(ck["codes"][:, :, :, :tq], cb["codes"][:, :, :, :tq])
    np.testing.assert_array_equal(ck["side"][:, :, :, :tq], cb["side"][:, :, :, :tq])
    assert not ck["codes"][:, :, :, tq:].any()


def test_kivi_keys_equal_block_uniform_on_transposed_tile():
    w, K, _ = _tensor(256)
    G = O.gauge_make(O.GAUGE_HAAR, 1, 2, 128, 32, seed=4)
    kivi = O.Codec(backend=O.KIVI, bits=3, key_tokens=32, val_channels=64, residual=128)
    ck, _ = O.kv_encode(kivi, 0, K, G, T_cap=256)
    assert O.kivi_tq(256, kivi) == 128
    b, h = 1, 0
    for grp in range(4):
        Z = np.stack([O.gauge_apply(G[0, 0, h], np.array([O.bf16_to_f32(v) for v in K[0, b, h, 32 * grp + u]],
                                                          np.float32)) for u in range(32)])
        for c in (0, 5, 127):
            q, mnb, scb, _ = O.quantize_block(Z[:, c], 3)
            np.testing.assert_array_equal(ck["codes"][0, b, h, grp, c], O.pack_codes(q, 3))
            assert tuple(ck["side"][0, b, h, grp, c]) == (mnb, scb)


def test_kivi_short_cache_is_all_window_and_decodes_bit_exact():
    w, K, V = _tensor(100)
    G = O.gauge_make(O.GAUGE_HAAR, 1, 2, 128, 32, seed=4)
    kivi = O.Codec(backend=O.KIVI, bits=3)
    for s, X in ((0, K), (1, V)):
        c, _ = O.kv_encode(kivi, s, X, G, T_cap=128)
        assert not c["codes"].any()
        Xh = O.kv_decode(kivi, s, G, c, 0, 100, lens=[100, 100])
        np.testing.assert_array_equal(Xh, X)


@pytest.mark.parametrize("backend", [O.BLOCK_UNIFORM, O.KIVI, O.PASSTHROUGH])
def test_rolling_append_equals_batch_encode(backend):
    """Appending tokens one at a time (section 4.4 rolling history) leaves the same cache
    and decodes the same history as one batch encode of all tokens."""
    T0, steps = 150, 50
    w, K, V = _tensor(T0 + steps, B=2)
    G = O.gauge_make(O.GAUGE_HAAR, 1, 2, 128, 32, seed=6)
    codec = O.Codec(backend=backend, bits=4, block_c=32, residual=128)
    T_cap = 224
    for s, X in ((0, K), (1, V)):
        roll, _ = O.kv_encode(codec, s, X[:, :, :, :T0], G, T_cap=T_cap)
        for t in range(T0, T0 + steps):
            O.kv_append(codec, s, np.ascontiguousarray(X[:, :, :, t]), G, roll, [t, t])
        full, _ = O.kv_encode(codec, s, X, G, T_cap=T_cap)
        T = T0 + steps
        if backend == O.KIVI:
            tq = O.kivi_tq(T, codec)
            if s == 0:
                np.testing.assert_array_equal(roll["codes"][:, :, :, :tq // 32], full["codes"][:, :, :, :tq // 32])
                np.testing.assert_array_equal(roll["side"][:, :, :, :tq // 32], full["side"][:, :, :, :tq // 32])
            else:
                np.testing.assert_array_equal(roll["codes"][:, :, :, :tq], full["codes"][:, :, :, :tq])
                np.testing.assert_array_equal(roll["side"][:, :, :, :tq], full["side"][:, :, :, :tq])
        else:
            np.testing.assert_array_equal(roll["codes"], full["codes"])
            if backend == O.BLOCK_UNIFORM:
                np.testing.assert_array_equal(roll["side"], full["side"])
        a = O.kv_decode(codec, s, G, roll, 0, T, lens=[T, T])
        b = O.kv_decode(codec, s, G, full, 0, T, lens=[T, T])
        np.testing.assert_array_equal(a, b)


def test_bits_per_value_closed_forms():
    """Block-uniform: b + 32/n (two binary16 per block); KIVI: keys b + 32/G_k, values
    b + 32/n_v on the quantised tokens, 16 bits on the window tokens."""
    bu = lambda b, n: O.Codec(backend=O.BLOCK_UNIFORM, bits=b, block_c=n)
    assert O.bits_per_value(bu(4, 32), 256, 64) == 5.0          # tiny
    assert O.bits_per_value(bu(4, 64), 8192, 128) == 4.5        # Llama-3-8B shaped
    for b, ref in ((3, 3.5), (4, 4.5), (6, 6.5)):               # 27B sweep
        assert O.bits_per_value(bu(b, 64), 16384, 128) == ref
    kivi = O.Codec(backend=O.KIVI, bits=3, key_tokens=32, val_channels=64, residual=128)
    T, tq = 32768, 32640
    ref = (tq * (3 + 1.0) + tq * (3 + 0.5) + 2 * (T - tq) * 16) / (2 * T)
    assert abs(O.bits_per_value(kivi, T, 128) - ref) < 1e-12
    assert round(ref, 4) == 3.7979


def test_lossy_codec_error_is_bounded_per_block():
    """End to end, BU decode error in gauge space stays within the per-block half-step, so
    the bf16 output is within half a step plus bf16 rounding (the gauge is an isometry)."""
    w, K, V = _tensor(64, B=1, H=1)
    G = O.gauge_make(O.GAUGE_HAAR, 1, 1, 128, 128, seed=8)
    codec = O.Codec(backend=O.BLOCK_UNIFORM, bits=4, block_c=64)
    cache, _ = O.kv_encode(codec, 0, K, G, T_cap=64)
    Xh = O.kv_decode(codec, 0, G, cache, 0, 64, out_bf16=False)
    x = np.array([[O.bf16_to_f32(v) for v in row] for row in K[0, 0, 0]], np.float64)
    sc = np.vectorize(O.f16_value)(cache["side"][0, 0, 0, :, :, 1])
    err = np.linalg.norm(Xh[0, 0, 0] - x, axis=1)
    assert np.all(err <= np.sqrt(64 * (sc[:, 0] / 2) ** 2 + 64 * (sc[:, 1] / 2) ** 2) * (1 + 1e-5))


# ------------------------------------------------------------------------------------------
# block-uniform token-channel tiles (section 4.3: one range per T_b x d block, T_b = 16 in the
# experimental setup of section 5): the same n channels of Tb consecutive tokens share a range
# ------------------------------------------------------------------------------------------
def _tile(bits=4, n=128, bt=16):
    return O.Codec(backend=O.BLOCK_UNIFORM, bits=bits, block_c=n, block_t=bt)


def _z_rows(K, G, b, h, t0, t1, s=0):
    return np.stack([O.gauge_apply(G[0, s, h], np.array([O.bf16_to_f32(v) for v in K[0, b, h, t]], np.float32))
                     for t in range(t0, t1)])


@pytest.mark.parametrize("bits,n", [(4, 128), (3, 64), (6, 32), (2, 128)])
def test_tile_range_covers_the_whole_tile(bits, n):
    """The side information of a tile is the binary16 range of all its Tb x n gauge-space
    values (checked in numpy against the passthrough z): mn_h is the largest binary16 at or
    below the tile minimum, the grid reaches the maximum, and every token of the tile is
    within half a step of its reconstruction."""
    bt = 16
    w, K, _ = _tensor(64)
    G = O.gauge_make(O.GAUGE_HAAR, 1, 2, 128, 32, seed=11)
    codec = _tile(bits, n, bt)
    cache, flags = O.kv_encode(codec, 0, K, G, T_cap=64)
    assert flags == 0
    zpass, _ = O.kv_encode(O.Codec(backend=O.PASSTHROUGH), 0, K, G, T_cap=64)
    zh = O.kv_decode(O.Codec(backend=O.BLOCK_UNIFORM, bits=bits, block_c=n, block_t=bt), 0,
                     O.gauge_make(O.GAUGE_IDENTITY, 1, 2, 128, 32), cache, 0, 64, lens=[64, 64], out_bf16=False)
    qmax = (1 << bits) - 1
    for b in range(2):
        for h in range(2):
            for tile in range(4):
                for k in range(128 // n):
                    blk = zpass["codes"][0, b, h, bt * tile:bt * tile + bt, n * k:n * k + n].astype(np.float64)
                    mnb, scb = cache["side"][0, b, h, tile, k]
                    mn, sc = _f16(mnb), _f16(scb)
                    assert mn <= blk.min()
                    nxt = float(np.nextafter(np.float16(mn), np.float16(np.inf), dtype=np.float16))
                    assert nxt > blk.min()
                    assert mn + qmax * sc >= blk.max() * (1 - 2.0 ** -22) - 2.0 ** -22
                    rec = zh[0, b, h, bt * tile:bt * tile + bt, n * k:n * k + n].astype(np.float64)
                    assert np.abs(rec - blk).max() <= sc / 2 * (1 + 2.0 ** -20) + 2.0 ** -22 * np.abs(blk).max()


def test_tile_of_repeated_token_equals_per_token_block():
    """A tile whose Tb tokens are one vector repeated has that vector's own block range, so
    its codes and side words equal the per-token block-uniform ones."""
    w, K, _ = _tensor(4)
    Kr = np.ascontiguousarray(np.repeat(K[:, :, :, :1], 16, axis=3))
    G = O.gauge_make(O.GAUGE_HAAR, 1, 2, 128, 32, seed=12)
    for bits, n in ((4, 128), (3, 32)):
        tile, _ = O.kv_encode(_tile(bits, n, 16), 0, Kr, G, T_cap=16)
        per, _ = O.kv_encode(O.Codec(backend=O.BLOCK_UNIFORM, bits=bits, block_c=n), 0, Kr, G, T_cap=16)
        np.testing.assert_array_equal(tile["codes"], per["codes"])
        for t in range(16):
            np.testing.assert_array_equal(tile["side"][:, :, :, 0], per["side"][:, :, :, t])


def test_tile_equals_quantiser_on_the_token_channel_block():
    """A tile's codes are those of one block made of its Tb x n values, token by token, with
    each token's n codes in its own row at the block's place."""
    w, K, _ = _tensor(48)
    G = O.gauge_make(O.GAUGE_HAAR, 1, 2, 128, 32, seed=13)
    cache, _ = O.kv_encode(_tile(3, 64, 16), 0, K, G, T_cap=48)
    b, h = 1, 1
    for tile in range(3):
        Z = _z_rows(K, G, b, h, 16 * tile, 16 * tile + 16)
        for k in range(2):
            q, mnb, scb, _ = O.quantize_block(np.ascontiguousarray(Z[:, 64 * k:64 * k + 64]).reshape(-1), 3)
            assert tuple(cache["side"][0, b, h, tile, k]) == (mnb, scb)
            for u in range(16):
                np.testing.assert_array_equal(cache["codes"][0, b, h, 16 * tile + u, 24 * k:24 * k + 24],
                                              O.pack_codes(q[64 * u:64 * u + 64], 3))


def test_tile_unfinished_tokens_stay_raw():
    """Tokens past the last whole tile wait in the bf16 staging window and decode bit for bit;
    a cache shorter than one tile is all staging."""
    G = O.gauge_make(O.GAUGE_HAAR, 1, 2, 128, 32, seed=14)
    codec = _tile(4, 128, 16)
    for T in (40, 9):
        w, K, V = _tensor(T)
        for s, X in ((0, K), (1, V)):
            c, _ = O.kv_encode(codec, s, X, G, T_cap=48)
            tq = O.tile_tq(T, codec)
            assert tq == (32 if T == 40 else 0)
            assert not c["codes"][:, :, :, tq:].any()
            Xh = O.kv_decode(codec, s, G, c, 0, T, lens=[T, T])
            np.testing.assert_array_equal(Xh[:, :, :, tq:], X[:, :, :, tq:])
            for t in range(tq, T):
                np.testing.assert_array_equal(c["residual"][:, :, :, t % 16], X[:, :, :, t])


def test_tile_rolling_append_equals_batch_encode():
    """Appending tokens one at a time (staged until a tile is whole) leaves the same codes,
    side information and staging window as one batch encode, and decodes the same history."""
    T0, steps = 37, 46
    w, K, V = _tensor(T0 + steps, B=2)
    G = O.gauge_make(O.GAUGE_HAAR, 1, 2, 128, 32, seed=15)
    codec = _tile(4, 64, 16)
    T_cap, T = 96, T0 + steps
    for s, X in ((0, K), (1, V)):
        roll, _ = O.kv_encode(codec, s, np.ascontiguousarray(X[:, :, :, :T0]), G, T_cap=T_cap)
        for t in range(T0, T):
            O.kv_append(codec, s, np.ascontiguousarray(X[:, :, :, t]), G, roll, [t, t])
        full, _ = O.kv_encode(codec, s, X, G, T_cap=T_cap)
        for key in ("codes", "side"):
            np.testing.assert_array_equal(roll[key], full[key])
        for t in range(O.tile_tq(T, codec), T):   # slots of flushed tokens keep stale rows
            np.testing.assert_array_equal(roll["residual"][:, :, :, t % 16], full["residual"][:, :, :, t % 16])
        np.testing.assert_array_equal(O.kv_decode(codec, s, G, roll, 0, T, lens=[T, T]),
                                      O.kv_decode(codec, s, G, full, 0, T, lens=[T, T]))


def test_tile_bits_per_value_closed_form():
    """Tiles carry two binary16 per Tb x n values: b + 32 / (Tb n) bits per value, e.g.
    4 + 1/64 for the 16 x 128 tile at 4 bits; unfinished tokens count 16 bits."""
    for b in (3, 4, 6):
        assert O.bits_per_value(_tile(b, 128, 16), 8192, 128) == b + 32 / 2048
    ref = (8192 * (4 + 32 / 2048) + 8 * 16) / 8200
    assert abs(O.bits_per_value(_tile(4, 128, 16), 8200, 128) - ref) < 1e-12


# ------------------------------------------------------------------------------------------
# spectral statistics of the gauge training objective (section 4.2)
# ------------------------------------------------------------------------------------------
def _bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bits (x exactly representable in bf16 here)."""
    return (np.ascontiguousarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def test_spectral_dct_matches_scipy_and_radius_closed_form():
    from scipy.fft import dctn

    rng = np.random.default_rng(3)
    Z = rng.standard_normal((16, 64))
    U = O.dct2_matrix(16) @ Z @ O.dct2_matrix(64).T
    np.testing.assert_allclose(U, dctn(Z, type=2, norm="ortho"), rtol=0, atol=1e-12)
    rho = O.spectral_radius(16, 64)
    assert rho[0, 0] == 0.0 and abs(rho[15, 63] - 1.0) < 1e-15
    assert abs(rho[15, 0] - np.sqrt(0.5)) < 1e-15


def test_spectral_stats_of_a_constant_cache():
    """A cache whose every vector is one constant: all energy at the DC coefficient, so
    L_freq = 0, concentration 1, sum E = the field's energy, and L_rate is the DC term over
    the Tb d coefficients of a block."""
    L, B, H, T, d = 1, 2, 2, 40, 64
    X = _bits(np.full((L, B, H, T, d), 0.75, np.float32))
    G = O.gauge_make(O.GAUGE_IDENTITY, L, H, d, 16)
    st, en = O.spectral_stats(X, G, 0, Tb=16)
    assert st[0, 0] < 1e-20 and abs(st[0, 2] - 1.0) < 1e-20     # off-DC energy is rounding only
    nblk = T // 16
    assert abs(st[0, 3] - B * H * nblk * 16 * d * 0.75 ** 2) < 1e-9
    dc = 0.75 * np.sqrt(16 * d)
    assert abs(st[0, 1] - np.log1p(dc / 0.04) / (16 * d)) < 1e-12
    assert np.count_nonzero(np.abs(en[0]) > 1e-20) == 1 and en[0, 0, 0] > 0


@pytest.mark.parametrize("u0,v0", [(3, 5), (15, 63), (0, 7), (9, 0)])
def test_spectral_stats_of_a_single_frequency(u0, v0):
    """x[t][c] = cos(pi (2t+1) u0 / 32) cos(pi (2c+1) v0 / 128) (identity gauge) is one basis
    function: L_freq = rho(u0, v0) and the only coefficient is 1 / (s_u0 s_v0) with
    s_k = sqrt((1 if k == 0 else 2) / N)."""
    Tb, d = 16, 64
    t = np.arange(Tb)[:, None]
    c = np.arange(d)[None, :]
    blk = np.cos(np.pi * (2 * t + 1) * u0 / (2 * Tb)) * np.cos(np.pi * (2 * c + 1) * v0 / (2 * d))
    Z = O.dct2_matrix(Tb) @ blk @ O.dct2_matrix(d).T
    s_u = np.sqrt((1.0 if u0 == 0 else 2.0) / Tb)
    s_v = np.sqrt((1.0 if v0 == 0 else 2.0) / d)
    assert abs(Z[u0, v0] - 1.0 / (s_u * s_v)) < 1e-9
    # through the statistics (float32 input, exact float64 gauge)
    X = blk.astype(np.float32)[None, None, None]
    G = O.gauge_make(O.GAUGE_IDENTITY, 1, 1, d, 16)
    st, _ = O.spectral_stats(X, G, 0, Tb=Tb)
    rho = np.sqrt((u0 / 15) ** 2 + (v0 / 63) ** 2) / np.sqrt(2)
    assert abs(st[0, 0] - rho) < 1e-6


def test_spectral_energy_is_preserved_by_gauge_and_dct():
    """Parseval: with an orthogonal gauge and the orthonormal DCT, the layer energy equals the
    energy of X over the whole blocks, and so does its split across layers."""
    w, K, V = _tensor(50, L=2)
    G = O.gauge_make(O.GAUGE_HAAR, 2, 2, 128, 32, seed=21)
    x = (K.astype(np.uint32) << 16).view(np.float32).astype(np.float64)[:, :, :, :48]
    st, en = O.spectral_stats(K, G, 0, Tb=16)
    for l in range(2):
        # the binary32 gauge is orthogonal to 1e-6 (its own pin), the DCT to rounding
        assert abs(st[l, 3] - float((x[l] ** 2).sum())) <= 2e-6 * st[l, 3]
        assert abs(en[l].sum() - st[l, 3]) <= 1e-9 * st[l, 3]
        assert 0.0 < st[l, 0] < 1.0 and st[l, 1] > 0.0


# ------------------------------------------------------------------------------------------
# attention over the decoded cache
# ------------------------------------------------------------------------------------------
def test_attend_over_error_free_cache_is_plain_attention():
    """Passthrough backend: the decoded cache is X to the gauge's rounding, so the oracle's
    attention equals torch's scaled-dot-product attention on X (binary64)."""
    import torch
    L, B, H, grp, T, d = 1, 2, 2, 3, 40, 64
    w, K, V = _tensor(T, d=d, B=B, H=H)
    G = O.gauge_make(O.GAUGE_HAAR, L, H, d, 16, seed=31)
    pc = O.Codec(backend=O.PASSTHROUGH)
    kc, _ = O.kv_encode(pc, 0, K, G, T_cap=T)
    vc, _ = O.kv_encode(pc, 1, V, G, T_cap=T)
    rng = np.random.default_rng(5)
    q = rng.standard_normal((L, B, H * grp, d)).astype(np.float32)
    lens = [T, 23]
    got = O.attend(pc, G, kc, vc, q, lens, 1 / np.sqrt(d))
    x = lambda a: torch.from_numpy((a.astype(np.uint32) << 16).view(np.float32).astype(np.float64))
    Kx, Vx = x(K), x(V)
    for b in range(B):
        n = lens[b]
        qq = torch.from_numpy(q[0, b].astype(np.float64))[:, None, :]            # [Hq][1][d]
        kk = Kx[0, b].repeat_interleave(grp, dim=0)[:, :n]                          # [Hq][n][d]
        vv = Vx[0, b].repeat_interleave(grp, dim=0)[:, :n]
        ref = torch.nn.functional.scaled_dot_product_attention(qq, kk, vv, scale=1 / np.sqrt(d))[:, 0]
        np.testing.assert_allclose(got[0, b], ref.numpy(), rtol=0, atol=1e-5)


def test_attend_closed_forms():
    """Equal keys give equal weights (the output is the mean of the decoded values); a single
    position gives its decoded value."""
    L, B, H, T, d = 1, 1, 2, 32, 64
    G = O.gauge_make(O.GAUGE_HAAR, L, H, d, 32, seed=32)
    codec = O.Codec(backend=O.BLOCK_UNIFORM, bits=4, block_c=32)
    w, _, V = _tensor(T, d=d, B=B, H=H)
    K = np.ascontiguousarray(np.repeat(V[:, :, :, :1], T, axis=3))          # one key repeated
    kc, _ = O.kv_encode(codec, 0, K, G, T_cap=T)
    vc, _ = O.kv_encode(codec, 1, V, G, T_cap=T)
    q = np.random.default_rng(6).standard_normal((L, B, H, d)).astype(np.float32)
    Vh = O.kv_decode(codec, 1, G, vc, 0, T, out_bf16=False).astype(np.float64)
    got = O.attend(codec, G, kc, vc, q, [T], 0.125)
    np.testing.assert_allclose(got[0, 0], Vh[0, 0].mean(axis=1), rtol=0, atol=1e-12)
    got1 = O.attend(codec, G, kc, vc, q, [1], 0.125)
    np.testing.assert_allclose(got1[0, 0], Vh[0, 0, :, 0], rtol=0, atol=1e-12)
    # a row with no positions: the empty softmax is taken as a zero output
    assert (O.attend(codec, G, kc, vc, q, [0], 0.125) == 0).all()
    # hard-max limit: with the value cache also serving as the key cache (decoded as keys, with
    # the key gauge) and a scale large enough that the best score leads the next by more than
    # 60 / scale, the output is the decoded value of the best position
    big = O.attend(codec, G, vc, vc, q, [T], 1e3)
    Kv = O.kv_decode(codec, 0, G, vc, 0, T, out_bf16=False).astype(np.float64)
    sc = np.einsum("htc,hc->ht", Kv[0, 0], q[0, 0].astype(np.float64))
    srt = np.sort(sc, axis=1)
    for h in range(H):
        assert (srt[h, -1] - srt[h, -2]) * 1e3 > 60
        np.testing.assert_allclose(big[0, 0, h], Vh[0, 0, h, sc[h].argmax()], rtol=0, atol=1e-12)
