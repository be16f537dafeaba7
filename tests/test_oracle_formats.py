"""Pins of the oracle's number formats and counter-based generator against independent
definitions: published known-answer vectors, numpy's binary16 and torch's bfloat16 casts,
and distribution tests of the normal sampler."""
import os

import numpy as np
import pytest
import torch

import oracle as O


def test_philox_known_answers(golden_dir):
    rows = [ln.split() for ln in open(os.path.join(golden_dir, "philox4x32_10_kat.txt")) if ln.strip() and
            not ln.startswith("#")]
    assert len(rows) == 3
    for r in rows:
        v = [int(x, 16) for x in r]
        out = O.philox4x32_10(v[0:4], v[4:6])
        assert [int(x) for x in out] == v[6:10]


def test_gaussian_stream_is_standard_normal():
    from scipy import stats

    xs = np.array([O.gaussian(1234, 7, k) for k in range(40000)])
    assert abs(xs.mean()) < 4.0 / np.sqrt(xs.size)
    assert abs(xs.var() - 1.0) < 4.0 * np.sqrt(2.0 / xs.size)
    assert stats.kstest(xs, "norm").pvalue > 1e-3
    # counter-based: the value depends only on (seed, stream, k)
    assert O.gaussian(1234, 7, 12345) == xs[12345]
    assert O.gaussian(1234, 8, 5) != O.gaussian(1234, 7, 5)


def test_bf16_round_to_nearest_even_matches_torch():
    rng = np.random.default_rng(0)
    vals = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * np.float32(10.0) ** rng.integers(-30, 30, 20000),
        # exact ties: bit 15 set, low bits clear, both parities of bit 16
        (np.arange(4000, dtype=np.uint32) << 16 | 0x8000).view(np.float32),
        np.array([0.0, -0.0, np.inf, -np.inf, 3.3895314e38, 1e-45], dtype=np.float32),
    ]).astype(np.float32)
    ref = torch.from_numpy(vals).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([O.f32_to_bf16(v) for v in vals], dtype=np.uint16)
    np.testing.assert_array_equal(got, ref)
    back = np.array([O.bf16_to_f32(int(b)) for b in ref[:2000]], dtype=np.float32)
    np.testing.assert_array_equal(back, torch.from_numpy(ref[:2000].view(np.int16)).view(torch.bfloat16).float()
                                  .numpy())


def test_f16_value_and_bits_match_numpy_for_every_pattern():
    pats = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = pats.view(np.float16).astype(np.float64)
    for p, r in zip(pats, ref):
        v = O.f16_value(int(p))
        if np.isnan(r):
            assert np.isnan(v)
            continue
        assert v == r and np.signbit(v) == np.signbit(r)
        assert O.f16_bits(v) == int(p)


def _numpy_directed(v, direction):
    """Largest binary16 <= v (direction -1) or smallest >= v (+1), via numpy's RNE cast."""
    h = np.float16(v)
    if direction < 0 and float(h) > v:
        h = np.nextafter(h, np.float16(-np.inf), dtype=np.float16)
    if direction > 0 and float(h) < v:
        h = np.nextafter(h, np.float16(np.inf), dtype=np.float16)
    r = float(h)
    if r == 0.0:
        r = 0.0
    return r


@pytest.mark.parametrize("direction", [-1, 1])
def test_f16_directed_rounding_matches_numpy(direction):
    rng = np.random.default_rng(1 + direction)
    v = (rng.standard_normal(30000) * 10.0 ** rng.uniform(-9, 4.7, 30000)).astype(np.float32)
    v = np.concatenate([v, np.array([0.0, -0.0, 65504.0, -65504.0, 6e-8, -6e-8, 1e-9, -1e-9, 2.0 ** -14,
                                     65519.0, -65519.0], dtype=np.float32)])
    with np.errstate(over="ignore"):
        for x in v:
            got = O.f16_round_dir(float(x), direction)
            ref = _numpy_directed(float(x), direction)
            if abs(float(x)) > 65504.0:
                # IEEE directed overflow: toward -inf gives +max for +huge and -inf for -huge
                if direction < 0:
                    ref = 65504.0 if x > 0 else -np.inf
                else:
                    ref = np.inf if x > 0 else -65504.0
            assert got == ref, (x, got, ref)
            assert not (got == 0.0 and np.signbit(got))


def test_f16_directed_rounding_brackets_value():
    rng = np.random.default_rng(5)
    for x in (rng.standard_normal(5000) * 100).astype(np.float32):
        lo, hi = O.f16_round_dir(float(x), -1), O.f16_round_dir(float(x), 1)
        assert lo <= x <= hi
        if lo != hi:
            assert np.nextafter(np.float16(lo), np.float16(np.inf), dtype=np.float16) == np.float16(hi)
