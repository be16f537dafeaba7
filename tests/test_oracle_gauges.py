"""Pins of the oracle's gauges (paper section 3 Table 1; section 4.1 eq. G = exp(A - A^T),
G^-1 = G^T; section 4.3 identity / random orthogonal / Hadamard / DCT controls) and of the
gauge application, against closed forms, library routines and the paper's sanity rows."""
import os

import numpy as np
import pytest
import scipy.fft
import scipy.linalg

import oracle as O
from paper_2607_20538_amd import synth

GROUPS = [8, 16, 32, 64, 128]


def _blocks(G):
    g = G.shape[-1]
    return G.reshape(-1, g, g)


@pytest.mark.parametrize("g", GROUPS)
@pytest.mark.parametrize("kind", [O.GAUGE_IDENTITY, O.GAUGE_HAAR, O.GAUGE_DCT2, O.GAUGE_HADAMARD])
def test_every_gauge_is_orthogonal(kind, g):
    G = O.gauge_make(kind, L=1, H=2, d=128, g=g, seed=11)
    for blk in _blocks(G)[:8]:
        assert O.orthogonality_error(blk) <= 1e-6
        # same check in numpy, independent of the oracle's own routine
        e = np.abs(blk.astype(np.float64) @ blk.astype(np.float64).T - np.eye(g)).max()
        assert e <= 1e-6


@pytest.mark.parametrize("g", GROUPS)
def test_dct2_matches_scipy_orthonormal_dct(g):
    G = O.gauge_make(O.GAUGE_DCT2, 1, 1, g, g)[0, 0, 0, 0]
    ref = scipy.fft.dct(np.eye(g), type=2, norm="ortho", axis=0)   # column n = DCT of e_n
    diff = np.abs(G.astype(np.float64) - ref)
    ulp = np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)
    assert np.all(diff <= ulp + 1e-12)
    # DCT of a constant vector: sqrt(g) c in frequency 0, zero elsewhere
    z = O.gauge_apply(G[None], np.full(g, 3.0, dtype=np.float32))
    assert abs(z[0] - 3.0 * np.sqrt(g)) <= 1e-5 * 3.0 * np.sqrt(g)
    assert np.abs(z[1:]).max() <= 1e-5


def _fwht(x):
    x = x.astype(np.float64).copy()
    h = 1
    while h < x.size:
        for i in range(0, x.size, 2 * h):
            a, b = x[i:i + h].copy(), x[i + h:i + 2 * h].copy()
            x[i:i + h], x[i + h:i + 2 * h] = a + b, a - b
        h *= 2
    return x / np.sqrt(x.size)


@pytest.mark.parametrize("g", GROUPS)
def test_hadamard_matches_sylvester_and_fwht(g):
    G = O.gauge_make(O.GAUGE_HADAMARD, 1, 1, g, g)[0, 0, 0, 0]
    ref = scipy.linalg.hadamard(g) / np.sqrt(g)
    np.testing.assert_array_equal(np.sign(G), np.sign(ref))
    assert np.all(np.abs(np.abs(G) - np.float32(1.0 / np.sqrt(g))) == 0)
    e0 = np.zeros(g, dtype=np.float32)
    e0[0] = 1.0
    assert np.allclose(O.gauge_apply(G[None], e0), 1.0 / np.sqrt(g), rtol=0, atol=1e-7)
    x = np.random.default_rng(g).standard_normal(g).astype(np.float32)
    assert np.allclose(O.gauge_apply(G[None], x), _fwht(x), rtol=0, atol=1e-5)


def test_haar_is_deterministic_per_seed_and_independent_per_block():
    A = O.gauge_make(O.GAUGE_HAAR, 2, 2, 64, 16, seed=99)
    B = O.gauge_make(O.GAUGE_HAAR, 2, 2, 64, 16, seed=99)
    C = O.gauge_make(O.GAUGE_HAAR, 2, 2, 64, 16, seed=100)
    np.testing.assert_array_equal(A, B)
    assert np.abs(A - C).max() > 0.1
    blocks = _blocks(A)
    for i in range(len(blocks)):
        for j in range(i + 1, len(blocks)):
            assert np.abs(blocks[i] - blocks[j]).max() > 0.1


@pytest.mark.parametrize("g", [8, 32])
def test_haar_equals_lapack_qr_with_sign_fix(g):
    """Mezzadri (2007): Q of numpy/LAPACK's QR of the same Gaussian matrix times sign(diag R)."""
    G = O.gauge_make(O.GAUGE_HAAR, 1, 1, g, g, seed=7)[0, 0, 0, 0]
    M = np.array([[O.gaussian(7, 0, i * g + j) for j in range(g)] for i in range(g)])
    Q, R = np.linalg.qr(M)
    Q = Q * np.sign(np.diag(R))[None, :]
    assert np.abs(G - Q).max() <= 1e-6


def test_haar_moments():
    """Haar measure on O(g): E[G_ij] = 0, E[G_ij^2] = 1/g, E[tr G] = 0, E[(tr G)^2] = 1
    (Diaconis-Shahshahani); a QR without the sign fix has E[Q_00] < 0 and fails."""
    g, n = 8, 4096
    G = _blocks(O.gauge_make(O.GAUGE_HAAR, 1, 1, g * n, g, seed=2024)).astype(np.float64)
    tr = np.trace(G, axis1=1, axis2=2)
    assert abs(tr.mean()) < 4 * 1.0 / np.sqrt(n)
    assert abs((tr ** 2).mean() - 1.0) < 4 * np.sqrt(2.0 / n)
    m = G.mean(axis=0)
    assert np.abs(m).max() < 4.5 * np.sqrt(1.0 / g / n)
    assert abs((G ** 2).mean() - 1.0 / g) < 1e-3
    # power of the entry-mean test: unfixed Householder QR of the same Gaussians
    bad = []
    for k in range(256):
        M = np.array([[O.gaussian(5, k, i * g + j) for j in range(g)] for i in range(g)])
        bad.append(np.linalg.qr(M)[0])
    bad = np.array(bad)
    assert abs(bad[:, 0, 0].mean()) > 4.5 * np.sqrt(1.0 / g / 256)


def test_expm_closed_forms():
    # A = 0 -> identity
    G = O.gauge_make(O.GAUGE_EXPM, 1, 1, 16, 16, params=np.zeros((1, 2, 1, 1, 16, 16), np.float32))
    np.testing.assert_array_equal(G[0, 0, 0, 0], np.eye(16, dtype=np.float32))
    # g = 2: A - A^T = [[0, a], [-a, 0]] -> rotation [[cos a, sin a], [-sin a, cos a]]
    for a in (0.1, 1.0, 2.5, -4.0):
        A = np.zeros((1, 2, 1, 1, 2, 2), np.float32)
        A[..., 0, 1] = a
        G = O.gauge_make(O.GAUGE_EXPM, 1, 1, 2, 2, params=A)[0, 0, 0, 0]
        ref = np.array([[np.cos(a), np.sin(a)], [-np.sin(a), np.cos(a)]])
        assert np.abs(G - ref).max() <= 1e-7


@pytest.mark.parametrize("g", [8, 32, 64])
def test_expm_matches_scipy(g):
    rng = np.random.default_rng(g)
    A = (rng.standard_normal((1, 2, 1, 1, g, g)) * 0.3).astype(np.float32)
    G = O.gauge_make(O.GAUGE_EXPM, 1, 1, g, g, params=A)
    for s in range(2):
        a = A[0, s, 0, 0].astype(np.float64)
        ref = scipy.linalg.expm(a - a.T)
        assert np.abs(G[0, s, 0, 0] - ref).max() <= 1e-6
        assert abs(np.linalg.det(G[0, s, 0, 0].astype(np.float64)) - 1.0) <= 1e-5
        assert O.orthogonality_error(G[0, s, 0, 0]) <= 1e-6


def test_user_gauge_rejects_non_orthogonal():
    G = O.gauge_make(O.GAUGE_HAAR, 1, 1, 16, 16, seed=3)
    np.testing.assert_array_equal(O.gauge_make(O.GAUGE_USER, 1, 1, 16, 16, params=G), G)
    bad = G.copy()
    bad[0, 0, 0, 0, 3, 5] += 1e-3
    with pytest.raises(ValueError):
        O.gauge_make(O.GAUGE_USER, 1, 1, 16, 16, params=bad)


@pytest.mark.parametrize("g", [8, 16, 128])
def test_gauge_apply_is_exact_then_round(g):
    """z = fl32(G x) with the exact sum: equal to numpy's binary64 product rounded to
    binary32 (a sum of fp32 x bf16 products in binary64), within one binary32 ulp; the
    inverse uses G^T (a transposed operand would fail the comparison)."""
    d = 128
    G = O.gauge_make(O.GAUGE_HAAR, 1, 1, d, g, seed=g)[0, 0, 0]
    rng = np.random.default_rng(3)
    for _ in range(20):
        x = rng.standard_normal(d).astype(np.float32) * 3
        z = O.gauge_apply(G, x)
        ref = np.concatenate([G[r].astype(np.float64) @ x[r * g:(r + 1) * g].astype(np.float64)
                              for r in range(d // g)])
        ulp = np.spacing(np.abs(ref.astype(np.float32)))
        assert np.all(np.abs(z.astype(np.float64) - ref) <= ulp)
        xi = O.gauge_inverse(G, z)
        refi = np.concatenate([G[r].astype(np.float64).T @ z[r * g:(r + 1) * g].astype(np.float64)
                               for r in range(d // g)])
        assert np.all(np.abs(xi.astype(np.float64) - refi) <= np.spacing(np.abs(refi.astype(np.float32))))


def _read_golden(golden_dir):
    vals = {}
    for ln in open(os.path.join(golden_dir, "sanity_rows.txt")):
        if ln.strip() and not ln.startswith("#"):
            k, v = ln.split()
            vals[k] = float(v)
    return vals


def test_passthrough_round_trip_reproduces_paper_sanity_rows(golden_dir):
    """Paper section 4.4: identity clone has zero cache error; random inverse rows at g = 16
    stay below 5.1e-8 max cache NRMSE (fp32 transformed tensors)."""
    gold = _read_golden(golden_dir)
    g = int(gold["group_size"])
    w = synth.WORKLOADS["tiny"]
    assert w.g == g
    codec = O.Codec(backend=O.PASSTHROUGH)
    worst = 0.0
    for kind, seed in ((O.GAUGE_IDENTITY, 0), (O.GAUGE_HAAR, 1), (O.GAUGE_HAAR, 2), (O.GAUGE_HAAR, 3)):
        G = O.gauge_make(kind, w.L, w.H, w.d, w.g, seed=seed)
        for s in (0, 1):
            X = synth.kv_tensor(w, s)
            cache, flags = O.kv_encode(codec, s, X, G, T_cap=w.T)
            assert flags == 0
            Xh = O.kv_decode(codec, s, G, cache, 0, w.T, out_bf16=False)
            e = O.nrmse(X, Xh)
            if kind == O.GAUGE_IDENTITY:
                assert e == gold["identity_clone_nrmse"]
                np.testing.assert_array_equal(Xh, X)
            else:
                worst = max(worst, e)
    assert 0.0 < worst < gold["inverse_gauge_max_nrmse_below"]


def test_passthrough_round_trip_bf16_is_bit_exact():
    w = synth.WORKLOADS["llama8b"]
    G = O.gauge_make(O.GAUGE_HAAR, 1, 2, 128, 128, seed=5)
    X = synth.kv_tensor(w, 0, L=1, B=1, H=2, T=64)
    codec = O.Codec(backend=O.PASSTHROUGH)
    cache, _ = O.kv_encode(codec, 0, X, G, T_cap=64)
    Xh = O.kv_decode(codec, 0, G, cache, 0, 64, out_bf16=True)
    np.testing.assert_array_equal(Xh, X)
