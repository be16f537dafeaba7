"""Pins of the oracle's gradient of the training objective (sections 4.1-4.2, CPU only).

* expm64 (power series with scaling and squaring) against scipy's Pade expm, the 2 x 2 rotation
  closed form and orthogonality of exp(S) for skew-symmetric S;
* expm_frechet64 (block matrix exponential) against scipy's expm_frechet, central differences
  of expm64, and the adjoint identity <Y, L(M, E)> = <L(M^T, Y), E> the gradient relies on;
* spectral_train_grad against central differences of spectral_train_loss: every step of the
  chain rule (the two loss terms separately and together, keys and values, one and two gauge
  groups, token blocks of 8 and 16, binary32 and bf16 input).
"""
import numpy as np
import pytest
import scipy.linalg

import oracle as O


def test_expm64_matches_scipy_and_closed_forms():
    rng = np.random.default_rng(3)
    for n, scale in ((1, 1.0), (5, 0.3), (8, 2.0), (12, 6.0)):
        W = scale * rng.standard_normal((n, n))
        ref = scipy.linalg.expm(W)
        assert np.abs(O.expm64(W) - ref).max() <= 1e-12 * max(1.0, np.abs(ref).max())
    for th in (0.0, 0.3, 2.5, -7.0):
        R = O.expm64(np.array([[0.0, -th], [th, 0.0]]))
        np.testing.assert_allclose(R, [[np.cos(th), -np.sin(th)], [np.sin(th), np.cos(th)]], atol=1e-13)
    A = rng.standard_normal((16, 16))
    Q = O.expm64(A - A.T)
    assert np.abs(Q.T @ Q - np.eye(16)).max() < 1e-12


def test_expm_frechet_matches_scipy_differences_and_adjoint():
    rng = np.random.default_rng(4)
    for n, scale in ((3, 0.5), (8, 1.5), (10, 4.0)):
        M = scale * rng.standard_normal((n, n))
        E = rng.standard_normal((n, n))
        Lf = O.expm_frechet64(M, E)
        ref = scipy.linalg.expm_frechet(M, E, compute_expm=False)
        assert np.abs(Lf - ref).max() <= 1e-11 * max(1.0, np.abs(ref).max())
        h = 1e-5
        fd = (O.expm64(M + h * E) - O.expm64(M - h * E)) / (2 * h)
        assert np.abs(Lf - fd).max() <= 1e-6 * max(1.0, np.abs(fd).max())
        Y = rng.standard_normal((n, n))
        lhs = float((Y * Lf).sum())
        rhs = float((O.expm_frechet64(M.T, Y) * E).sum())
        assert abs(lhs - rhs) <= 1e-11 * max(1.0, abs(lhs))


def _fd_check(X, A, s, Tb, lam_f, lam_r, entries, rtol=2e-6):
    gr = O.spectral_train_grad(X, A, s, Tb=Tb, lam_f=lam_f, lam_r=lam_r)
    L_, _, H, R, g, _ = A.shape
    assert gr.shape == (L_, H, R, g, g)
    scale = np.abs(gr).max()
    assert scale > 0
    h = 1e-6
    for (l, hh, r, i, j) in entries:
        Ap = A.copy()
        Ap[l, s, hh, r, i, j] += h
        Am = A.copy()
        Am[l, s, hh, r, i, j] -= h
        lp = O.spectral_train_loss(X, Ap, s, Tb=Tb, lam_f=lam_f, lam_r=lam_r)
        lm = O.spectral_train_loss(X, Am, s, Tb=Tb, lam_f=lam_f, lam_r=lam_r)
        fd = (lp[l] - lm[l]) / (2 * h)
        assert abs(fd - gr[l, hh, r, i, j]) <= rtol * scale, (l, hh, r, i, j, fd, gr[l, hh, r, i, j])
        # the other layers do not depend on this layer's gauge
        others = [k for k in range(L_) if k != l]
        assert np.all(lp[others] == lm[others])
    return gr


@pytest.mark.parametrize("lam_f,lam_r", [(1.0, 0.0), (0.0, 1.0), (1.0, 0.02)])
def test_gradient_matches_central_differences(lam_f, lam_r):
    rng = np.random.default_rng(11)
    X = rng.standard_normal((2, 2, 2, 28, 16)).astype(np.float32)   # 28 tokens: 3 blocks of 8, 4 unused
    A = 0.4 * rng.standard_normal((2, 2, 2, 2, 8, 8))
    entries = [(0, 0, 0, 0, 1), (0, 1, 1, 3, 5), (1, 0, 1, 7, 2), (1, 1, 0, 6, 6), (1, 1, 1, 2, 4)]
    for s in (0, 1):
        _fd_check(X, A, s, 8, lam_f, lam_r, entries)


def test_gradient_full_head_gauge_bf16_input_and_16_token_blocks():
    rng = np.random.default_rng(12)
    X = (rng.standard_normal((1, 1, 1, 40, 16)) * 3).astype(np.float32)
    Xb = ((X.view(np.uint32) + 0x8000) >> 16).astype(np.uint16)      # bf16 bit patterns
    A = 0.7 * rng.standard_normal((1, 2, 1, 1, 16, 16))
    gr = _fd_check(Xb, A, 1, 16, 1.0, 0.02, [(0, 0, 0, 0, 15), (0, 0, 0, 9, 3), (0, 0, 0, 12, 12)])
    np.testing.assert_allclose(gr, -np.swapaxes(gr, -1, -2), atol=0)   # A enters through A - A^T


def test_loss_at_zero_generators_is_the_identity_gauge_statistic():
    rng = np.random.default_rng(13)
    X = rng.standard_normal((1, 1, 2, 32, 16)).astype(np.float32)
    A = np.zeros((1, 2, 2, 2, 8, 8))
    I = O.gauge_make(O.GAUGE_IDENTITY, 1, 2, 16, 8)
    st, _ = O.spectral_stats(X, I, 0, Tb=16)
    np.testing.assert_allclose(O.spectral_train_loss(X, A, 0, Tb=16, lam_f=1.0, lam_r=0.02),
                               st[:, 0] + 0.02 * st[:, 1], rtol=1e-14)
