"""Pins for the oracle's encoders (CPU only): residual k-means (App. C initialisation) and
exhaustive / beam code search (App. C code optimisation) on tiny groups.

These also pin the distortion behaviour the paper's method relies on: on i.i.d. Gaussian
weights (the source model of §4), the distortion of W^(k) does not increase with k, and it
never beats the Gaussian rate-distortion bound D >= sigma^2 2^(-2R) (App. E, Eq. (gaussian-rd)).
"""
import numpy as np
import pytest

import oracle


@pytest.fixture(scope="module")
def gaussian_encoded():
    rng = np.random.default_rng(2024)
    W = rng.normal(0, 0.02, size=(128, 512))      # 8192 groups of 8: 32 groups per codeword
    codes, C, s = oracle.encode_residual_kmeans(W, M=4, B=8, g=8, seed=1, iters=6)
    return W, codes, C, s


def test_mse_non_increasing_in_k(gaussian_encoded):
    W, codes, C, s = gaussian_encoded
    I = np.eye(W.shape[1])
    d = [oracle.wmse_frobenius(W, oracle.reconstruct(codes, C, s, k), I) for k in range(1, 5)]
    assert all(d[k] <= d[k - 1] for k in range(1, 4)), d
    assert d[0] < np.var(W)       # even one codebook beats the zero reconstruction


def test_wmse_non_increasing_gaussian_x(gaussian_encoded):
    W, codes, C, s = gaussian_encoded
    X = np.random.default_rng(5).normal(size=(W.shape[1], 4 * W.shape[1]))
    d = [oracle.wmse_trace(W, oracle.reconstruct(codes, C, s, k), X) for k in range(1, 5)]
    assert all(d[k] < d[k - 1] for k in range(1, 4)), d


def test_shannon_lower_bound(gaussian_encoded):
    """Rate of k codebooks is R = k*B/g bits per weight (§6); no code can beat sigma^2 2^(-2R)."""
    W, codes, C, s = gaussian_encoded
    var = float(np.var(W))
    for k in range(1, 5):
        mse = float(np.mean((W - oracle.reconstruct(codes, C, s, k)) ** 2))
        assert mse / var >= 2.0 ** (-2 * k * 8 / 8), (k, mse / var)


def test_single_codeword_is_the_mean():
    """B = 0: each codebook holds one codeword; k-means puts it at the mean of the groups,
    and the next stage's codeword is the mean of the residuals, i.e. zero."""
    rng = np.random.default_rng(3)
    W = rng.normal(1.0, 0.5, size=(6, 16))
    codes, C, s = oracle.encode_residual_kmeans(W, M=2, B=0, g=4, seed=0)
    assert np.allclose(C[0, 0], W.reshape(-1, 4).mean(axis=0), atol=1e-14)
    assert np.allclose(C[1, 0], 0.0, atol=1e-14)
    assert np.all(codes == 0)


def test_exactly_representable_weights_are_recovered():
    rng = np.random.default_rng(8)
    C = rng.integers(-16, 16, size=(2, 4, 2)) / 16.0
    codes_true = rng.integers(0, 4, size=(2, 3, 3))
    s = np.array([1.0, 0.5, 2.0])
    W = oracle.reconstruct(codes_true, C, s, 2)
    codes, err = oracle.brute_force_codes(W, C, s, 2)
    assert err == 0.0
    assert np.array_equal(oracle.reconstruct(codes, C, s, 2), W)


@pytest.mark.parametrize("k,nb,g", [(1, 4, 2), (2, 4, 2), (3, 4, 2), (2, 16, 4)])
def test_brute_force_is_optimal_and_consistent(k, nb, g):
    rng = np.random.default_rng(k * 10 + nb)
    M = 3
    C = rng.normal(size=(M, nb, g))
    s = rng.uniform(0.5, 1.5, 4)
    W = rng.normal(size=(4, 3 * g))
    codes, err = oracle.brute_force_codes(W, C, s, k)
    # the reported minimum is the error of the reconstruction of the returned codes
    recon_err = float(np.sum((W - oracle.reconstruct(codes, C[:k], s, k)) ** 2))
    assert abs(recon_err - err) <= 1e-12 * max(1.0, err)
    # no random code tuple does better
    for t in range(200):
        rc = rng.integers(0, nb, size=(k, 4, 3))
        assert float(np.sum((W - oracle.reconstruct(rc, C[:k], s, k)) ** 2)) >= err - 1e-12
    # beam search: greedy is never better; a beam of (2^B)^(k-1) is exhaustive
    _, greedy = oracle.beam_search_codes(W, C, s, k, beam=1)
    assert greedy >= err - 1e-12
    full_codes, full = oracle.beam_search_codes(W, C, s, k, beam=nb ** (k - 1))
    assert abs(full - err) <= 1e-12 * max(1.0, err)
    assert np.array_equal(full_codes, codes)      # same tie-break: lexicographically smallest
