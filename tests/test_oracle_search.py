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


# ---- beam search with decisions in binary32 (the reference of the GPU search) ----

def _int_case(rng, M, nb, g, d_out, G):
    C = rng.integers(-4, 5, size=(M, nb, g)).astype(np.float64)
    s = rng.choice(np.array([0.5, 1.0, 2.0]), size=d_out)
    W = rng.integers(-16, 17, size=(d_out, G * g)).astype(np.float64)
    return C, s, W


@pytest.mark.parametrize("k,nb,beam", [(1, 16, 4), (2, 16, 1), (2, 16, 3), (3, 8, 4), (3, 8, 64), (4, 4, 2)])
def test_f32_beam_equals_exact_beam_on_integer_data(k, nb, beam):
    """On integer-valued inputs every binary32 operation of the search is exact, so its decisions
    are those of the fp64 search (itself pinned against exhaustive search below)."""
    rng = np.random.default_rng(100 + 10 * k + beam)
    C, s, W = _int_case(rng, 4, nb, 4, 5, 6)
    c32, e32 = oracle.beam_search_codes_f32(W, C, s, k, beam)
    c64, t64 = oracle.beam_search_codes(W, C, s, k, beam)
    assert np.array_equal(c32, c64)
    assert float(e32.astype(np.float64).sum()) == t64


def test_f32_full_beam_is_exhaustive_on_integer_data():
    rng = np.random.default_rng(7)
    C, s, W = _int_case(rng, 3, 8, 4, 4, 5)
    codes, best = oracle.brute_force_codes(W, C, s, 3)
    c32, e32 = oracle.beam_search_codes_f32(W, C, s, 3, beam=8 * 8)
    assert np.array_equal(c32, codes)
    assert float(e32.astype(np.float64).sum()) == best


def test_f32_beam_recovers_signed_digit_codes():
    """Codebook m holds the codewords (d * 16^(2-m)) * (1, ..., 1) with signed digits d in [-7, 8];
    a weight group built from one codeword per codebook is recovered exactly by any beam, greedy
    included (every stage's nearest codeword is the true digit), with error 0."""
    rng = np.random.default_rng(8)
    g, k = 8, 3
    digits = np.arange(-7, 9, dtype=np.float64)                       # 16 codewords
    C = np.stack([np.repeat((digits * 16.0 ** (k - 1 - m))[:, None], g, axis=1) for m in range(k)])
    true = rng.integers(0, 16, size=(k, 3, 4))
    s = np.array([1.0, 0.5, 0.25])
    W = oracle.reconstruct(true, C, s, k)
    for beam in (1, 2, 5):
        c32, e32 = oracle.beam_search_codes_f32(W, C, s, k, beam)
        assert np.array_equal(c32, true)
        assert np.all(e32 == 0)


def test_f32_beam_reported_error_reevaluates():
    """On Gaussian data the reported binary32 error is the squared error of the returned codes'
    reconstruction, up to binary32 rounding of the residual chain and of the sum."""
    rng = np.random.default_rng(9)
    f16 = lambda a: a.astype(np.float16).astype(np.float64)
    C = f16(rng.normal(0, 0.02, size=(3, 32, 8)))
    s = f16(rng.uniform(0.5, 1.5, size=6))
    W = f16(rng.normal(0, 0.02, size=(6, 40)))
    codes, e32 = oracle.beam_search_codes_f32(W, C, s, 3, beam=4)
    R = W - oracle.reconstruct(codes, C, s, 3)
    e64 = (R.reshape(6, 5, 8) ** 2).sum(axis=2)
    u = 2.0 ** -24
    # each d carries at most k roundings relative to |r| + |s c| terms; the sum g more
    mag = (np.abs(W) + np.abs(oracle.reconstruct(codes, C, s, 3))).reshape(6, 5, 8)
    bound = 2 * (3 + 1) * u * (np.sqrt(e64) * np.sqrt((mag ** 2).sum(axis=2))) * 2 + 10 * u * e64
    assert np.all(np.abs(e32.astype(np.float64) - e64) <= bound + 1e-30)


def test_f32_beam_groups_subset():
    """Searching a subset of groups gives the same results for those groups."""
    rng = np.random.default_rng(10)
    C, s, W = _int_case(rng, 2, 16, 4, 3, 4)
    full_c, full_e = oracle.beam_search_codes_f32(W, C, s, 2, 3)
    sub = [(0, 1), (2, 3)]
    c, e = oracle.beam_search_codes_f32(W, C, s, 2, 3, groups=sub)
    for (i, j) in sub:
        assert np.array_equal(c[:, i, j], full_c[:, i, j]) and e[i, j] == full_e[i, j]
    assert np.isnan(e[1, 0])


# ---- data-aware (weighted) code search: d^T H_jj d with H_jj the group's block of X X^T / n ----

def _block_x(rng, d_in, g, per_group):
    """Calibration inputs X [d_in][n] whose rows of different groups share no column: X X^T is
    then block diagonal, so the per-group weighted errors add up to the paper's WMSE exactly."""
    G = d_in // g
    X = np.zeros((d_in, G * per_group))
    for j in range(G):
        X[j * g:(j + 1) * g, j * per_group:(j + 1) * per_group] = rng.normal(size=(g, per_group))
    return X


def test_hessian_blocks_are_the_diagonal_blocks():
    rng = np.random.default_rng(30)
    X = rng.normal(size=(12, 7))
    Hb = oracle.group_hessian_blocks(X, 4)
    H = np.einsum("in,jn->ij", X, X) / 7           # X X^T / n written out elementwise
    for j in range(3):
        assert np.allclose(Hb[j], H[4 * j:4 * j + 4, 4 * j:4 * j + 4], rtol=0, atol=1e-14)


def test_weighted_search_with_identity_is_the_plain_search():
    """X = I (H = I) reduces the WMSE to the plain MSE (§2.2): same codes, same error."""
    rng = np.random.default_rng(31)
    C = rng.normal(size=(3, 8, 4))
    s = rng.uniform(0.5, 1.5, 4)
    W = rng.normal(size=(4, 12))
    eye = np.stack([np.eye(4)] * 3)
    for beam in (1, 3):
        c0, e0 = oracle.beam_search_codes(W, C, s, 3, beam)
        c1, e1 = oracle.beam_search_codes(W, C, s, 3, beam, H_blocks=eye)
        assert np.array_equal(c0, c1) and abs(e0 - e1) <= 1e-12 * max(1.0, e0)


@pytest.mark.parametrize("k,nb", [(1, 8), (2, 8), (3, 4)])
def test_weighted_exhaustive_search_minimises_the_papers_wmse(k, nb):
    """With block-diagonal X X^T the per-group weighted errors of the exhaustive search add up to
    the WMSE of Eq. (wmse-task) computed as (1/n) ||(W - W_hat) X||_F^2 (times d_out: the oracle's
    wmse_frobenius normalises by d_out n), and no random code assignment has a lower WMSE. The
    full-width beam finds the same codes."""
    rng = np.random.default_rng(40 + k)
    g, d_out, d_in = 4, 3, 12
    C = rng.normal(size=(3, nb, g))
    s = rng.uniform(0.5, 1.5, d_out)
    W = rng.normal(size=(d_out, d_in))
    X = _block_x(rng, d_in, g, 5)
    Hb = oracle.group_hessian_blocks(X, g)
    codes, total = oracle.brute_force_codes(W, C, s, k, H_blocks=Hb)
    wmse = oracle.wmse_frobenius(W, oracle.reconstruct(codes, C[:k], s, k), X)
    assert abs(total / d_out - wmse) <= 1e-12 * max(1.0, wmse)
    for _ in range(100):
        rc = rng.integers(0, nb, size=(k, d_out, d_in // g))
        assert oracle.wmse_frobenius(W, oracle.reconstruct(rc, C[:k], s, k), X) >= wmse - 1e-12
    full_codes, full = oracle.beam_search_codes(W, C, s, k, beam=nb ** (k - 1), H_blocks=Hb)
    assert np.array_equal(full_codes, codes) and abs(full - total) <= 1e-12 * max(1.0, total)
    # the plain search is never better in the weighted objective
    plain_codes, _ = oracle.brute_force_codes(W, C, s, k)
    assert oracle.wmse_frobenius(W, oracle.reconstruct(plain_codes, C[:k], s, k), X) >= wmse - 1e-12


def _int_spd_blocks(rng, G, g):
    """Integer symmetric positive semi-definite blocks A^T A with small integer A."""
    A = rng.integers(-2, 3, size=(G, g, g)).astype(np.float64)
    return np.einsum("jut,juv->jtv", A, A)


@pytest.mark.parametrize("k,nb,beam", [(1, 16, 4), (2, 16, 1), (2, 16, 3), (3, 8, 4), (3, 8, 64), (4, 4, 2)])
def test_weighted_f32_equals_exact_on_integer_data(k, nb, beam):
    """On integer inputs (weights, codewords, scales 1/2, 1, 2, integer blocks) every binary32
    operation of the weighted search is exact, so its decisions are those of the fp64 weighted
    search (pinned against the WMSE and exhaustive search above), and its reported error is the
    fp64 weighted error."""
    rng = np.random.default_rng(200 + 10 * k + beam)
    C, s, W = _int_case(rng, 4, nb, 4, 5, 6)
    Hb = _int_spd_blocks(rng, 6, 4)
    c32, e32 = oracle.beam_search_codes_weighted_f32(W, C, s, Hb, k, beam)
    c64, t64 = oracle.beam_search_codes(W, C, s, k, beam, H_blocks=Hb)
    assert np.array_equal(c32, c64)
    assert float(e32.astype(np.float64).sum()) == t64


def test_weighted_f32_reported_error_reevaluates():
    """On Gaussian data the reported binary32 error is d^T H d of the returned codes, up to the
    rounding of the expanded form (terms of size r^T H r, 2 s C^T H r and s^2 C^T H C)."""
    rng = np.random.default_rng(32)
    f16 = lambda a: a.astype(np.float16).astype(np.float64)
    C = f16(rng.normal(0, 0.02, size=(3, 32, 8)))
    s = f16(rng.uniform(0.5, 1.5, size=5))
    W = f16(rng.normal(0, 0.02, size=(5, 24)))
    Hb = oracle.group_hessian_blocks(rng.normal(size=(24, 40)), 8).astype(np.float32).astype(np.float64)
    codes, e32 = oracle.beam_search_codes_weighted_f32(W, C, s, Hb, 3, beam=4)
    R = (W - oracle.reconstruct(codes, C, s, 3)).reshape(5, 3, 8)
    e64 = np.einsum("ijt,jtu,iju->ij", R, Hb, R)
    rr = np.abs(W.reshape(5, 3, 8))
    u = 2.0 ** -24
    # |terms| <= ||H||_F (|w| + |s sum C|)^2 summed: a generous first-order bound of 64 roundings
    mag = np.einsum("ijt,ju,iju->ij", rr + np.abs(oracle.reconstruct(codes, C, s, 3)).reshape(5, 3, 8),
                    np.abs(Hb).sum(axis=2), rr + np.abs(oracle.reconstruct(codes, C, s, 3)).reshape(5, 3, 8))
    assert np.all(np.abs(e32.astype(np.float64) - e64) <= 64 * u * mag + 1e-30)
    assert np.all(e64 >= 0)


def test_weighted_f32_groups_subset():
    rng = np.random.default_rng(33)
    C, s, W = _int_case(rng, 2, 16, 4, 3, 4)
    Hb = _int_spd_blocks(rng, 4, 4)
    full_c, full_e = oracle.beam_search_codes_weighted_f32(W, C, s, Hb, 2, 3)
    sub = [(0, 1), (2, 3)]
    c, e = oracle.beam_search_codes_weighted_f32(W, C, s, Hb, 2, 3, groups=sub)
    for (i, j) in sub:
        assert np.array_equal(c[:, i, j], full_c[:, i, j]) and e[i, j] == full_e[i, j]
    assert np.isnan(e[1, 0])
