"""Pins for the oracle's reconstruction, linear layer, dequantization, GEMM reference,
weighted MSE and bits-per-weight (CPU only).

Each pin checks the oracle against something other than itself: the paper's
one-hot / concatenation notation evaluated element by element, exact
rational arithmetic, a codebook whose entries encode their own indices, the
worked numeric example of App. C, closed forms and invariants.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import formats
from workloads import CONFIGS, LayerSpec, make_layer, make_activations

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _tiny(seed=0, M=3, B=3, g=4, d_out=5, d_in=12, dyadic=True):
    """Small random layer. dyadic=True draws values that are exact in fp16 and Fraction."""
    rng = np.random.default_rng(seed)
    codes = rng.integers(0, 2 ** B, size=(M, d_out, d_in // g))
    if dyadic:
        C = rng.integers(-64, 64, size=(M, 2 ** B, g)) / 64.0
        s = rng.integers(1, 8, size=d_out) / 4.0
    else:
        C = rng.normal(0, 0.02, size=(M, 2 ** B, g))
        s = rng.uniform(0.5, 1.5, size=d_out)
    return codes, C, s


def _onehot_reconstruct(codes, C, s, k):
    """W^(k) from the paper's notation, element by element: C_m is a g x 2^B matrix,
    b_ijm a one-hot column of length 2^B, group (i,j) = sum_{m<=k} C_m b_ijm, and the
    groups of row i are concatenated along d_in; each row is then scaled by s_i."""
    M, d_out, G = codes.shape
    nc, g = C.shape[1], C.shape[2]
    W = [[None] * (G * g) for _ in range(d_out)]
    for i in range(d_out):
        row = []
        for j in range(G):
            group = [Fraction(0)] * g
            for m in range(k):
                b = [1 if c == codes[m, i, j] else 0 for c in range(nc)]          # one-hot b_ijm
                Cm = [[Fraction(C[m, c, t]) for c in range(nc)] for t in range(g)]  # g x 2^B matrix
                for t in range(g):
                    group[t] += sum(Cm[t][c] * b[c] for c in range(nc))
            row.extend(group)                                                      # concatenation
        W[i] = [Fraction(s[i]) * v for v in row]
    return W


@pytest.mark.parametrize("k", [1, 2, 3])
def test_reconstruct_matches_onehot_notation(k):
    codes, C, s = _tiny(seed=k)
    W = oracle.reconstruct(codes, C, s, k)
    ref = _onehot_reconstruct(codes, C, s, k)
    for i in range(W.shape[0]):
        for t in range(W.shape[1]):
            assert Fraction(W[i, t]) == ref[i][t]


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_reconstruct_index_revealing(k):
    """C_m[c][t] = (c + 256 t) * 4096^m makes every weight a base-4096 number whose digit m is
    the code of plane m at that group shifted by 256 t; digits of planes >= k must be zero."""
    M, B, g, d_out, d_in = 4, 8, 8, 7, 64
    rng = np.random.default_rng(11)
    codes = rng.integers(0, 256, size=(M, d_out, d_in // g))
    C = np.array([[[(c + 256 * t) * 4096.0 ** m for t in range(g)] for c in range(256)] for m in range(M)])
    W = oracle.reconstruct(codes, C, np.ones(d_out), k)
    Wi = W.astype(np.int64)
    assert np.array_equal(Wi.astype(np.float64), W)
    for i in range(d_out):
        for col in range(d_in):
            j, t = divmod(col, g)
            v = int(Wi[i, col])
            for m in range(M):
                digit = (v >> (12 * m)) & 4095
                expect = codes[m, i, j] + 256 * t if m < k else 0
                assert digit == expect, (i, col, m)


def test_scale_multiplies_rows():
    """With every codeword equal to 1, W^(k)[i, :] = k * s_i on a non-square layer."""
    M, d_out, d_in, g = 3, 6, 16, 8
    codes = np.random.default_rng(0).integers(0, 4, size=(M, d_out, d_in // g))
    C = np.ones((M, 4, g))
    s = 2.0 ** np.arange(d_out)
    for k in range(1, M + 1):
        W = oracle.reconstruct(codes, C, s, k)
        assert np.array_equal(W, np.outer(k * s, np.ones(d_in)))


def test_prefix_nesting_exact():
    """W^(k) = W^(k-1) + s (.) C_{k-1}[codes_{k-1}] exactly (the first codebooks' part is kept
    at every level, §5), and k = M is the full AQLM reconstruction (§3.2)."""
    codes, C, s = _tiny(seed=5, M=4, B=4, g=4, d_out=6, d_in=16)
    Cf = formats.f16_bits_to_f64(C.astype(np.float16).view(np.uint16))
    sf = s.astype(np.float16).astype(np.float64)
    prev = None
    for k in range(1, 5):
        Wk = oracle.reconstruct(codes, Cf, sf, k)
        if prev is not None:
            plane = Cf[k - 1][codes[k - 1]].reshape(Wk.shape[0], -1) * sf[:, None]
            for a, b, c in zip(Wk.ravel(), prev.ravel(), plane.ravel()):
                assert Fraction(a) == Fraction(b) + Fraction(c)
        prev = Wk
    full = _onehot_reconstruct(codes, Cf, sf, 4)
    W4 = oracle.reconstruct(codes, Cf, sf, 4)
    assert all(Fraction(W4[i, t]) == full[i][t] for i in range(W4.shape[0]) for t in range(W4.shape[1]))


def test_k_out_of_range_rejected():
    codes, C, s = _tiny()
    for bad in (0, 4, -1):
        with pytest.raises(ValueError):
            oracle.reconstruct(codes, C, s, bad)


def test_linear_unit_vectors_and_loops():
    codes, C, s = _tiny(seed=9, M=3, B=3, g=4, d_out=5, d_in=12)
    for k in (1, 3):
        W = oracle.reconstruct(codes, C, s, k)
        # y(e_t) is column t of W^(k)
        for t in range(12):
            e = np.zeros((1, 12)); e[0, t] = 1.0
            assert np.array_equal(oracle.linear(e, codes, C, s, k)[0], W[:, t])
        # a batch of random x against a pure-Python double loop over the one-hot reconstruction
        x = np.random.default_rng(k).integers(-8, 8, size=(3, 12)) / 8.0
        ref = _onehot_reconstruct(codes, C, s, k)
        y = oracle.linear(x, codes, C, s, k)
        for b in range(3):
            for i in range(5):
                assert Fraction(y[b, i]) == sum(Fraction(x[b, t]) * ref[i][t] for t in range(12))


def test_bits_per_weight_worked_example():
    ex = json.load(open(os.path.join(GOLD, "avg_bits_worked_example.json")))
    v = oracle.bits_per_weight(ex["d_out"], ex["d_in"], ex["g"], ex["M"], ex["B"])
    assert round(v, ex["printed_decimals"]) == ex["printed_value"]
    # the codes term counts every codebook's plane: without the factor M the example gives ~1.002
    assert abs(v - 2.00223) < 1e-5


def test_bits_per_weight_closed_forms():
    # §6: K codebooks of 8-bit indices per group of 8 weights -> K bits per weight for the codes
    for k in range(1, 6):
        assert oracle.code_bits_per_weight(8, 8, k) == k
    # 4096 x 4096, g=8, B=8, level k: (16*8*k*256 + 4096*512*8*k + 16*4096) / 4096^2
    for k in range(1, 5):
        expect = (16 * 8 * k * 256 + 4096 * 512 * 8 * k + 16 * 4096) / 4096 ** 2
        assert oracle.bits_per_weight(4096, 4096, 8, 4, 8, k) == expect
    assert abs(oracle.bits_per_weight(4096, 4096, 8, 4, 8, 1) - 1.006) < 1e-3


def test_wmse_forms_agree_and_reduce_to_mse():
    rng = np.random.default_rng(4)
    W = rng.normal(size=(6, 10)); Wh = W + 0.1 * rng.normal(size=(6, 10))
    X = rng.normal(size=(10, 23))
    a, b = oracle.wmse_frobenius(W, Wh, X), oracle.wmse_trace(W, Wh, X)
    assert abs(a - b) <= 1e-12 * abs(a)
    I = np.eye(10)
    mse = float(np.mean((W - Wh) ** 2))
    assert abs(oracle.wmse_frobenius(W, Wh, I) - mse) <= 1e-14
    assert abs(oracle.wmse_trace(W, Wh, I) - mse) <= 1e-14
    # hand example: W = [[1,2],[3,4]], W_hat = 0, X = I -> (1+4+9+16)/(2*2) = 7.5
    assert oracle.wmse_frobenius([[1, 2], [3, 4]], np.zeros((2, 2)), np.eye(2)) == 7.5
    # scaling X by c scales the distortion by c^2; duplicating the columns of X leaves it unchanged
    assert abs(oracle.wmse_trace(W, Wh, 3 * X) - 9 * b) <= 1e-12 * b
    assert abs(oracle.wmse_frobenius(W, Wh, np.concatenate([X, X], axis=1)) - a) <= 1e-12 * a


def test_prefix_distortions_explicit_sums():
    """D^(k) written out as a quintuple sum over rows, samples, groups, positions and planes."""
    rng = np.random.default_rng(9)
    M, d_out, G, g, n = 3, 4, 3, 8, 5
    codes = rng.integers(0, 4, size=(M, d_out, G))
    C = rng.integers(-8, 9, size=(M, 256, g)).astype(np.float64) / 16   # exact in fp16 and fp64
    s = np.array([1.0, 0.5, 2.0, 1.5])
    W = rng.integers(-32, 33, size=(d_out, G * g)).astype(np.float64) / 32
    Xr = rng.integers(-4, 5, size=(n, G * g)).astype(np.float64) / 4
    got = oracle.prefix_distortions(W, codes, C, s, Xr)
    for k in range(1, M + 1):
        tot = Fraction(0)
        for i in range(d_out):
            for t in range(n):
                r = Fraction(0)
                for j in range(G):
                    for q in range(g):
                        w_hat = Fraction(s[i]) * sum(Fraction(C[m, codes[m, i, j], q]) for m in range(k))
                        r += (Fraction(W[i, j * g + q]) - w_hat) * Fraction(Xr[t, j * g + q])
                tot += r * r
        assert got[k - 1] == float(tot / (d_out * n)), k
    # with every plane reproducing W exactly the full level has zero distortion
    Wm = oracle.reconstruct(codes, C, s, M)
    assert oracle.prefix_distortions(Wm, codes, C, s, Xr)[-1] == 0.0


# ----------------------------------------------------------------------------- dequant

def _f16bits(a):
    return np.asarray(a, dtype=np.float64).astype(np.float16).view(np.uint16)


def test_dequant_index_revealing_codebook():
    """k = 1, s = 1, C_0[c][t] = c + 256 t (exact in fp16): the dequantized matrix spells out the
    codes, so group orientation, codeword orientation and indexing are pinned bit-exactly."""
    rng = np.random.default_rng(7)
    codes = rng.integers(0, 256, size=(2, 9, 6)).astype(np.uint8)
    C = np.zeros((2, 256, 8)); C[0] = [[c + 256 * t for t in range(8)] for c in range(256)]
    C[1] = 1e4  # plane 1 must not contribute at k = 1
    for out in ("f32", "f16"):
        w = oracle.dequant_canonical(codes, _f16bits(C), _f16bits(np.ones(9)), 1, out)
        v = w.astype(np.float64) if out == "f32" else formats.f16_bits_to_f64(w)
        j, t = np.divmod(np.arange(48), 8)
        assert np.array_equal(v, codes[0][:, j] + 256.0 * t[None, :])


def test_dequant_fp32_fold_hand_case():
    """Hand case for the stated evaluation order. C_0 = 1, C_1 = 2^-24 (an fp16 subnormal):
    1 + 2^-24 is a binary32 tie and rounds to even (1.0), while the exact value is 1 + 2^-24;
    alone, 2^-24 survives (subnormals are honoured) in every output format."""
    codes = np.zeros((2, 1, 1), dtype=np.uint8)
    C = np.zeros((2, 1, 8)); C[0] = 1.0; C[1] = 2.0 ** -24
    cb, s = _f16bits(C), _f16bits([1.0])
    assert np.all(oracle.dequant_canonical(codes, cb, s, 2, "f32") == np.float32(1.0))
    # three planes 1, 2^-24, 2^-24: the binary32 left fold stays at 1.0 (two ties to even),
    # whereas a wider accumulator would reach 1 + 2^-23, a representable binary32 value
    codes3 = np.zeros((3, 1, 1), dtype=np.uint8)
    C3f = np.zeros((3, 1, 8)); C3f[0] = 1.0; C3f[1] = 2.0 ** -24; C3f[2] = 2.0 ** -24
    assert np.all(oracle.dequant_canonical(codes3, _f16bits(C3f), s, 3, "f32") == np.float32(1.0))
    assert np.all(oracle.dequant_canonical(codes3, _f16bits(C3f), s, 3, "bf16") == 0x3F80)
    C2 = np.zeros((1, 1, 8)); C2[0] = 2.0 ** -24
    assert np.all(oracle.dequant_canonical(codes[:1], _f16bits(C2), s, 1, "f32") == np.float32(2.0 ** -24))
    assert np.all(oracle.dequant_canonical(codes[:1], _f16bits(C2), s, 1, "f16") == 0x0001)
    assert np.all(oracle.dequant_canonical(codes[:1], _f16bits(C2), s, 1, "bf16") == 0x3380)
    # scale applied after the fold with one binary32 rounding: (1 + 2^-10) * (1 + 2^-10)
    # = 1 + 2^-9 + 2^-20 is exact in binary32 and rounds to fp16 1 + 2^-9
    C3 = np.zeros((1, 1, 8)); C3[0] = 1 + 2.0 ** -10
    w = oracle.dequant_canonical(codes[:1], _f16bits(C3), _f16bits([1 + 2.0 ** -10]), 1, "f32")
    assert np.all(w == np.float32(1 + 2.0 ** -9 + 2.0 ** -20))
    w16 = oracle.dequant_canonical(codes[:1], _f16bits(C3), _f16bits([1 + 2.0 ** -10]), 1, "f16")
    assert np.all(formats.f16_bits_to_f64(w16) == 1 + 2.0 ** -9)


@pytest.mark.parametrize("out", ["f32", "f16", "bf16"])
def test_dequant_within_rounding_of_exact(out):
    """On a Gaussian-codebook layer, the canonical dequant differs from the exact fp64 W^(k)
    by at most half an output ulp plus the binary32 fold/scale error k * 2^-24 * s * sum|C|,
    and equals the correctly rounded exact value almost everywhere."""
    spec = LayerSpec("t", 48, 256, seed=3)
    L = make_layer(spec)
    C = formats.f16_bits_to_f64(L.codebooks); s = formats.f16_bits_to_f64(L.scales)
    for k in range(1, 5):
        exact = oracle.reconstruct(L.codes, C, s, k)
        w = oracle.dequant_canonical(L.codes, L.codebooks, L.scales, k, out)
        v = w.astype(np.float64) if out == "f32" else (formats.f16_bits_to_f64(w) if out == "f16"
                                                         else formats.bf16_bits_to_f64(w))
        absC = np.zeros_like(exact)
        for m in range(k):
            absC += np.abs(C[m][L.codes[m]]).reshape(exact.shape)
        bound = 0.5 * formats.ulp_of(exact, out) + (k + 1) * 2.0 ** -24 * s[:, None] * absC
        assert np.all(np.abs(v - exact) <= bound)
        assert np.mean(v == formats.round_to_format(exact, out)) > 0.99


def test_dequant_prefix_nesting_of_fold():
    """The unscaled binary32 fold at level k equals the fold at k-1 plus plane k-1, rounded once."""
    L = make_layer(LayerSpec("t", 16, 64, seed=8))
    ones = _f16bits(np.ones(16))
    prev = oracle.dequant_canonical(L.codes, L.codebooks, ones, 1, "f32")
    C32 = formats.f16_bits_to_f32(L.codebooks)
    for k in range(2, 5):
        cur = oracle.dequant_canonical(L.codes, L.codebooks, ones, k, "f32")
        plane = C32[k - 1][L.codes[k - 1]].reshape(cur.shape)
        assert np.array_equal(cur, (prev + plane).astype(np.float32))
        prev = cur


# ----------------------------------------------------------------------------- GEMM reference

def test_gemm_reference_definition_and_bound():
    L = make_layer(LayerSpec("t", 40, 128, seed=12, act_dtype="bf16"))
    X = formats.bf16_bits_to_f64(make_activations(L, 24, "bf16"))
    C = formats.f16_bits_to_f64(L.codebooks); s = formats.f16_bits_to_f64(L.scales)
    for k in (1, 4):
        G = oracle.gemm_reference(X, L.codes, L.codebooks, L.scales, k)
        # element by element from its description: bf16 rounding of the binary32 fold, then scale
        fold = np.zeros((40, 16, 8), dtype=np.float32)
        C32 = formats.f16_bits_to_f32(L.codebooks)
        for i in range(40):
            for j in range(16):
                acc = C32[0][L.codes[0, i, j]].copy()
                for m in range(1, k):
                    acc = (acc + C32[m][L.codes[m, i, j]]).astype(np.float32)
                fold[i, j] = acc
        wb = formats.round_to_format(fold.reshape(40, 128).astype(np.float64), "bf16")
        for n in (0, 7, 23):
            for i in (0, 13, 39):
                ref = sum(Fraction(X[n, t]) * Fraction(wb[i, t]) for t in range(128)) * Fraction(s[i])
                assert abs(Fraction(G[n, i]) - ref) <= abs(ref) * Fraction(1, 2 ** 50) + Fraction(1, 2 ** 80)
        # and it stays within the bf16 weight-rounding bound of the exact layer output
        y = oracle.linear(X, L.codes, C, s, k)
        W = oracle.reconstruct(L.codes, C, s, k)
        bound = (np.abs(X) @ np.abs(W).T) * (2.0 ** -8 + (k + 1) * 2.0 ** -24)
        assert np.all(np.abs(G - y) <= bound + 1e-15)
