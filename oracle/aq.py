"""The quantized linear layer of Drop-by-Drop, written out in fp64.

Notation follows the paper: a weight matrix W has d_out rows and d_in columns;
each row is cut into d_in/g groups of g consecutive weights; M codebooks
C_1..C_M each hold 2^B codewords of length g; b_{ijm} selects the codeword of
codebook m for group j of row i (§3.2, "Additive Quantization and AQLM").
Storage indexes codebooks from 0: plane m of ``codes`` holds, for every
(row i, group j), the index of the codeword taken from codebook m. The paper's
"first k codebooks" C_1..C_k are planes 0..k-1 here.

Shapes used throughout:
  codes      [M][d_out][d_in/g]  integer indices in [0, 2^B)
  codebooks  [M][2^B][g]         fp64 values (decode fp16 bits first)
  scales     [d_out]             fp64 values, one per output row
"""
from __future__ import annotations

import numpy as np

from . import formats


def _check_k(codes, k):
    M = codes.shape[0]
    if not (1 <= k <= M):
        raise ValueError(f"k must be in [1, {M}], got {k}")


def reconstruct(codes, codebooks, scales, k: int) -> np.ndarray:
    """Partial reconstruction W^(k) from the first k codebooks, in fp64.

    §5 ("Our Application: Drop-by-Drop"): row i of W^(k) is the concatenation,
    over the groups j = 1..d_in/g, of the sums over m = 1..k of the codeword that
    b_{ijm} selects from C_m. With k = M this is AQLM's full reconstruction
    (§3.2). The per-output scale s multiplies the whole reconstructed row i and
    is the same for every k (reading: the paper stores one s per layer next to
    C and b, App. C "Scales: d_out * 16" and the AQLMFormat(C, b, s) output of
    Alg. 1, but leaves it out of the reconstruction formula).
    """
    codes = np.asarray(codes)
    codebooks = np.asarray(codebooks, dtype=np.float64)
    scales = np.asarray(scales, dtype=np.float64)
    _check_k(codes, k)
    M, d_out, n_groups = codes.shape
    g = codebooks.shape[2]
    group_sums = np.zeros((d_out, n_groups, g), dtype=np.float64)
    for m in range(k):                          # only planes 0..k-1 are read
        group_sums += codebooks[m][codes[m]]    # [d_out][n_groups][g]
    W = group_sums.reshape(d_out, n_groups * g)  # groups are consecutive along d_in
    return W * scales[:, None]


def linear(x, codes, codebooks, scales, k: int) -> np.ndarray:
    """y = x . (W^(k))^T in fp64 for activations x of shape [batch][d_in].

    The paper writes the layer as Y = W X with X in R^{d_in x n} (§2.2); with
    row-major activations that is the same product transposed.
    """
    W = reconstruct(codes, codebooks, scales, k)
    x = np.asarray(x, dtype=np.float64)
    return x @ W.T


def dequant_canonical(codes, codebook_bits, scale_bits, k: int, out: str) -> np.ndarray:
    """W^(k) in a stated floating-point evaluation order, as a kernel must produce it.

    The paper gives W^(k) exactly (§5) and no rounding. This is the reading
    used for the bit-exact dequantization: every codeword entry is an fp16
    value taken exactly to binary32; the codewords of planes 0..k-1 are summed
    in binary32 as a left fold (C_0 + C_1, then + C_2, ...), each addition
    rounded to nearest even; the sum is multiplied by the row's scale in
    binary32 (one rounding, no fused multiply-add); the product is rounded to
    nearest even into the output format ``out`` in {"f32", "f16", "bf16"}.

    Returns float32 values for "f32" and uint16 bit patterns for "f16"/"bf16",
    shaped [d_out][d_in].
    """
    codes = np.asarray(codes)
    _check_k(codes, k)
    C32 = formats.f16_bits_to_f32(codebook_bits)          # [M][2^B][g] float32, exact
    s32 = formats.f16_bits_to_f32(scale_bits)             # [d_out] float32, exact
    M, d_out, n_groups = codes.shape
    acc = C32[0][codes[0]].astype(np.float32)             # [d_out][n_groups][g]
    for m in range(1, k):
        acc = (acc + C32[m][codes[m]]).astype(np.float32)  # float32 + float32 -> float32 (RNE)
    w = (acc * s32[:, None, None]).astype(np.float32)
    w = w.reshape(d_out, n_groups * acc.shape[2])
    if out == "f32":
        return w
    if out == "f16":
        return formats.f32_to_f16_bits(w)
    if out == "bf16":
        return formats.f32_to_bf16_bits(w)
    raise ValueError(out)


def gemm_reference(X, codes, codebook_bits, scale_bits, k: int) -> np.ndarray:
    """Reference for the prefill product fed to bf16 matrix cores, in fp64.

    The prefill GEMM multiplies bf16 activations by a bf16 weight tile. Its
    weight tile is the unscaled binary32 left fold of the first k codewords
    (the fold of ``dequant_canonical``) rounded to nearest-even bf16; the row
    scale is applied to the fp32 accumulator afterwards. This function computes
    X . RNE_bf16(fold)^T exactly in fp64 and multiplies column i by s_i, so the
    only differences left to a kernel are its fp32 accumulation order and the
    final rounding of the output.
    """
    codes = np.asarray(codes)
    _check_k(codes, k)
    C32 = formats.f16_bits_to_f32(codebook_bits)
    s = formats.f16_bits_to_f64(scale_bits)
    M, d_out, n_groups = codes.shape
    acc = C32[0][codes[0]].astype(np.float32)
    for m in range(1, k):
        acc = (acc + C32[m][codes[m]]).astype(np.float32)
    w_bf16 = formats.bf16_bits_to_f64(formats.f32_to_bf16_bits(acc)).reshape(d_out, -1)
    X = np.asarray(X, dtype=np.float64)
    return (X @ w_bf16.T) * s[None, :]


def wmse_frobenius(W, W_hat, X) -> float:
    """Weighted MSE, first form of Eq. (1) (§2.2): ||(W - W_hat) X||_F^2 / (d_out n).

    X has shape [d_in][n]. With X = I (n = d_in) it is the plain mean squared
    error of the weights.
    """
    W = np.asarray(W, dtype=np.float64)
    E = W - np.asarray(W_hat, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    d_out, n = W.shape[0], X.shape[1]
    R = E @ X
    return float(np.sum(R * R) / (d_out * n))


def wmse_trace(W, W_hat, X) -> float:
    """Weighted MSE, second form of Eq. (1) (§2.2): tr[E (X X^T / n) E^T] / d_out."""
    W = np.asarray(W, dtype=np.float64)
    E = W - np.asarray(W_hat, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    d_out, n = W.shape[0], X.shape[1]
    H = (X @ X.T) / n
    return float(np.trace(E @ H @ E.T) / d_out)


def prefix_distortions(W, codes, codebooks, scales, X_rows) -> np.ndarray:
    """D^(k) for k = 1..M (§5, the distortion of each partial reconstruction): the weighted MSE
    of Eq. (1), ||(W - W^(k)) X||_F^2 / (d_out n), with W^(k) from the first k codebooks.

    X_rows holds the n calibration inputs as rows, [n][d_in] (X of the paper is its transpose).
    Returns an array of M values, entry k - 1 for level k.
    """
    X = np.asarray(X_rows, dtype=np.float64).T
    M = np.asarray(codes).shape[0]
    return np.array([wmse_frobenius(W, reconstruct(codes, codebooks, scales, k), X) for k in range(1, M + 1)])


def bits_per_weight(d_out: int, d_in: int, g: int, M: int, B: int, k=None) -> float:
    """Average bits per weight of a stored layer, Eq. (avg_bits) of App. C.

    Codebooks g*M*2^B*16 bits, codes d_out*(d_in/g)*B bits for *each* codebook,
    scales d_out*16 bits, divided by d_out*d_in. The printed codes term has no
    factor M, but the worked example (Llama-2-70B gate_proj, g=8, M=2, B=8 at
    about 2.002 bits) only comes out with it, so the factor is included. At
    precision level k only the first k codebooks and their code planes are
    counted (k = M by default).
    """
    k = M if k is None else k
    if not (1 <= k <= M):
        raise ValueError("k out of range")
    if d_in % g:
        raise ValueError("d_in must be a multiple of g")
    codebook_bits = 16 * g * k * (2 ** B)
    code_bits = d_out * (d_in // g) * B * k
    scale_bits = 16 * d_out
    return (codebook_bits + code_bits + scale_bits) / (d_out * d_in)


def code_bits_per_weight(g: int, B: int, k: int) -> float:
    """Bits per weight spent on codes alone: k codebooks of B-bit indices per g weights (§6)."""
    return k * B / g
