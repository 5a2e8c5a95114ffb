"""Encoders that produce codes: residual k-means initialisation and code search.

Neither is on the inference hot path. They produce fixtures (codes for Gaussian
weights, on which distortion must fall with k) and pin the meaning of "codes
that minimise the quantization error" on tiny groups.

App. C ("AQLM's Optimization Process") describes the initialisation: k-means
on the weight groups gives the first codebook and its assignments; the
differences between the weights and their centroids are clustered again to
give the next codebook, and so on. The code-optimisation phase searches
combinations of codewords that minimise the quantization error (beam search).
"""
from __future__ import annotations

import itertools

import numpy as np


def _lloyd(points: np.ndarray, n_centroids: int, iters: int, rng: np.random.Generator):
    """Lloyd's k-means on the rows of ``points``.

    Initial centroids are distinct rows drawn without replacement (all rows,
    repeated cyclically, if there are fewer rows than centroids). Each
    iteration assigns every point to its nearest centroid (squared Euclidean
    distance, ties to the lowest index) and moves every non-empty cluster's
    centroid to its mean; empty clusters keep their centroid. The run ends
    with one more assignment, so the returned assignment is nearest-centroid
    for the returned centroids, which come from a mean update.
    """
    n = points.shape[0]
    if n >= n_centroids:
        idx = rng.choice(n, size=n_centroids, replace=False)
    else:
        idx = np.arange(n_centroids) % n
    C = points[idx].copy()

    def assign(C):
        d = ((points[:, None, :] - C[None, :, :]) ** 2).sum(axis=2)   # [n][n_centroids]
        return np.argmin(d, axis=1)

    for _ in range(max(1, iters)):
        a = assign(C)
        for c in range(n_centroids):
            members = points[a == c]
            if len(members):
                C[c] = members.mean(axis=0)
    return C, assign(C)


def encode_residual_kmeans(W, M: int, B: int, g: int, seed: int = 0, iters: int = 8):
    """Residual k-means encoding of W into M codebooks of 2^B codewords (App. C, initialisation).

    Returns (codes [M][d_out][d_in/g] int64, codebooks [M][2^B][g] fp64,
    scales [d_out] fp64). Scales are 1: the paper's initialisation produces s
    but does not say how; unit scales keep W^(k) = sum of codewords.
    """
    W = np.asarray(W, dtype=np.float64)
    d_out, d_in = W.shape
    if d_in % g:
        raise ValueError("d_in must be a multiple of g")
    rng = np.random.Generator(np.random.PCG64(seed))
    residual = W.reshape(-1, g).copy()          # groups of g consecutive weights, row by row
    codes = np.zeros((M, d_out, d_in // g), dtype=np.int64)
    codebooks = np.zeros((M, 2 ** B, g), dtype=np.float64)
    for m in range(M):
        C, a = _lloyd(residual, 2 ** B, iters, rng)
        codebooks[m] = C
        codes[m] = a.reshape(d_out, d_in // g)
        residual = residual - C[a]
    return codes, codebooks, np.ones(d_out)


def group_hessian_blocks(X, g: int) -> np.ndarray:
    """The g x g diagonal blocks of H = X X^T / n (§2.2, Eq. wmse-task), in fp64.

    X holds the n calibration inputs as columns ([d_in][n], the orientation of
    ||(W - W_hat) X||_F^2). Block j covers inputs j g .. j g + g - 1: it weights
    the error of group j of every row, d^T H_jj d, when the other groups' errors
    are left out (the per-group reading of the data-aware objective).
    """
    X = np.asarray(X, dtype=np.float64)
    d_in, n = X.shape
    if d_in % g:
        raise ValueError("d_in must be a multiple of g")
    H = X @ X.T / n
    return np.stack([H[j * g:(j + 1) * g, j * g:(j + 1) * g] for j in range(d_in // g)])


def _group_errors(w_group: np.ndarray, codebooks: np.ndarray, scale: float, tuples: np.ndarray,
                  H=None) -> np.ndarray:
    """Error of every code tuple (rows of ``tuples``): with d = w - s * sum_m C_m[c_m], the
    squared error d^T d, or with a g x g weight block H the weighted error d^T H d."""
    recon = np.zeros((tuples.shape[0], codebooks.shape[2]))
    for m in range(tuples.shape[1]):
        recon += codebooks[m][tuples[:, m]]
    diff = w_group[None, :] - scale * recon
    if H is None:
        return (diff * diff).sum(axis=1)
    return ((diff @ np.asarray(H, dtype=np.float64)) * diff).sum(axis=1)


def brute_force_codes(W, codebooks, scales, k: int, H_blocks=None):
    """Exhaustive code search with the first k codebooks, group by group.

    For every (row i, group j) it tries all (2^B)^k code tuples and keeps one
    with the smallest squared error ||W_ij - s_i sum_{m<k} C_m[c_m]||^2 (the
    plain MSE, X = I, of §2.2), or with ``H_blocks`` ([G][g][g], see
    group_hessian_blocks) the smallest weighted error d^T H_jj d; ties go to the
    lexicographically smallest tuple.
    Returns (codes [k][d_out][d_in/g], total error).
    Only for tiny g and 2^B: the cost is (2^B)^k per group.
    """
    W = np.asarray(W, dtype=np.float64)
    codebooks = np.asarray(codebooks, dtype=np.float64)
    scales = np.asarray(scales, dtype=np.float64)
    n_cw, g = codebooks.shape[1], codebooks.shape[2]
    d_out, d_in = W.shape
    tuples = np.array(list(itertools.product(range(n_cw), repeat=k)), dtype=np.int64)  # lexicographic
    codes = np.zeros((k, d_out, d_in // g), dtype=np.int64)
    total = 0.0
    for i in range(d_out):
        for j in range(d_in // g):
            Hj = None if H_blocks is None else H_blocks[j]
            err = _group_errors(W[i, j * g:(j + 1) * g], codebooks, scales[i], tuples, Hj)
            best = int(np.argmin(err))          # argmin returns the first (smallest) tuple on ties
            codes[:, i, j] = tuples[best]
            total += float(err[best])
    return codes, total


def beam_search_codes(W, codebooks, scales, k: int, beam: int, H_blocks=None):
    """Beam search over codebooks 0..k-1 in order, group by group (App. C, code optimisation).

    Stage m extends every kept partial tuple (c_0..c_{m-1}) by every codeword
    of codebook m and keeps the ``beam`` extensions with the smallest error of
    the partial reconstruction (squared error, or with ``H_blocks`` the
    weighted error d^T H_jj d); the last stage returns the best full tuple.
    With beam >= (2^B)^(k-1) nothing is ever dropped before the last stage, so
    the result equals exhaustive search; beam = 1 is greedy residual coding.
    Returns (codes [k][d_out][d_in/g], total error).
    """
    W = np.asarray(W, dtype=np.float64)
    codebooks = np.asarray(codebooks, dtype=np.float64)
    scales = np.asarray(scales, dtype=np.float64)
    n_cw, g = codebooks.shape[1], codebooks.shape[2]
    d_out, d_in = W.shape
    codes = np.zeros((k, d_out, d_in // g), dtype=np.int64)
    total = 0.0
    for i in range(d_out):
        for j in range(d_in // g):
            w = W[i, j * g:(j + 1) * g]
            Hj = None if H_blocks is None else H_blocks[j]
            kept = np.zeros((1, 0), dtype=np.int64)
            for m in range(k):
                ext = np.concatenate([np.repeat(kept, n_cw, axis=0),
                                      np.tile(np.arange(n_cw), len(kept))[:, None]], axis=1)
                err = _group_errors(w, codebooks, scales[i], ext, Hj)
                order = np.lexsort(tuple(ext[:, c] for c in range(ext.shape[1] - 1, -1, -1)) + (err,))
                kept = ext[order[:beam]] if m < k - 1 else ext[order[:1]]
            codes[:, i, j] = kept[0]
            total += float(_group_errors(w, codebooks, scales[i], kept, Hj)[0])
    return codes, total


def beam_search_codes_f32(W, codebooks, scales, k: int, beam: int, groups=None):
    """Beam search of App. C (code optimisation) with every comparison decided in binary32.

    The paper fixes no precision for the search. Reading: the candidate errors are evaluated
    in binary32 in one stated order, the order the GPU search uses, so that both sides take
    the same decisions. Inputs are fp16-representable values (weights, codewords, scales).

    Per group (row i, group j), with s = s_i and S_m[c][t] = s * C_m[c][t] (a product of two
    fp16 values, exact in binary32) and the residual r = w (the group's g weights):
      stage m = 0..k-1 extends every kept entry (tuple, r) by every codeword c of codebook m:
          d_t = fl32(r_t - S_m[c][t]),
          e   = fl32(...fl32(fl32(d_0 * d_0) + fl32(d_1 * d_1)) ... + fl32(d_{g-1} * d_{g-1}))
                (added left to right, no fused multiply-add);
      and keeps the `beam` candidates with the smallest e, equal e ordered by the tuple
      (lexicographically); a kept candidate's residual is its d. The last stage keeps one.
    Stage 0 starts from the single empty tuple, so it ranks the 2^B codewords of codebook 0.

    Returns (codes [k][d_out][d_in/g] int64, errors [d_out][d_in/g] float32: e of the kept
    tuple). With `groups` (an iterable of (i, j)) only those groups are searched; the others
    keep code 0 and error NaN.
    """
    f32 = np.float32
    W32 = np.asarray(W, dtype=np.float64).astype(f32)
    C32 = np.asarray(codebooks, dtype=np.float64).astype(f32)
    s32 = np.asarray(scales, dtype=np.float64).astype(f32)
    n_cw, g = C32.shape[1], C32.shape[2]
    d_out, d_in = W32.shape
    G = d_in // g
    codes = np.zeros((k, d_out, G), dtype=np.int64)
    errors = np.full((d_out, G), np.nan, dtype=f32)
    if groups is None:
        groups = [(i, j) for i in range(d_out) for j in range(G)]
    for (i, j) in groups:
        S = [s32[i] * C32[m] for m in range(k)]                   # exact products
        kept = [((), W32[i, j * g:(j + 1) * g])]                  # (tuple, residual)
        for m in range(k):
            # the kept tuples' ranks in lexicographic order: (parent rank, c) orders the
            # extended tuples lexicographically
            lex = {tup: q for q, tup in enumerate(sorted(tup for tup, _ in kept))}
            E, parent, cw = [], [], []
            for p, (tup, r) in enumerate(kept):
                D = r[None, :] - S[m]                             # [n_cw][g], binary32
                e = D[:, 0] * D[:, 0]
                for t in range(1, g):
                    e = e + D[:, t] * D[:, t]                     # binary32, left to right
                E.append(e)
                parent.append(np.full(n_cw, p))
                cw.append(np.arange(n_cw))
            E, parent, cw = np.concatenate(E), np.concatenate(parent), np.concatenate(cw)
            prank = np.array([lex[kept[p][0]] for p in parent])
            order = np.lexsort((cw, prank, E))                    # by e, then the tuple
            n_keep = beam if m < k - 1 else 1
            new = []
            for q in order[:n_keep]:
                tup, r = kept[parent[q]]
                new.append((tup + (int(cw[q]),), r - S[m][cw[q]]))  # the candidate's d
            kept = new
            best_err = E[order[0]]
        codes[:, i, j] = kept[0][0]
        errors[i, j] = best_err
    return codes, errors


def _sum_f32(terms):
    """fl32 sum of binary32 terms, left to right."""
    acc = terms[0]
    for t in terms[1:]:
        acc = np.float32(acc + t)
    return acc


def beam_search_codes_weighted_f32(W, codebooks, scales, H_blocks, k: int, beam: int, groups=None):
    """The beam search of App. C with the data-aware objective of §2.2, decisions in binary32.

    The objective of group (row i, group j) is d^T H d with H = H_jj, the g x g diagonal block of
    X X^T / n for the group's inputs (group_hessian_blocks; symmetric), and d = w - s_i sum_m C_m[c_m].
    Reading (the paper fixes no precision or evaluation order): with v = s C the scaled candidate
    codeword and r the kept tuple's residual, d^T H d = r^T H r - 2 s C^T (H r) + s^2 C^T H C, and
    both sides evaluate it in binary32 in this order, every product and sum rounded, sums left to
    right over t = 0..g-1, no fused multiply-add:
        per kept tuple:   b_t = sum_u fl(H_tu r_u),   A = sum_t fl(r_t b_t)
        per codeword:     q_t = sum_u fl(H_tu C_u),   Q = sum_t fl(C_t q_t)
        per candidate:    T = sum_t fl(C_t b_t),      e = fl(fl(A - fl(fl(2 s) T)) + fl(fl(s s) Q))
    (2 s and s s are exact for an fp16 scale). Candidates are ranked by e, equal e by the tuple
    (lexicographically); a kept tuple's residual is r - S_m[c] (S_m[c] = s C_m[c], exact; each
    subtraction rounded), as in beam_search_codes_f32. Stage 0 starts from r = w.

    Returns (codes [k][d_out][d_in/g] int64, errors [d_out][d_in/g] float32: e of the kept
    tuple). With ``groups`` only those (i, j) are searched; the others keep code 0 and error NaN.
    """
    f32 = np.float32
    W32 = np.asarray(W, dtype=np.float64).astype(f32)
    C32 = np.asarray(codebooks, dtype=np.float64).astype(f32)
    s32 = np.asarray(scales, dtype=np.float64).astype(f32)
    H32 = np.asarray(H_blocks, dtype=np.float64).astype(f32)
    n_cw, g = C32.shape[1], C32.shape[2]
    d_out, d_in = W32.shape
    G = d_in // g
    codes = np.zeros((k, d_out, G), dtype=np.int64)
    errors = np.full((d_out, G), np.nan, dtype=f32)
    if groups is None:
        groups = [(i, j) for i in range(d_out) for j in range(G)]

    def matvec(H, v):                      # [n][g] rows v -> rows of sum_u fl(H_tu v_u), t = 0..g-1
        out = np.empty_like(v)
        for t in range(g):
            out[:, t] = _sum_f32([H[t, u] * v[:, u] for u in range(g)])
        return out

    def dot(a, b):                         # rows: sum_t fl(a_t b_t), left to right
        return _sum_f32([a[:, t] * b[:, t] for t in range(g)])

    for (i, j) in groups:
        H = H32[j]
        s = s32[i]
        two_s, ss = f32(2 * s), f32(s * s)
        Q = [dot(C32[m], matvec(H, C32[m])) for m in range(k)]      # [n_cw] per codebook
        kept = [((), W32[i, j * g:(j + 1) * g])]
        for m in range(k):
            lex = {tup: q for q, tup in enumerate(sorted(tup for tup, _ in kept))}
            R = np.stack([r for _, r in kept])                        # [P][g]
            b = matvec(H, R)
            A = dot(R, b)                                             # [P]
            E, parent, cw = [], [], []
            for p in range(len(kept)):
                T = dot(C32[m], np.broadcast_to(b[p], C32[m].shape))  # [n_cw]
                e = (A[p] - two_s * T).astype(f32)
                e = (e + ss * Q[m]).astype(f32)
                E.append(e)
                parent.append(np.full(n_cw, p))
                cw.append(np.arange(n_cw))
            E, parent, cw = np.concatenate(E), np.concatenate(parent), np.concatenate(cw)
            prank = np.array([lex[kept[p][0]] for p in parent])
            order = np.lexsort((cw, prank, E))
            n_keep = beam if m < k - 1 else 1
            new = []
            for q in order[:n_keep]:
                tup, r = kept[parent[q]]
                new.append((tup + (int(cw[q]),), (r - s * C32[m][cw[q]]).astype(f32)))
            kept = new
            best_err = E[order[0]]
        codes[:, i, j] = kept[0][0]
        errors[i, j] = best_err
    return codes, errors
