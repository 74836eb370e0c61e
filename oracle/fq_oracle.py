"""CPU float64 oracle for FrameQuant's per-layer quantization pass.

TEST INFRASTRUCTURE ONLY.  Only the tests, the package smoke check and the benchmark's
CPU-baseline leg may import this module.  It shares no code with the device library and
never calls it.

Plain numpy/LAPACK in float64.  Inputs are the exact values the device consumed (rounded
once to the device dtype, upcast exactly).  Each function follows the passage of the
paper (FrameQuant, Adepu et al., ICML 2024) named in its docstring; where the paper
defers to OPTQ/GPTQ (Frantar et al. 2023), the published algorithm is written out step by
step.  Readings of silent or garbled passages are listed where they are used:

* Alg. 1 step 3 prints "D = 2 sigma clip(...)"; read as the clip alone at
  mu +/- clip_sigmas * sigma, mu and sigma scalars over all of D, sigma with N - 1.
* The quantization grid is OPTQ's asymmetric per-row min/max grid (the paper stores a
  per-row scale and bias, appendix "Storage benefits"): lo = min(0, min row),
  hi = max(0, max row), lo = hi = 0 -> (-1, 1); scale = (hi - lo) / (2^bits - 1),
  rounded to float32 (the stored precision); zero = round-half-even(-lo / scale).
* H is the unscaled X^T X; OPTQ's damping is relative (damp * mean of the diagonal) and
  its updates are scale-free, so a constant factor on H changes nothing.
* OPTQ with act-order off, one group per row, dead columns (zero diagonal) get a unit
  diagonal and zero weights; damping damp * mean(diag) is added to the diagonal.
* Rounding is half-to-even everywhere.

Parity unpinned: the grid variant, sigma's N - 1, the rotation law of the frames and the
act-order choice are readings; the paper prints no quantized layer to pin them against.
"""
from __future__ import annotations

import numpy as np
import scipy.linalg as sla

TIE_EPS = 1e-6


# --------------------------------------------------------------------------- operators
def frame_analysis_vectors(X, P):
    """Analysis operator of the fusion frame on each row x of X (Sec. 2 "Operators in Fusion
    Frames"): the dot products of x with every column of P = [w_1 P_1 ... w_k P_k], i.e. the
    rows P^T x, stacked: U = X P.  X: n x d; U: n x (k rho)."""
    return np.asarray(X, dtype=np.float64) @ np.asarray(P, dtype=np.float64)


def frame_synthesis_vectors(U, P):
    """Synthesis operator (the adjoint of the analysis operator, same passage) on each row
    u of U: sum_i w_i P_i u_i = P u, stacked: Y = U P^T.  U: n x (k rho); Y: n x d."""
    return np.asarray(U, dtype=np.float64) @ np.asarray(P, dtype=np.float64).T


# --------------------------------------------------------------------------- stage 1
def hessian(X_chunks) -> np.ndarray:
    """Calibration Hessian H = X^T X = A_prev A_prev^T (Sec. 3, proxy loss: the FF-space
    Hessian is C C^T with C = P_prev^T A_prev, so C C^T = P_prev^T (X^T X) P_prev).

    X_chunks: one (n x d_in) array or an iterable of row chunks; summed in float64.
    """
    if isinstance(X_chunks, np.ndarray):
        X_chunks = [X_chunks]
    H = None
    for X in X_chunks:
        X = np.asarray(X, dtype=np.float64)
        G = X.T @ X
        H = G if H is None else H + G
    return H


# --------------------------------------------------------------------------- stage 2
def frame_analysis(W, P_out, P_in, H):
    """FF-space weights and Hessian (Sec. 3; Alg. 1 step 1):
    D = P_l^T Theta P_prev and H~ = P_prev^T H P_prev (= C_prev C_prev^T)."""
    W = np.asarray(W, dtype=np.float64)
    P_out = np.asarray(P_out, dtype=np.float64)
    P_in = np.asarray(P_in, dtype=np.float64)
    D = P_out.T @ W @ P_in
    Ht = None if H is None else P_in.T @ np.asarray(H, dtype=np.float64) @ P_in
    return D, Ht


# --------------------------------------------------------------------------- stage 3a
def clip_bounds(D, clip_sigmas: float = 2.0):
    """mu = mean(D), sigma = std(D) (ddof 1) over the whole matrix; the clip interval
    [mu - c sigma, mu + c sigma] (Alg. 1 steps 2-3; Sec. 3, clipping at 2 sigma)."""
    D = np.asarray(D, dtype=np.float64)
    mu = D.mean()
    sigma = D.std(ddof=1) if D.size > 1 else 0.0
    return mu, sigma, mu - clip_sigmas * sigma, mu + clip_sigmas * sigma


def apply_clip(D, lo_b: float, hi_b: float):
    return np.minimum(np.maximum(np.asarray(D, dtype=np.float64), lo_b), hi_b)


def row_grid(D, bits: int = 2):
    """Per-row asymmetric min/max grid (OPTQ's quantizer; per-row scale and bias stored
    with the codes, appendix "Storage benefits").  Returns (scale, zero) as float64
    holding the float32 scale and the integer zero point."""
    D = np.asarray(D, dtype=np.float64)
    maxq = 2 ** bits - 1
    lo = np.minimum(D.min(axis=1), 0.0)
    hi = np.maximum(D.max(axis=1), 0.0)
    both0 = (lo == 0) & (hi == 0)
    lo = np.where(both0, -1.0, lo)
    hi = np.where(both0, 1.0, hi)
    scale = ((hi - lo) / maxq).astype(np.float32).astype(np.float64)
    zero = np.round(-lo / scale)
    return scale, zero


def rtn_codes(x, scale, zero, bits: int = 2):
    """Round to nearest on the grid: code = clamp(rne(x / scale) + zero, 0, 2^bits - 1).
    Also returns the pre-rounding value t = x / scale in code units."""
    maxq = 2 ** bits - 1
    t = x / scale
    q = np.clip(np.round(t) + zero, 0, maxq)
    return q, t


def near_tie(t, eps: float = TIE_EPS):
    """|frac(t) - 1/2| < eps: t lies within eps of a rounding boundary."""
    return np.abs((t - np.floor(t)) - 0.5) < eps


# --------------------------------------------------------------------------- stage 3b
def damped_hessian(Ht, damp: float = 0.01):
    """OPTQ's conditioning of the FF Hessian: dead columns (H~_jj = 0) get H~_jj = 1, then
    damp * mean(diag) is added to the diagonal.  Returns (damped H~, dead mask)."""
    H = np.array(Ht, dtype=np.float64, copy=True)
    dead = np.diag(H) == 0
    H[dead, dead] = 1.0
    lam = damp * np.mean(np.diag(H))
    H[np.diag_indices_from(H)] += lam
    return H, dead


def gptq_prepare(Ht, damp: float = 0.01):
    """OPTQ preparation on the FF Hessian (Sec. 3, "quantize(D, C, B) // modified GPTQ"):
    dead columns (H~_jj = 0) get H~_jj = 1; H~ += damp * mean(diag H~) I;
    U = upper Cholesky factor of H~^{-1} (U^T U = H~^{-1}).
    Returns (U, dead mask, damped H~).  Raises numpy.linalg.LinAlgError when the damped
    H~ is not positive definite."""
    H, dead = damped_hessian(Ht, damp)
    L = np.linalg.cholesky(H)                       # H = L L^T
    Linv = sla.solve_triangular(L, np.eye(H.shape[0]), lower=True)
    Hinv = Linv.T @ Linv                            # H^{-1}
    Hinv = 0.5 * (Hinv + Hinv.T)
    U = np.linalg.cholesky(Hinv).T                  # U^T U = H^{-1}
    return U, dead, H


# --------------------------------------------------------------------------- stage 3c/3d
def gptq(D, U, scale, zero, bits: int = 2, block: int = 128, dead=None,
         forced_codes=None, tie_eps: float = TIE_EPS):
    """OPTQ's column-sequential rounding with Cholesky error feedback and lazy block
    updates (Alg. 1 step 4).  For each block [i1, i2) of width `block`, for each column j
    in order: q = grid-round(w_j); err = (w_j - dq) / U_jj; later columns of the block
    w_l -= err * U_jl; after the block, columns >= i2 get -= E_block @ U[i1:i2, i2:].

    forced_codes (same shape as D): where the pre-rounding value is within tie_eps of a
    rounding boundary, adopt that code instead of the oracle's own (teacher forcing).
    Returns dict(codes, t, tie, E)."""
    W = np.array(D, dtype=np.float64, copy=True)
    if dead is not None:
        W[:, dead] = 0.0
    rows, n = W.shape
    maxq = 2 ** bits - 1
    codes = np.zeros((rows, n), dtype=np.int64)
    tvals = np.zeros((rows, n))
    ties = np.zeros((rows, n), dtype=bool)
    E = np.zeros((rows, n))
    for i1 in range(0, n, block):
        i2 = min(i1 + block, n)
        W1 = W[:, i1:i2].copy()
        E1 = np.zeros((rows, i2 - i1))
        for jj in range(i2 - i1):
            j = i1 + jj
            w = W1[:, jj]
            q, t = rtn_codes(w, scale, zero, bits)
            tie = near_tie(t, tie_eps)
            if forced_codes is not None:
                q = np.where(tie, forced_codes[:, j], q)
            q = np.clip(q, 0, maxq)
            dq = scale * (q - zero)
            err = (w - dq) / U[j, j]
            W1[:, jj:] -= np.outer(err, U[j, j:i2])
            E1[:, jj] = err
            codes[:, j] = q
            tvals[:, j] = t
            ties[:, j] = tie
        W[:, i2:] -= E1 @ U[i1:i2, i2:]
        E[:, i1:i2] = E1
    return {"codes": codes, "t": tvals, "tie": ties, "E": E}


def gptq_obs(D, Hd, scale, zero, bits: int = 2, dead=None):
    """Second, independent formulation (optimal brain surgeon form): for column j the
    inverse S of the trailing damped Hessian block H[j:, j:] gives err = (w - dq) / S_00
    and the update D[:, j:] -= err * S[0, :]; S is downdated by one Schur step."""
    W = np.array(D, dtype=np.float64, copy=True)
    if dead is not None:
        W[:, dead] = 0.0
    n = W.shape[1]
    S = np.linalg.inv(np.asarray(Hd, dtype=np.float64))
    codes = np.zeros(W.shape, dtype=np.int64)
    for j in range(n):
        w = W[:, j]
        q, _ = rtn_codes(w, scale, zero, bits)
        dq = scale * (q - zero)
        err = (w - dq) / S[0, 0]
        W[:, j:] -= np.outer(err, S[0, :])
        codes[:, j] = q
        S = S[1:, 1:] - np.outer(S[1:, 0], S[0, 1:]) / S[0, 0]
    return codes


def gptq_tail_pre_rounding(Dc, dq, Ht, first: int, damp: float = 0.01):
    """OPTQ's pre-rounding values w_j of the trailing columns j >= first, given the
    dequantized values dq of every column: the consistency property of Alg. 1 step 4
    that each code is the grid point nearest to its w_j, usable where a full replay
    (a factorization of all of H~) is too large.

    The feedback gives D - DQ = E U (E the column errors, U^T U = H^{-1}, U upper), so
    w_j = DQ_j + E_j U_jj.  Writing the damped H~ = M M^T with M upper (M = J L J, L the
    lower factor of the reversed J H~ J), U = M^{-1}; hence E = (D - DQ) M and
    w_j = DQ_j + E_j / M_jj.  The columns j >= first of M are the leading n - first columns
    of L, read backwards, so only a panel of the factorization is formed.
    Dc: clipped D (rows x n); dead columns are zeroed here as in gptq."""
    D = np.array(Dc, dtype=np.float64, copy=True)
    H, dead = damped_hessian(Ht, damp)
    D[:, dead] = 0.0
    n = H.shape[0]
    p = n - first
    A = np.ascontiguousarray(H[::-1, ::-1])             # J H~ J
    del H
    # LAPACK's Cholesky on the leading block (symmetric, so its transpose is the same
    # matrix in column-major order and is factored in place; the upper triangle of the
    # result is not part of the factor)
    L11, info = sla.lapack.dpotrf(A[:p, :p].T, lower=1, clean=1, overwrite_a=1)
    if info != 0:
        raise np.linalg.LinAlgError("damped H~ is not positive definite")
    if p < n:
        L21 = sla.solve_triangular(L11, A[p:, :p].T, lower=True).T
        Lp = np.vstack([L11, L21])                      # leading p columns of L
    else:
        Lp = L11
    del A
    # columns first..n-1 of M are Mt = Lp[::-1, ::-1], so E = X Mt with X = D - DQ is
    # (X[:, ::-1] Lp)[:, ::-1]: the product reads Lp in its stored order
    X = D - np.asarray(dq, dtype=np.float64)
    E = (np.ascontiguousarray(X[:, ::-1]) @ Lp)[:, ::-1]   # E_j for j >= first
    diag = Lp[n - 1 - first - np.arange(p), p - 1 - np.arange(p)]
    return np.asarray(dq, dtype=np.float64)[:, first:] + E / diag[None, :]


def dequant(codes, scale, zero):
    """D^ = scale * (q - zero) per row (appendix "Storage benefits": codes plus a
    per-row scale and bias)."""
    return np.asarray(scale)[:, None] * (np.asarray(codes, dtype=np.float64) - np.asarray(zero)[:, None])


def proxy_loss(D, Dhat, H):
    """L(D^) = tr((D - D^) H (D - D^)^T) (Sec. 3, proxy loss in FF space)."""
    R = np.asarray(D, dtype=np.float64) - np.asarray(Dhat, dtype=np.float64)
    return float(np.einsum("ij,jk,ik->", R, H, R))


# --------------------------------------------------------------------------- filter
def wiener_row_gains(D, Dhat, Ht):
    """Diagonal approximation of the Wiener (linear MMSE) filter at synthesis (appendix
    "LMMSE estimation from fusion frame measurements"; Sec. 3 "Robustness of Fusion
    Frames" (b)).  The layer output is Z = P_l D C (C = P_prev^T A_prev, H~ = C C^T); the
    filter replaces the synthesis P_l D^ C by F D^ C.  Reading: F = P_l diag(g), one gain
    per frame-coefficient row, each minimising the row's share of the output error on the
    calibration set, ||(D_i - g_i D^_i) C||^2, i.e.
        g_i = (D H~ D^^T)_ii / (D^ H~ D^^T)_ii,
    with D the unclipped analysis output (the only D with P_l D C = Theta A_prev).  A
    row with (D^ H~ D^^T)_ii = 0 keeps g_i = 1.  The gains fold into the stored per-row
    scale (scale_i g_i), so synthesis and inference are unchanged."""
    D = np.asarray(D, dtype=np.float64)
    Dh = np.asarray(Dhat, dtype=np.float64)
    M = Dh @ np.asarray(Ht, dtype=np.float64)            # D^ H~
    num = np.einsum("ij,ij->i", D, M)
    den = np.einsum("ij,ij->i", Dh, M)
    g = np.ones(D.shape[0])
    ok = den != 0
    g[ok] = num[ok] / den[ok]
    return g


# --------------------------------------------------------------------------- stage 3e
def pack2(codes) -> np.ndarray:
    """2-bit codes -> uint32 words, 16 codes per word, row-major; column j sits in bits
    2*(j mod 16) .. 2*(j mod 16)+1 of word floor(j / 16); pad bits are zero."""
    c = np.asarray(codes, dtype=np.uint64)
    rows, n = c.shape
    nw = (n + 15) // 16
    padded = np.zeros((rows, nw * 16), dtype=np.uint64)
    padded[:, :n] = c
    padded = padded.reshape(rows, nw, 16)
    shifts = (2 * np.arange(16, dtype=np.uint64))[None, None, :]
    return np.bitwise_or.reduce(padded << shifts, axis=2).astype(np.uint32)


def unpack2(words, n: int) -> np.ndarray:
    w = np.asarray(words, dtype=np.uint64)
    shifts = (2 * np.arange(16, dtype=np.uint64))[None, None, :]
    c = (w[:, :, None] >> shifts) & np.uint64(3)
    return c.reshape(w.shape[0], -1)[:, :n].astype(np.int64)


def codes_per_word(bits: int) -> int:
    """b-bit codes per uint32 word: floor(32 / b) (16, 10, 8 for 2, 3, 4 bits)."""
    return 32 // bits


def pack_bits(codes, bits: int) -> np.ndarray:
    """b-bit codes -> uint32 words, floor(32/b) codes per word, row-major; column j sits in
    bits b*(j mod cpw) .. b*(j mod cpw)+b-1 of word floor(j / cpw); pad bits are zero (the
    storage appendix keeps the codes of D^ plus a per-row scale and bias)."""
    cpw = codes_per_word(bits)
    c = np.asarray(codes, dtype=np.uint64)
    rows, n = c.shape
    nw = (n + cpw - 1) // cpw
    padded = np.zeros((rows, nw * cpw), dtype=np.uint64)
    padded[:, :n] = c
    shifts = (bits * np.arange(cpw, dtype=np.uint64))[None, None, :]
    return np.bitwise_or.reduce(padded.reshape(rows, nw, cpw) << shifts, axis=2).astype(np.uint32)


def unpack_bits(words, n: int, bits: int) -> np.ndarray:
    cpw = codes_per_word(bits)
    w = np.asarray(words, dtype=np.uint64)
    shifts = (bits * np.arange(cpw, dtype=np.uint64))[None, None, :]
    c = (w[:, :, None] >> shifts) & np.uint64((1 << bits) - 1)
    return c.reshape(w.shape[0], -1)[:, :n].astype(np.int64)


# --------------------------------------------------------------------------- stage 4
def synthesis(codes, scale, zero, P_out, P_in):
    """Reconstructed weights Theta^ = P_l D^ P_prev^T (Alg. 1 return value without the
    activations; appendix "Computational Complexity during Inference")."""
    Dhat = dequant(codes, scale, zero)
    return np.asarray(P_out, dtype=np.float64) @ Dhat @ np.asarray(P_in, dtype=np.float64).T


def frame_apply(X, codes, scale, zero, P_out, P_in):
    """Layer outputs of the quantized layer (Sec. 3 "Inference Procedure"), by their plain
    definition Y = X Theta^T with Theta^ = P_l D^ P_prev^T (appendix "Computational
    Complexity during Inference").  X: tokens x d_in; Y: tokens x d_out."""
    Wh = synthesis(codes, scale, zero, P_out, P_in)
    return np.asarray(X, dtype=np.float64) @ Wh.T


# --------------------------------------------------------------------------- activations
def activation_rtn(C, bits: int = 8):
    """Round-to-nearest of the frame representation of activations (appendix "FrameQuant
    for Activation Quantization?": C^ = round(C / Delta_C), Delta_C = max|C| /
    (2^(N-1) - 1)), one Delta per token (row of C: the per-token form the same passage
    names as the one that admits integer matrix products).  The decision is taken in
    float32, the precision the device computes C in: Delta = float32(max|C_t|) / float32(qmax)
    and C / Delta are float32 divisions; ties go to even.  A token with max|C_t| = 0 gets
    Delta = 0 and C^ = 0.  Returns (C^ as int64, Delta as float32)."""
    C = np.asarray(C, dtype=np.float32)
    qmax = np.float32(2 ** (bits - 1) - 1)
    mx = np.max(np.abs(C), axis=1) if C.shape[1] else np.zeros(C.shape[0], np.float32)
    delta = (mx / qmax).astype(np.float32)
    Cq = np.zeros(C.shape, dtype=np.int64)
    nz = delta > 0
    Cq[nz] = np.rint(C[nz] / delta[nz, None]).astype(np.int64)
    return Cq, delta


def frame_apply_rtn_activations(C, codes, scale, zero, P_out, bits: int = 8):
    """Layer outputs from the rounded frame representation of the inputs (same appendix;
    Sec. 3 "Inference Procedure" for the rest): C^, Delta = activation_rtn(C), then
    V = Delta * C^ (q - zero)^T diag(scale) and Y = V P_l^T, in float64.  C: tokens x K_in
    (the analysis X P_prev as the device computed it)."""
    Cq, delta = activation_rtn(C, bits)
    V = (delta.astype(np.float64)[:, None] * Cq.astype(np.float64)) @ dequant(codes, scale, zero).T
    return V @ np.asarray(P_out, dtype=np.float64).T


# --------------------------------------------------------------------------- pipeline
def quantize_frames(D, Ht, bits=2, block=128, damp=0.01, clip_sigmas=2.0,
                    forced_codes=None, tie_eps=TIE_EPS):
    """Alg. 1 steps 2-4 on FF-space inputs: clip, per-row grid, OPTQ rounding."""
    mu, sigma, lo_b, hi_b = clip_bounds(D, clip_sigmas)
    Dc = apply_clip(D, lo_b, hi_b)
    scale, zero = row_grid(Dc, bits)
    U, dead, Hd = gptq_prepare(Ht, damp)
    r = gptq(Dc, U, scale, zero, bits, block, dead, forced_codes, tie_eps)
    r.update(scale=scale, zero=zero, mu=mu, sigma=sigma, Dc=Dc, U=U, dead=dead, Hd=Hd)
    return r


def quantize_layer(W, X_chunks, P_out, P_in, bits=2, block=128, damp=0.01,
                   clip_sigmas=2.0, H=None):
    """The whole per-layer pass (Alg. 1): H, analysis, clip, OPTQ, pack, synthesis."""
    if H is None:
        H = hessian(X_chunks)
    D, Ht = frame_analysis(W, P_out, P_in, H)
    r = quantize_frames(D, Ht, bits, block, damp, clip_sigmas)
    r["H"], r["D"], r["Ht"] = H, D, Ht
    r["packed"] = pack2(r["codes"])
    r["W_hat"] = synthesis(r["codes"], r["scale"], r["zero"], P_out, P_in)
    return r


# --------------------------------------------------------------------------- frame choice
def spectral_tetris_untf(rho_c: int, d_c: int):
    """Spectral tetris (appendix "Synopsis of Construction of Tight Fusion Frames"): a
    rho_c x d_c matrix F whose d_c columns are unit vectors and whose rows are orthogonal
    with squared norm d_c / rho_c (a unit-norm tight frame for C^rho_c), or None when the
    construction does not go through.  Rows are filled left to right; a row takes 1s while
    it still lacks at least 1 of squared norm; a remainder 0 < x < 1 is placed with the
    2 x 2 block [[sqrt(x/2), sqrt(x/2)], [sqrt(1-x/2), -sqrt(1-x/2)]] on this row and the
    next, which then lacks 2 - x less.  The bookkeeping is exact (fractions)."""
    from fractions import Fraction
    if rho_c < 1 or d_c < rho_c:
        return None
    F = np.zeros((rho_c, d_c))
    target = Fraction(d_c, rho_c)
    j = 0
    given = Fraction(0)                 # squared norm the row already has from a block
    for r in range(rho_c):
        need = target - given
        given = Fraction(0)
        if need < 0:
            return None
        while need >= 1:
            if j >= d_c:
                return None
            F[r, j] = 1.0
            j += 1
            need -= 1
        if need > 0:
            if r + 1 >= rho_c or j + 2 > d_c:
                return None
            a, b = np.sqrt(float(need) / 2.0), np.sqrt(1.0 - float(need) / 2.0)
            F[r, j], F[r, j + 1] = a, a
            F[r + 1, j], F[r + 1, j + 1] = b, -b
            j += 2
            given = 2 - need
    return F if j == d_c else None


def modulated_frame_is_tight(F, k: int, tol: float = 1e-9) -> bool:
    """The fusion frame of Sec. 2.2 built from F: subspace s (s < k) is spanned by the rows
    of F multiplied entrywise by (w^(j s))_j, w = exp(2 pi i / k).  By definition it is a
    tight fusion frame when each subspace's rows, divided by sqrt(d_c / rho_c), form an
    orthonormal basis and the sum of the k orthogonal projections is (k rho_c / d_c) I."""
    rho_c, d_c = F.shape
    jj = np.arange(d_c)
    S = np.zeros((d_c, d_c), dtype=np.complex128)
    for s in range(k):
        B = F * np.exp(2j * np.pi * s * jj / k)[None, :] / np.sqrt(d_c / rho_c)
        if np.abs(B @ B.conj().T - np.eye(rho_c)).max() > tol:
            return False
        S += B.conj().T @ B
    return np.abs(S - (k * rho_c / d_c) * np.eye(d_c)).max() <= tol


def tff_frame_valid(d: int, k: int, rho: int) -> bool:
    """A real (k, rho, d) frame by realification of the complex (k, rho/2, d/2) one exists
    by this construction when d and rho are even, spectral tetris goes through for
    (rho/2, d/2) and the modulation is tight (checked by its definition)."""
    if d % 2 or rho % 2 or k < 1 or d < 2 or rho < 2:
        return False
    F = spectral_tetris_untf(rho // 2, d // 2)
    return F is not None and modulated_frame_is_tight(F, k)


def untf_max_row_support(F) -> int:
    """Length of the longest run of columns from a row's first nonzero to its last."""
    best = 0
    for row in F:
        nz = np.flatnonzero(row)
        best = max(best, int(nz[-1] - nz[0] + 1))
    return best


def tff_choose_k(d: int, r: float, rho: int, valid=None) -> int:
    """The constructible frame nearest a requested redundancy r = k rho / d (Sec. 2.2
    remarks: take a valid (k, rho), else a lower redundancy): k = round(r d / rho), ties to
    even, lowered until valid.  valid: the validity test (default: by definition, small d
    only); returns 0 when no k >= 1 is valid."""
    valid = valid or tff_frame_valid
    k = int(round(r * d / rho))
    while k >= 1 and not valid(d, k, rho):
        k -= 1
    return max(k, 0)


# --------------------------------------------------------------------------- seeded rotation
# The rotation factors of a frame drawn from a 64-bit seed (Sec. 2.2 and the appendix on
# constructing TFFs take a random rotation; the storage appendix keeps only (k, rho, d)
# and what regenerates the rotation).  Recipe (a reading: the paper names no generator):
#   * Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC'11), key = (seed mod 2^32,
#     seed div 2^32), counter = (p mod 2^32, p div 2^32, f, 0) for pair p of factor f;
#   * its 4 output words (x0, x1, x2, x3) give u1 from (x0, x1) and u2 from (x2, x3):
#     u = (2^21 x_odd + floor(x_even / 2^11) + 1/2) / 2^53, in (0, 1);
#   * Box-Muller: entries 2p and 2p + 1 of the row-major n x n matrix G are
#     sqrt(-2 ln u1) cos(2 pi u2) and sqrt(-2 ln u1) sin(2 pi u2);
#   * the factor is Q of G = Q R with R's diagonal made positive (the signs of R's
#     diagonal moved into Q), a Haar-distributed orthogonal matrix.
PHILOX_M = (0xD2511F53, 0xCD9E8D57)
PHILOX_W = (0x9E3779B9, 0xBB67AE85)


def philox4x32_10(counters, key):
    """Philox4x32 with 10 rounds on an (N, 4) array of uint32 counters and a key of two
    uint32 words (Salmon et al., SC'11): each round multiplies words 0 and 2 by the two
    multipliers, mixes the halves of the products with words 1, 3 and the key, and the
    key is bumped by the two Weyl constants between rounds."""
    c = np.asarray(counters, dtype=np.uint64).reshape(-1, 4).copy()
    k0, k1 = np.uint64(key[0]), np.uint64(key[1])
    mask = np.uint64(0xFFFFFFFF)
    for _ in range(10):
        p0 = np.uint64(PHILOX_M[0]) * c[:, 0]
        p1 = np.uint64(PHILOX_M[1]) * c[:, 2]
        hi0, lo0 = p0 >> np.uint64(32), p0 & mask
        hi1, lo1 = p1 >> np.uint64(32), p1 & mask
        c = np.stack([(hi1 ^ c[:, 1] ^ k0) & mask, lo1, (hi0 ^ c[:, 3] ^ k1) & mask, lo0], axis=1)
        k0 = (k0 + np.uint64(PHILOX_W[0])) & mask
        k1 = (k1 + np.uint64(PHILOX_W[1])) & mask
    return c.astype(np.uint32)


def seeded_gaussian(seed: int, f: int, n: int) -> np.ndarray:
    """The n x n Gaussian matrix of factor f drawn from `seed` by the recipe above."""
    total = n * n
    npair = (total + 1) // 2
    p = np.arange(npair, dtype=np.uint64)
    ctr = np.stack([p & np.uint64(0xFFFFFFFF), p >> np.uint64(32),
                    np.full(npair, f, np.uint64), np.zeros(npair, np.uint64)], axis=1)
    x = philox4x32_10(ctr, (seed & 0xFFFFFFFF, seed >> 32)).astype(np.uint64)

    def unif(lo_w, hi_w):
        m = (hi_w << np.uint64(21)) | (lo_w >> np.uint64(11))
        return (m.astype(np.float64) + 0.5) / 2.0 ** 53

    u1, u2 = unif(x[:, 0], x[:, 1]), unif(x[:, 2], x[:, 3])
    rad = np.sqrt(-2.0 * np.log(u1))
    g = np.empty(2 * npair)
    g[0::2] = rad * np.cos(2.0 * np.pi * u2)
    g[1::2] = rad * np.sin(2.0 * np.pi * u2)
    return g[:total].reshape(n, n)


def seeded_haar(seed: int, f: int, n: int) -> np.ndarray:
    """Factor f (0: R1, 1: R2) of the rotation drawn from `seed`: Q of the QR of the
    seeded Gaussian matrix with R's diagonal made positive (LAPACK QR; the positive-
    diagonal QR is unique, so any QR algorithm gives the same Q)."""
    G = seeded_gaussian(seed, f, n)
    Q, R = np.linalg.qr(G)
    sg = np.sign(np.diag(R))
    sg[sg == 0] = 1.0
    return Q * sg[None, :]
