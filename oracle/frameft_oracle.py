"""FrameFT reference oracle: plain, slow, fp64 CPU implementation.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library
and its Python binding) may import, call or execute this module; only the
tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` use it.  It shares no code, tables or constants with the HIP
path.  It consumes plain numpy arrays (fp64, or fp32/bf16-valued arrays that
it widens to fp64) and returns fp64 arrays.

What it computes (paper "Fine-Tuning of Transformer models with Frames"):

* ``spectral_tetris``  -- the unit-norm tight frame F of d_c vectors in C^rho_c
  built by Spectral Tetris (Sec. 3.2, "Constructing Tight Fusion Frames";
  Appendix "Fusion Frames Construction: an example", subsection Spectral
  Tetris).  The remaining row norm is carried as an exact rational.
* ``modulate``         -- modulation of F by the k-th roots of unity into k
  subspaces of C^d_c (same appendix, subsection Modulation), scaled by
  1/sqrt(k) so that the fusion frame is Parseval (Sec. 2, "We will focus on
  Parseval fusion frames").
* ``realify``          -- the entrywise real extension x+iy -> [[x,-y],[y,x]]
  (same appendix, first paragraph of subsection Spectral Tetris).
* ``tight_fusion_frame`` -- the composition, returning the real d x (k rho)
  matrix P = [P_1, ..., P_k] (Sec. 3.1, definition of P_n and P_m), with
  tightness verified rather than assumed.
* ``adapter_fwd``      -- y_a = s * P_out C P_in^T x per token (Sec. 3.1
  update equation; Algorithm 1 steps 5-6 applied to an input).
* ``adapter_bwd``      -- dX_a = s * P_in C^T P_out^T g per token and
  dC = s * (P_out^T G^T X P_in) restricted to supp(C) (Appendix A, the
  coefficient gradient grad f(C) = P_m^T grad f(W) P_n).
* ``coeff_grad_entries`` -- the same dC, but only for a chosen subset of
  support entries (for checking large problems entry by entry).
* ``merge_delta`` / ``merge_delta_rows`` -- dW = s * P_out C P_in^T
  (Algorithm 1, step 5), all rows or a chosen subset of rows.

Index conventions (the paper leaves these open; the readings are listed in
the design notes and fixed here):

* real dimensions (d, rho) correspond to complex (d/2, rho/2); d and rho even;
* complex coordinate j maps to real coordinates 2j (real part), 2j+1
  (imaginary part);
* complex frame vector (i, r) -- subspace i, F row r -- is complex column
  c = i*(rho/2) + r of the synthesis matrix and maps to real columns 2c
  (image of [Re; Im]) and 2c+1 (image of [-Im; Re]); hence real column
  i*rho + 2r + s, subspace-major, matching P = [P_1, ..., P_k];
* rows of C index columns of P_out, columns of C index columns of P_in.

Every function above is pinned by a ``-m "not gpu"`` test against something
other than itself: the paper's worked (6,3,11) example and its printed table,
textbook DFTs (numpy.fft), the k=1 special case (P = I), finite differences
and exact norm identities.  None is "parity unpinned".
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np
import scipy.sparse as sp


class NotATightFusionFrame(ValueError):
    """(k, rho, d) for which the construction does not give a tight fusion frame."""


# ---------------------------------------------------------------------------
# Frame construction
# ---------------------------------------------------------------------------

def tetris_block(x: Fraction) -> np.ndarray:
    """The 2x2 block T(x) = (1/sqrt 2) [[sqrt x, sqrt x], [sqrt(2-x), -sqrt(2-x)]].

    Appendix, subsection Spectral Tetris: T(x) T(x)^* = diag(x, 2-x), used to
    place a leftover row norm x < 1 into two columns of unit norm.
    """
    x = Fraction(x)
    a = math.sqrt(x / 2)
    b = math.sqrt((2 - x) / 2)
    return np.array([[a, a], [b, -b]], dtype=np.float64)


def spectral_tetris(rho_c: int, d_c: int) -> np.ndarray:
    """Unit-norm tight frame F (rho_c x d_c, real entries) by Spectral Tetris.

    Appendix, subsection Spectral Tetris: every row must reach the squared
    norm lam = d_c / rho_c.  Walking left to right, a row is filled with 1s
    while at least 1 of its norm is missing; a leftover x in (0, 1) is placed
    with the block T(x), whose second row starts the next row with norm 2-x
    already filled.  The leftover is held as an exact Fraction, so "exactly 1
    missing" and "nothing missing" are decided without rounding.  When a row
    ends with nothing missing, no T block is placed (reading: the paper adds
    T(x) only to fill a leftover, and its example's last row ends on 1s).
    """
    if rho_c < 1 or d_c < rho_c:
        raise NotATightFusionFrame(f"need d_c >= rho_c >= 1, got rho_c={rho_c}, d_c={d_c}")
    lam = Fraction(d_c, rho_c)
    F = np.zeros((rho_c, d_c), dtype=np.float64)
    col = 0
    carried = Fraction(0)          # norm already placed in this row by the previous T block
    for r in range(rho_c):
        missing = lam - carried
        if missing < 0:
            raise NotATightFusionFrame(f"row {r} overfilled (lam={lam} < 2 - x)")
        while missing >= 1:
            if col >= d_c:
                raise NotATightFusionFrame("ran out of columns")
            F[r, col] = 1.0
            col += 1
            missing -= 1
        if missing > 0:
            if r + 1 >= rho_c or col + 2 > d_c:
                raise NotATightFusionFrame(f"leftover {missing} in the last row")
            F[r:r + 2, col:col + 2] = tetris_block(missing)
            col += 2
            carried = 2 - missing
        else:
            carried = Fraction(0)
    if col != d_c:
        raise NotATightFusionFrame(f"filled {col} of {d_c} columns")
    return F


def modulate(F: np.ndarray, k: int) -> sp.csc_matrix:
    """Synthesis matrix Phi (d_c x k*rho_c, complex) of the modulated frame.

    Appendix, subsection Modulation: for subspace i = 0..k-1, each row r of F
    is multiplied entrywise by w_i = (e^{2 pi i i/k})^j, j = 0..d_c-1; the
    resulting vectors (one per F row) span subspace i.  Vector (i, r) becomes
    column i*rho_c + r (subspace-major, P = [P_1, ..., P_k] of Sec. 3.1) and is
    scaled by 1/sqrt(k) so that the frame operator is the identity (Parseval).
    The exponent i*j is reduced mod k before the cosine and sine.
    """
    rho_c, d_c = F.shape
    r_idx, j_idx = np.nonzero(F)
    vals = F[r_idx, j_idx]
    i_idx = np.arange(k, dtype=np.int64)
    # one entry per (nonzero of F, subspace i)
    rows = np.repeat(j_idx.astype(np.int64), k)
    cols = (np.tile(i_idx, len(j_idx)) * rho_c + np.repeat(r_idx.astype(np.int64), k))
    expo = (np.tile(i_idx, len(j_idx)) * np.repeat(j_idx.astype(np.int64), k)) % k
    phase = np.exp(2j * np.pi * expo / k)
    data = np.repeat(vals, k) * phase / math.sqrt(k)
    return sp.csc_matrix((data, (rows, cols)), shape=(d_c, k * rho_c), dtype=np.complex128)


def realify(Phi: sp.spmatrix) -> sp.csr_matrix:
    """Real extension of a complex matrix, entrywise x+iy -> [[x, -y], [y, x]].

    Appendix, subsection Spectral Tetris (first paragraph): the map doubles
    every dimension, so complex row j -> real rows 2j, 2j+1 and complex
    column c -> real columns 2c, 2c+1.
    """
    coo = Phi.tocoo()
    re, im = coo.data.real, coo.data.imag
    r2, c2 = 2 * coo.row.astype(np.int64), 2 * coo.col.astype(np.int64)
    rows = np.concatenate([r2, r2, r2 + 1, r2 + 1])
    cols = np.concatenate([c2, c2 + 1, c2, c2 + 1])
    data = np.concatenate([re, -im, im, re])
    keep = data != 0.0
    shape = (2 * Phi.shape[0], 2 * Phi.shape[1])
    return sp.csr_matrix((data[keep], (rows[keep], cols[keep])), shape=shape, dtype=np.float64)


def tight_fusion_frame(k: int, rho: int, d: int, tol: float = 1e-12) -> sp.csr_matrix:
    """Real Parseval (k, rho, d) tight fusion frame P, a d x (k*rho) sparse fp64 matrix.

    Sec. 3.2: Spectral Tetris UNTF of d_c vectors in C^rho_c, modulation by
    the k-th roots of unity, real extension.  Real (d, rho) are read as
    complex (d/2, rho/2).  Tightness is checked: P P^T must equal the identity
    (the frame operator of a Parseval fusion frame, Sec. 2.1) to ``tol``,
    otherwise NotATightFusionFrame is raised.
    """
    if k < 1 or rho < 2 or d < 2 or rho % 2 or d % 2:
        raise NotATightFusionFrame(f"need k>=1 and even rho, d >= 2; got k={k}, rho={rho}, d={d}")
    F = spectral_tetris(rho // 2, d // 2)
    P = realify(modulate(F, k))
    S = (P @ P.T).tocoo()
    diag = S.row == S.col
    off_max = np.max(np.abs(S.data[~diag]), initial=0.0)
    dvals = np.zeros(d)
    np.add.at(dvals, S.row[diag], S.data[diag])
    err = max(off_max, float(np.max(np.abs(dvals - 1.0))))
    if err > tol:
        raise NotATightFusionFrame(f"(k={k}, rho={rho}, d={d}): ||P P^T - I||_max = {err:.3e}")
    return P


def subspace_basis(P: sp.spmatrix, rho: int, i: int) -> sp.csc_matrix:
    """Columns of subspace i, the block P_i of P = [P_1, ..., P_k] (Sec. 3.1)."""
    return sp.csc_matrix(P)[:, i * rho:(i + 1) * rho]


# ---------------------------------------------------------------------------
# Adapter hot path
# ---------------------------------------------------------------------------

def _coeff_matrix(rows, cols, vals, shape) -> sp.csr_matrix:
    """Sparse C with C[rows[e], cols[e]] = vals[e] (Algorithm 1, step 4 'rearrange')."""
    rows = np.asarray(rows, dtype=np.int64)
    cols = np.asarray(cols, dtype=np.int64)
    vals = np.asarray(vals, dtype=np.float64)
    return sp.csr_matrix((vals, (rows, cols)), shape=shape)


def adapter_fwd(P_in, P_out, rows, cols, vals, scale, X) -> np.ndarray:
    """Adapter branch of the forward pass, y_a = s * P_out C P_in^T x, per token.

    Sec. 3.1: W' = W + s * P_m C P_n^T with s = alpha / sqrt(mn), so the
    adapter adds s * P_out (C (P_in^T x)) to W0 x.  X is T x n (one token per
    row); the result is T x m.  Steps: analysis z = P_in^T x (Sec. 2.1
    analysis operator), coefficient product v = C z, synthesis s * P_out v
    (Sec. 2.1 synthesis operator).
    """
    X = np.asarray(X, dtype=np.float64)
    C = _coeff_matrix(rows, cols, vals, (P_out.shape[1], P_in.shape[1]))
    Z = np.asarray((P_in.T @ X.T)).T           # T x (k rho_n)
    V = np.asarray((C @ Z.T)).T                # T x (k rho_m)
    return float(scale) * np.asarray((P_out @ V.T)).T


def adapter_bwd(P_in, P_out, rows, cols, vals, scale, X, G, nnz_chunk: int = 8192):
    """Backward of the adapter branch for upstream gradient G (T x m).

    dX_a = s * P_in C^T P_out^T g per token (chain rule through the forward).
    dC_e = s * sum_t u_t[rows[e]] * z_t[cols[e]] with u = P_out^T g and
    z = P_in^T x, i.e. s * (P_out^T G^T X P_in) at the support entries
    (Appendix A: grad f(C) = P_m^T grad f(W) P_n with grad f(W) = G^T X,
    the scalar s folded in).  Returns (dX_a: T x n, dC: nnz), dC in the
    order of the given support arrays.
    """
    X = np.asarray(X, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    rows = np.asarray(rows, dtype=np.int64)
    cols = np.asarray(cols, dtype=np.int64)
    C = _coeff_matrix(rows, cols, vals, (P_out.shape[1], P_in.shape[1]))
    U = np.asarray((P_out.T @ G.T)).T          # T x (k rho_m)
    Q = np.asarray((C.T @ U.T)).T              # T x (k rho_n)
    dX = float(scale) * np.asarray((P_in @ Q.T)).T
    Z = np.asarray((P_in.T @ X.T)).T           # T x (k rho_n)
    dC = np.empty(len(rows), dtype=np.float64)
    for e0 in range(0, len(rows), nnz_chunk):
        e1 = min(e0 + nnz_chunk, len(rows))
        dC[e0:e1] = np.sum(U[:, rows[e0:e1]] * Z[:, cols[e0:e1]], axis=0)
    return dX, float(scale) * dC


def coeff_grad_entries(P_in, P_out, rows_sub, cols_sub, scale, X, G) -> np.ndarray:
    """dC at the chosen support entries only (same definition as in adapter_bwd).

    Column b of Z = X P_in needs only column b of P_in, so a subset of
    entries is cheap even when T, n and m are large.
    """
    X = np.asarray(X, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    rows_sub = np.asarray(rows_sub, dtype=np.int64)
    cols_sub = np.asarray(cols_sub, dtype=np.int64)
    Pin_c = sp.csc_matrix(P_in)[:, cols_sub]
    Pout_c = sp.csc_matrix(P_out)[:, rows_sub]
    Zs = np.asarray((Pin_c.T @ X.T)).T         # T x |sub|
    Us = np.asarray((Pout_c.T @ G.T)).T        # T x |sub|
    return float(scale) * np.sum(Us * Zs, axis=0)


def merge_delta(P_in, P_out, rows, cols, vals, scale) -> np.ndarray:
    """Dense dW = s * P_out C P_in^T (Algorithm 1, step 5), an m x n fp64 array."""
    C = _coeff_matrix(rows, cols, vals, (P_out.shape[1], P_in.shape[1]))
    return float(scale) * (sp.csr_matrix(P_out) @ C @ sp.csr_matrix(P_in).T).toarray()


def merge_delta_rows(P_in, P_out, rows, cols, vals, scale, out_rows) -> np.ndarray:
    """Rows ``out_rows`` of dW = s * P_out C P_in^T, a len(out_rows) x n fp64 array."""
    C = _coeff_matrix(rows, cols, vals, (P_out.shape[1], P_in.shape[1]))
    Pr = sp.csr_matrix(P_out)[np.asarray(out_rows, dtype=np.int64), :]
    return float(scale) * (Pr @ C @ sp.csr_matrix(P_in).T).toarray()
