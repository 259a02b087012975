"""Pins for the fp64 oracle: each check compares it with something other than itself.

* the paper's worked (6,3,11) example: the Spectral Tetris matrix F and the
  printed table of modulated vectors (fixtures under tests/golden/);
* the defining properties of the objects (unit-norm tight frame, T(x) T(x)^*,
  Parseval fusion frame with subspace projectors computed by QR);
* textbook routines: numpy.fft.fft / ifft (an integer-lambda frame acts blockwise
  as the unitary DFT), and the k = 1 case where P = I and the adapter is a
  plain sparse matrix product;
* finite differences of the forward pass for both gradients;
* exact norm identities of orthogonal frames.
"""
import math
import os
import re
from fractions import Fraction

import numpy as np
import pytest

from oracle import frameft_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _parse_entry(tok: str) -> complex:
    if tok == "0":
        return 0.0
    m = re.fullmatch(r"(-?)sqrt\((\d+)/(\d+)\)(?:\*w\^(\d+))?", tok)
    assert m, tok
    sign = -1.0 if m.group(1) else 1.0
    mag = math.sqrt(int(m.group(2)) / int(m.group(3)))
    e = int(m.group(4)) if m.group(4) else 0
    return sign * mag * np.exp(1j * np.pi * e / 3.0)   # w = e^{i pi/3}


def _load(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            rows.append([_parse_entry(t) for t in line.split()])
    return np.array(rows)


# ---------------------------------------------------------------- Spectral Tetris

def test_spectral_tetris_matches_worked_example():
    want = _load("spectral_tetris_F_3x11.txt").real
    got = O.spectral_tetris(3, 11)
    assert got.shape == (3, 11)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-15)


@pytest.mark.parametrize("x", [Fraction(1, 3), Fraction(2, 3), Fraction(1, 2), Fraction(7, 9)])
def test_tetris_block_identity(x):
    T = O.tetris_block(x)
    np.testing.assert_allclose(T @ T.T, np.diag([float(x), float(2 - x)]), atol=1e-15)


@pytest.mark.parametrize("rho_c,d_c", [(3, 11), (2, 3), (5, 12), (7, 23), (8, 128), (32, 2048),
                                       (32, 5504), (64, 14336), (4, 4), (6, 6)])
def test_spectral_tetris_is_unit_norm_tight_frame(rho_c, d_c):
    F = O.spectral_tetris(rho_c, d_c)
    np.testing.assert_allclose(np.sum(F * F, axis=0), 1.0, atol=1e-14)
    np.testing.assert_allclose(F @ F.T, (d_c / rho_c) * np.eye(rho_c), atol=1e-12)
    assert np.max(np.count_nonzero(F, axis=0)) <= 2


def test_spectral_tetris_integer_lambda_is_block_of_ones():
    # lam = d_c / rho_c integer: no leftover ever appears, row r holds ones at r*lam .. r*lam+lam-1
    F = O.spectral_tetris(4, 24)
    want = np.kron(np.eye(4), np.ones((1, 6)))
    np.testing.assert_array_equal(F, want)


# ---------------------------------------------------------------- modulation / table

def test_modulation_matches_paper_table():
    table = _load("tff_6_3_11_table.txt")            # 18 x 11, row r*6 + i = vector (i, r)
    Phi = O.modulate(O.spectral_tetris(3, 11), 6).toarray() * math.sqrt(6)   # undo Parseval scaling
    assert Phi.shape == (11, 18)
    for r in range(3):
        for i in range(6):
            np.testing.assert_allclose(Phi[:, i * 3 + r], table[r * 6 + i], atol=1e-14,
                                       err_msg=f"vector (i={i}, r={r})")


# ---------------------------------------------------------------- fusion frame

FRAMES = [(6, 6, 22), (2, 4, 8), (1, 8, 8), (4, 12, 48), (5, 8, 40), (16, 16, 256),
          (3, 10, 30), (12, 64, 768), (36, 64, 2304)]


@pytest.mark.parametrize("k,rho,d", FRAMES)
def test_parseval_and_subspace_projectors(k, rho, d):
    P = O.tight_fusion_frame(k, rho, d).toarray()
    assert P.shape == (d, k * rho)
    np.testing.assert_allclose(P @ P.T, np.eye(d), atol=1e-12)
    lam = Fraction(d, rho)
    S = np.zeros((d, d))
    for i in range(k):
        Pi = P[:, i * rho:(i + 1) * rho]
        # basis of subspace i is orthogonal with squared norm lam / k
        np.testing.assert_allclose(Pi.T @ Pi, float(lam / k) * np.eye(rho), atol=1e-12)
        # orthogonal projector onto span(P_i) from an independent QR factorisation
        Qf, _ = np.linalg.qr(Pi)
        S += float(lam / k) * (Qf @ Qf.T)
    # fusion frame operator sum_i w_i^2 pi_i with w_i^2 = lam / k equals the identity
    np.testing.assert_allclose(S, np.eye(d), atol=1e-11)


def test_analysis_preserves_norm():
    g = np.random.default_rng(3)
    for (k, rho, d) in [(6, 6, 22), (4, 12, 48), (64, 64, 4096)]:
        P = O.tight_fusion_frame(k, rho, d)
        x = g.standard_normal((5, d))
        z = np.asarray(P.T @ x.T).T
        np.testing.assert_allclose(np.linalg.norm(z, axis=1), np.linalg.norm(x, axis=1), rtol=1e-12)


def test_not_a_tight_fusion_frame_is_rejected():
    with pytest.raises(O.NotATightFusionFrame):
        O.tight_fusion_frame(2, 4, 10)      # columns j and j+2 of F share a row
    with pytest.raises(O.NotATightFusionFrame):
        O.tight_fusion_frame(4, 3, 12)      # odd real subspace dimension
    with pytest.raises(O.NotATightFusionFrame):
        O.spectral_tetris(4, 3)             # fewer vectors than the dimension


# ---------------------------------------------------------------- textbook DFT route

def fft_analysis(x, k, rho):
    """z = P^T x for k*rho = d via numpy's unitary DFT, written into the canonical index i*rho+2r+s."""
    d = x.shape[-1]
    rho_c = rho // 2
    xc = x[..., 0::2] + 1j * x[..., 1::2]
    Zc = np.fft.fft(xc.reshape(x.shape[:-1] + (rho_c, k)), axis=-1, norm="ortho")   # [r, i]
    Zc = np.swapaxes(Zc, -1, -2).reshape(x.shape[:-1] + (d // 2,))                   # [i, r]
    z = np.empty(x.shape)
    z[..., 0::2], z[..., 1::2] = Zc.real, Zc.imag
    return z


def fft_synthesis(v, k, rho):
    """P v for k*rho = d via numpy's unitary inverse DFT."""
    d = v.shape[-1]
    rho_c = rho // 2
    vc = (v[..., 0::2] + 1j * v[..., 1::2]).reshape(v.shape[:-1] + (k, rho_c))        # [i, r]
    xc = np.fft.ifft(np.swapaxes(vc, -1, -2), axis=-1, norm="ortho")                   # [r, tau]
    xc = xc.reshape(v.shape[:-1] + (d // 2,))
    x = np.empty(v.shape)
    x[..., 0::2], x[..., 1::2] = xc.real, xc.imag
    return x


@pytest.mark.parametrize("k,rho,d", [(16, 16, 256), (64, 64, 4096), (172, 64, 11008), (12, 64, 768),
                                     (36, 64, 2304), (1, 8, 8), (4, 2, 8), (64, 128, 8192)])
def test_integer_lambda_frame_is_blockwise_unitary_dft(k, rho, d):
    P = O.tight_fusion_frame(k, rho, d)
    x = np.random.default_rng(k + d).standard_normal((3, d))
    np.testing.assert_allclose(np.asarray(P.T @ x.T).T, fft_analysis(x, k, rho), atol=1e-12)
    v = np.random.default_rng(k * d).standard_normal((3, d))
    np.testing.assert_allclose(np.asarray(P @ v.T).T, fft_synthesis(v, k, rho), atol=1e-12)


def _problem(seed, n, m, nnz, T):
    g = np.random.default_rng(seed)
    flat = g.choice(m * n, size=nnz, replace=False)
    rows, cols = flat // n, flat % n
    vals = g.standard_normal(nnz) * 0.02
    X = g.standard_normal((T, n))
    G = g.standard_normal((T, m))
    return rows, cols, vals, X, G


@pytest.mark.parametrize("fin,fout,nnz", [((4, 12, 48), (5, 8, 40), 300), ((16, 16, 256), (16, 16, 256), 512),
                                          ((12, 64, 768), (36, 64, 2304), 3000)])
def test_adapter_matches_textbook_dft_route(fin, fout, nnz):
    (kn, rn, n), (km, rm, m) = fin, fout
    Pin, Pout = O.tight_fusion_frame(kn, rn, n), O.tight_fusion_frame(km, rm, m)
    rows, cols, vals, X, G = _problem(11, n, m, nnz, 7)
    s = 0.37
    C = np.zeros((m, n))
    C[rows, cols] = vals
    Z = fft_analysis(X, kn, rn)
    U = fft_analysis(G, km, rm)
    y_ref = s * fft_synthesis(Z @ C.T, km, rm)
    dx_ref = s * fft_synthesis(U @ C, kn, rn)
    dc_ref = s * np.einsum("te,te->e", U[:, rows], Z[:, cols])
    np.testing.assert_allclose(O.adapter_fwd(Pin, Pout, rows, cols, vals, s, X), y_ref, atol=1e-12)
    dX, dC = O.adapter_bwd(Pin, Pout, rows, cols, vals, s, X, G)
    np.testing.assert_allclose(dX, dx_ref, atol=1e-12)
    np.testing.assert_allclose(dC, dc_ref, rtol=1e-10, atol=1e-12)
    dW_ref = s * fft_synthesis(fft_synthesis(C, kn, rn).T, km, rm).T   # P_out C P_in^T, columns then rows
    np.testing.assert_allclose(O.merge_delta(Pin, Pout, rows, cols, vals, s), dW_ref, atol=1e-12)


# ---------------------------------------------------------------- k = 1: P = I

def test_k1_frame_is_identity_and_adapter_is_plain_spmm():
    n, m = 10, 6
    Pin, Pout = O.tight_fusion_frame(1, n, n), O.tight_fusion_frame(1, m, m)
    np.testing.assert_array_equal(Pin.toarray(), np.eye(n))
    rows, cols, vals, X, G = _problem(5, n, m, 25, 9)
    s = 1.7
    C = np.zeros((m, n))
    C[rows, cols] = vals
    np.testing.assert_allclose(O.adapter_fwd(Pin, Pout, rows, cols, vals, s, X), s * X @ C.T, atol=1e-14)
    dX, dC = O.adapter_bwd(Pin, Pout, rows, cols, vals, s, X, G)
    np.testing.assert_allclose(dX, s * G @ C, atol=1e-14)
    np.testing.assert_allclose(dC, s * (G.T @ X)[rows, cols], atol=1e-13)
    np.testing.assert_allclose(O.merge_delta(Pin, Pout, rows, cols, vals, s), s * C, atol=1e-15)


# ---------------------------------------------------------------- finite differences

@pytest.mark.parametrize("fin,fout", [((6, 6, 22), (2, 4, 8)), ((4, 12, 48), (5, 8, 40))])
def test_gradients_match_finite_differences(fin, fout):
    (kn, rn, n), (km, rm, m) = fin, fout
    Pin, Pout = O.tight_fusion_frame(kn, rn, n), O.tight_fusion_frame(km, rm, m)
    cn, cm = Pin.shape[1], Pout.shape[1]
    rows, cols, vals, _, _ = _problem(7, cn, cm, 40, 4)     # C is (k rho_m) x (k rho_n)
    X = np.random.default_rng(2).standard_normal((4, n))
    W0 = np.random.default_rng(3).standard_normal((m, n)) / math.sqrt(n)
    s = 2.3

    def loss(v, Xv):
        y = Xv @ W0.T + O.adapter_fwd(Pin, Pout, rows, cols, v, s, Xv)
        return np.sum(np.sin(y))

    y = X @ W0.T + O.adapter_fwd(Pin, Pout, rows, cols, vals, s, X)
    G = np.cos(y)                      # dL/dy
    dXa, dC = O.adapter_bwd(Pin, Pout, rows, cols, vals, s, X, G)
    h = 1e-5
    for e in range(len(vals)):
        vp, vm = vals.copy(), vals.copy()
        vp[e] += h
        vm[e] -= h
        fd = (loss(vp, X) - loss(vm, X)) / (2 * h)
        assert abs(fd - dC[e]) <= 1e-7 * max(1.0, abs(fd)), (e, fd, dC[e])
    dX = G @ W0 + dXa
    for (t, j) in [(0, 0), (1, n - 1), (2, n // 2), (3, 3)]:
        Xp, Xm = X.copy(), X.copy()
        Xp[t, j] += h
        Xm[t, j] -= h
        fd = (loss(vals, Xp) - loss(vals, Xm)) / (2 * h)
        assert abs(fd - dX[t, j]) <= 1e-7 * max(1.0, abs(fd)), (t, j, fd, dX[t, j])


# ---------------------------------------------------------------- exact identities

def test_merge_norm_and_two_routes():
    Pin, Pout = O.tight_fusion_frame(4, 12, 48), O.tight_fusion_frame(5, 8, 40)
    rows, cols, vals, X, G = _problem(21, 48, 40, 200, 6)
    s = 0.8
    dW = O.merge_delta(Pin, Pout, rows, cols, vals, s)
    # orthogonal frames: ||P_out C P_in^T||_F = ||C||_F
    assert abs(np.linalg.norm(dW) - abs(s) * np.linalg.norm(vals)) <= 1e-12 * np.linalg.norm(dW)
    # the merged weight reproduces the factored forward pass
    np.testing.assert_allclose(X @ dW.T, O.adapter_fwd(Pin, Pout, rows, cols, vals, s, X), atol=1e-12)
    # with the full support, ||dC||_F = |s| ||G^T X||_F
    full_r, full_c = np.divmod(np.arange(40 * 48), 48)
    _, dC = O.adapter_bwd(Pin, Pout, full_r, full_c, np.zeros(40 * 48), s, X, G)
    assert abs(np.linalg.norm(dC) - abs(s) * np.linalg.norm(G.T @ X)) <= 1e-11 * np.linalg.norm(dC)


def test_subset_helpers_agree_with_full_results():
    Pin, Pout = O.tight_fusion_frame(12, 64, 768), O.tight_fusion_frame(36, 64, 2304)
    rows, cols, vals, X, G = _problem(31, 768, 2304, 3000, 9)
    s = 0.05
    _, dC = O.adapter_bwd(Pin, Pout, rows, cols, vals, s, X, G)
    sub = np.array([0, 5, 77, 2999])
    np.testing.assert_allclose(O.coeff_grad_entries(Pin, Pout, rows[sub], cols[sub], s, X, G), dC[sub],
                               rtol=1e-12, atol=1e-15)
    dW = O.merge_delta(Pin, Pout, rows, cols, vals, s)
    rsub = np.array([0, 1000, 2303])
    np.testing.assert_allclose(O.merge_delta_rows(Pin, Pout, rows, cols, vals, s, rsub), dW[rsub], atol=1e-15)
