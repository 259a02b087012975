"""Helpers shared by the GPU parity tests (no method arithmetic here)."""
import functools

import numpy as np

from oracle import frameft_oracle as O

TOL = {"f32": 1e-5, "bf16": 2e-2}   # normwise relative error bounds for fp32 / bf16 activations


@functools.lru_cache(maxsize=None)
def oracle_frame(k, rho, d):
    return O.tight_fusion_frame(k, rho, d)


def to_np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def rel(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    num = np.linalg.norm(got - ref)
    return float(num / den) if den > 0 else float(num)


def torch_act(a, dtype, device):
    """Host fp32 array (bf16-valued when dtype == 'bf16') -> device tensor, exactly."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(device=device, dtype=torch.bfloat16 if dtype == "bf16" else torch.float32)


def bf16_ulp(x):
    """Spacing of bf16 numbers at |x| (x finite, fp64 array)."""
    ax = np.maximum(np.abs(x), np.finfo(np.float32).tiny)
    e = np.floor(np.log2(ax))
    return np.exp2(e - 7)


def merged_bf16_ok(got, W0, dW, dW_abs=None, depth=0, split=False):
    """bf16 merge check: within one bf16 ulp of RNE(W0 + dW), widened by the fp32 rounding of
    W0 + dW (2^-22 (|W0| + |dW|)), which matters only where the two nearly cancel.

    With dW_abs (the sum of the absolute values of the terms of each dW element, i.e. the
    merge of |P_out| |C| |P_in|^T) and depth (the largest number of support entries summed into
    one element), also by the recursive-summation bound of the kernel's fp32 arithmetic,
    (depth + 4) 2^-24 dW_abs: each term is a product of four fp32-rounded factors and each fused
    multiply-add rounds the running sum once.  Near W0 + dW = 0 that error is not small next to
    the bf16 spacing of the result.

    split: the merge into a bf16 weight forms each term u v from bf16 hi / lo splits of its fp32
    factors (hi hi + hi lo + lo hi, each exact in fp32), which leaves at most 3.01 2^-16 |u v|
    per term, and sums three products per term: 3.01 2^-16 dW_abs + (3 depth + 5) 2^-24 dW_abs
    instead of the fp32 term."""
    from paper_2608_26430_amd import inputs
    exact = W0.astype(np.float64) + dW
    want = inputs.bf16_round(exact.astype(np.float32)).astype(np.float64)
    bound = bf16_ulp(want) + 2.0 ** -22 * (np.abs(W0) + np.abs(dW)) + 1e-30
    if dW_abs is not None:
        dW_abs = np.asarray(dW_abs, dtype=np.float64)
        if split:
            bound = bound + (3.01 * 2.0 ** -16 + (3 * depth + 5) * 2.0 ** -24) * 1.01 * dW_abs
        else:
            bound = bound + (depth + 4) * 2.0 ** -24 * 1.01 * dW_abs
    return bool(np.all(np.abs(np.asarray(got, dtype=np.float64) - want) <= bound))


def merge_abs_terms(P_in, P_out, rows, cols, vals, scale, rho_in, rho_out, out_rows=None):
    """(dW_abs, depth) for merged_bf16_ok: the merge of the absolute values, and the largest
    number of support entries that meet in one element of dW.  With k rho = d the frame P is
    block diagonal with dense blocks, coefficient a lying in block (a mod rho) // 2, so the
    entries meeting in an element are those of its (output block, input block) pair."""
    import scipy.sparse as sp
    from oracle import frameft_oracle as O
    Pa_in, Pa_out = abs(sp.csr_matrix(P_in)), abs(sp.csr_matrix(P_out))
    if out_rows is None:
        A = O.merge_delta(Pa_in, Pa_out, rows, cols, np.abs(vals), abs(scale))
    else:
        A = O.merge_delta_rows(Pa_in, Pa_out, rows, cols, np.abs(vals), abs(scale), out_rows)
    rb = (np.asarray(rows, dtype=np.int64) % rho_out) // 2
    cb = (np.asarray(cols, dtype=np.int64) % rho_in) // 2
    depth = int(np.bincount(rb * (rho_in // 2) + cb).max()) if len(rows) else 0
    return A, depth


def plan_c(plan, vals, device):
    """User-order coefficient values -> device fp32 tensor in the plan's slot layout."""
    import torch
    return torch.from_numpy(plan.to_plan(vals)).to(device)


def user_dc(plan, dC):
    """Plan-layout dC (device tensor) -> fp64 host array in user order; padding slots must be 0."""
    d = to_np(dC)
    assert np.all(d[plan.order < 0] == 0), "padding slots of dC are not zero"
    return plan.to_user(d)


# ------------------------------------------------------------------ element-wise bounds
#
# Error model, covering every kernel of the library (activation precision with unit roundoff u:
# 2^-8 for bf16, 2^-24 for fp32; accumulation in fp32, u32 = 2^-24):
#   * the frame blocks are applied with entries rounded to the activation precision, directly
#     (kappa = 1) or as a product of factors (a radix-4 stage and a smaller DFT, kappa = 4: the
#     absolute products of the factors stay within a few times |P|);
#   * every coefficient s c_e may be rounded to that precision;
#   * every intermediate vector (z, v forward; u, q, z backward) may be rounded to it after an
#     fp32 accumulation of depth D (error <= D u32 times the sum of absolute terms);
#   * outputs y, dX are rounded to it after beta * old + new, and with beta != 0 possibly also
#     the new term alone before the sum; dC is fp32.
# The bounds below are the first-order propagation of those roundings, with 5% added for the
# second-order terms (products of two roundings, at most u^2 relative).
#
# y and dX are compared in coefficient space as well: with k rho = d the frame is orthogonal, so
# P_out^T (y_gpu - y) is the error of the coefficient vector v = s C z that y was synthesized
# from.  A dropped or misrouted support entry changes one coefficient per token there, by
# s c_e z_b, while in y it spreads over a whole 2k-wide block where the frame-rounding bound is
# about sqrt(2k) times larger than a single entry's effect.

U_ACT = {"bf16": 2.0 ** -8, "f32": 2.0 ** -24}   # 8 and 24 significant bits, round to nearest
U32 = 2.0 ** -24
SLACK = 1.05


def _abs(M):
    import scipy.sparse as sp
    return abs(sp.csr_matrix(M))


def _depth(P):
    """Most nonzeros in one column of the frame P (the contraction depth of one coefficient)."""
    import scipy.sparse as sp
    return int(np.diff(sp.csc_matrix(P).indptr).max()) if P.shape[1] else 0


def _kappa(k):
    """Frame application: direct for blocks up to 128 wide, one radix-4 stage up to 512 wide, two
    or three stages beyond (the stages' butterflies sum up to 4^S unit-modulus terms per value, so
    the absolute products of the factors reach a few times |P|; see above)."""
    return 1.0 if 2 * k <= 128 else 4.0 if 2 * k <= 512 else 8.0


def coef_matrix(rows, cols, vals, scale, m_coef, n_coef):
    import scipy.sparse as sp
    return sp.csr_matrix((float(scale) * np.asarray(vals, dtype=np.float64),
                          (np.asarray(rows, dtype=np.int64), np.asarray(cols, dtype=np.int64))),
                         shape=(m_coef, n_coef))


class FwdBounds:
    """Reference forward y = beta Y0 + s P_out C P_in^T x (fp64, from the oracle's frames) with
    element-wise error bounds: `y`, `by` in token space and `v`, `bv` in coefficient space."""

    def __init__(self, P_in, P_out, rows, cols, vals, scale, X, dtype, k_in, k_out, beta_y0=None):
        u = U_ACT[dtype]
        X = np.asarray(X, dtype=np.float64)
        sC = coef_matrix(rows, cols, vals, scale, P_out.shape[1], P_in.shape[1])
        aC = abs(sC)
        aPi, aPo = _abs(P_in), _abs(P_out)
        Din, Dout = _depth(P_in), _depth(P_out)
        Dc = int(np.diff(sC.indptr).max()) if sC.nnz else 0
        Z = np.asarray(P_in.T @ X.T).T
        V = np.asarray(sC @ Z.T).T
        y_ad = np.asarray(P_out @ V.T).T
        y = y_ad if beta_y0 is None else y_ad + beta_y0
        bz = u * np.abs(Z) + (_kappa(k_in) * u + Din * U32) * np.asarray(aPi.T @ np.abs(X).T).T
        bv = (u * np.abs(V) + (u + Dc * U32) * np.asarray(aC @ np.abs(Z).T).T
              + np.asarray(aC @ bz.T).T)
        syn = _kappa(k_out) * u + Dout * U32
        aV = np.abs(V)
        self.y = y
        # output rounding: of the total, and (with beta) possibly of the adapter term before the sum
        out = np.abs(y) + (np.abs(y_ad) if beta_y0 is not None else 0.0)
        self.by = SLACK * (u * out + syn * np.asarray(aPo @ aV.T).T + np.asarray(aPo @ bv.T).T) + 1e-30
        self.v = V                      # coefficient-space reference (beta term excluded)
        self.bv = SLACK * (u * np.asarray(aPo.T @ out.T).T
                           + syn * np.asarray(aPo.T @ (aPo @ aV.T)).T + bv) + 1e-30
        self.P_out = P_out
        self.beta_y0 = beta_y0

    def coef(self, y_gpu):
        """P_out^T (y_gpu - beta Y0): the coefficient vector the GPU output corresponds to."""
        d = np.asarray(y_gpu, dtype=np.float64)
        if self.beta_y0 is not None:
            d = d - self.beta_y0
        return np.asarray(self.P_out.T @ d.T).T


class BwdBounds:
    """Reference backward dX = beta dX0 + s P_in C^T P_out^T g and dC = s (P_out^T G^T X P_in)
    on the support, with element-wise bounds (`dx`/`bdx`, `q`/`bq`, `dc`/`bdc`)."""

    def __init__(self, P_in, P_out, rows, cols, vals, scale, X, G, dtype, k_in, k_out, beta_dx0=None):
        u = U_ACT[dtype]
        X = np.asarray(X, dtype=np.float64)
        G = np.asarray(G, dtype=np.float64)
        rows = np.asarray(rows, dtype=np.int64)
        cols = np.asarray(cols, dtype=np.int64)
        sC = coef_matrix(rows, cols, vals, scale, P_out.shape[1], P_in.shape[1])
        aC = abs(sC)
        aPi, aPo = _abs(P_in), _abs(P_out)
        Din, Dout = _depth(P_in), _depth(P_out)
        Dct = int(np.diff(sC.tocsc().indptr).max()) if sC.nnz else 0
        T = X.shape[0]
        Uc = np.asarray(P_out.T @ G.T).T
        Z = np.asarray(P_in.T @ X.T).T
        bu = u * np.abs(Uc) + (_kappa(k_out) * u + Dout * U32) * np.asarray(aPo.T @ np.abs(G).T).T
        bz = u * np.abs(Z) + (_kappa(k_in) * u + Din * U32) * np.asarray(aPi.T @ np.abs(X).T).T
        Q = np.asarray(sC.T @ Uc.T).T
        dx_ad = np.asarray(P_in @ Q.T).T
        dx = dx_ad if beta_dx0 is None else dx_ad + beta_dx0
        bq = (u * np.abs(Q) + (u + Dct * U32) * np.asarray(aC.T @ np.abs(Uc).T).T
              + np.asarray(aC.T @ bu.T).T)
        syn = _kappa(k_in) * u + Din * U32
        aQ = np.abs(Q)
        self.dx = dx
        out = np.abs(dx) + (np.abs(dx_ad) if beta_dx0 is not None else 0.0)
        self.bdx = SLACK * (u * out + syn * np.asarray(aPi @ aQ.T).T + np.asarray(aPi @ bq.T).T) + 1e-30
        self.q = Q
        self.bq = SLACK * (u * np.asarray(aPi.T @ out.T).T
                           + syn * np.asarray(aPi.T @ (aPi @ aQ.T)).T + bq) + 1e-30
        s = abs(float(scale))
        ua, zb = Uc[:, rows], Z[:, cols]
        self.dc = float(scale) * np.sum(ua * zb, axis=0)
        self.bdc = SLACK * (s * np.sum(bu[:, rows] * np.abs(zb) + np.abs(ua) * bz[:, cols], axis=0)
                            + s * (T + 2) * U32 * np.sum(np.abs(ua * zb), axis=0)) + 1e-30
        self.P_in = P_in
        self.beta_dx0 = beta_dx0

    def coef(self, dx_gpu):
        d = np.asarray(dx_gpu, dtype=np.float64)
        if self.beta_dx0 is not None:
            d = d - self.beta_dx0
        return np.asarray(self.P_in.T @ d.T).T


def merge_bound(dW_abs, depth):
    """Element-wise bound on an fp32 merge: the recursive-summation bound (depth + 4) 2^-24 dW_abs
    (each term a product of four fp32-rounded factors, each fused multiply-add rounding the running
    sum), plus 2^-24 max(dW_abs): frame entries that are zero in exact arithmetic (cosines of
    quarter turns) may be a rounding residue on either side, which the first term cannot cover."""
    dW_abs = np.asarray(dW_abs, dtype=np.float64)
    top = float(dW_abs.max()) if dW_abs.size else 0.0
    return (depth + 4) * 2.0 ** -24 * 1.01 * dW_abs + 2.0 ** -24 * top + 1e-30


def within(got, ref, bound):
    """(ok, worst): every |got - ref| <= bound element-wise; worst = max |got - ref| / bound."""
    got = np.asarray(got, dtype=np.float64)
    err = np.abs(got - ref)
    ok = bool(np.all(np.isfinite(got)) and np.all(err <= bound))
    worst = float(np.max(err / bound)) if err.size else 0.0
    return ok, worst


def max_rel(got, ref):
    """max |got - ref| / max |ref| (reported alongside the element-wise checks)."""
    got = np.asarray(got, dtype=np.float64)
    den = float(np.max(np.abs(ref))) if np.size(ref) else 0.0
    num = float(np.max(np.abs(got - ref))) if np.size(ref) else 0.0
    return num / den if den > 0 else num


# ------------------------------------------------------------------ guarded buffers

SENTINEL = {"bf16": 0x7FA5, "f32": 0x7FC0A5A5}   # NaN bit patterns no kernel produces
GUARD = 64                                         # guard elements before and after (16-byte multiple)


def guarded(rows, width, ld, dtype, device, init=None):
    """A rows x width device view with leading dimension ld inside a flat buffer whose guard
    regions and padding columns hold the sentinel bit pattern.  Returns (buf, view)."""
    import torch
    it = torch.int16 if dtype == "bf16" else torch.int32
    ft = torch.bfloat16 if dtype == "bf16" else torch.float32
    n = 2 * GUARD + rows * ld
    buf = torch.full((n,), SENTINEL[dtype], dtype=it, device=device)
    view = buf.view(ft)[GUARD:GUARD + rows * ld].view(rows, ld)[:, :width]
    if init is not None:
        view.copy_(torch.as_tensor(np.ascontiguousarray(init, dtype=np.float32)).to(device=device, dtype=ft))
    return buf, view


def guards_intact(buf, rows, width, ld, dtype):
    """True when every element of buf outside the rows x width view still holds the sentinel."""
    import torch
    b = buf.cpu().numpy().astype(np.int64)
    want = SENTINEL[dtype]
    if dtype == "bf16":
        b = b & 0xFFFF
    mask = np.ones(b.size, dtype=bool)
    idx = GUARD + (np.arange(rows)[:, None] * ld + np.arange(width)[None, :])
    mask[idx.ravel()] = False
    return bool(np.all(b[mask] == want))
