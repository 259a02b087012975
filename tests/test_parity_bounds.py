"""The element-wise parity bounds of the GPU tests, checked on the CPU.

A plain numpy emulation of a bf16 implementation (frame entries, coefficients, z, v, u, q and
outputs rounded to bf16 as the error model allows; written here from that model, sharing
nothing with the HIP kernels) must stay inside the bounds; the same emulation with one support
entry dropped or routed to a wrong column must fall outside them.  This is what makes the
element-wise checks able to see a single lost entry, which a normwise 2e-2 check cannot
(one entry out of 10,000 moves y by about 1% of its norm).
"""
import numpy as np
import pytest

from paper_2608_26430_amd import inputs
from tests.parity_util import BwdBounds, FwdBounds, max_rel, oracle_frame, within


def _bf16(a):
    return inputs.bf16_round(np.asarray(a, dtype=np.float32)).astype(np.float64)


def _emulate(P_in, P_out, rows, cols, vals, s, X, G, rnd):
    """One implementation inside the error model: every frame entry, coefficient, intermediate
    and output rounded by `rnd`; sums in fp64 (tighter than fp32 accumulation)."""
    Pi, Po = rnd(P_in.toarray()), rnd(P_out.toarray())
    c = rnd(s * np.asarray(vals, dtype=np.float64))
    m_c, n_c = P_out.shape[1], P_in.shape[1]
    z = rnd(X @ Pi)
    v = np.zeros((X.shape[0], m_c))
    np.add.at(v.T, rows, (z[:, cols] * c).T)
    y = rnd(rnd(v) @ Po.T)
    u = rnd(G @ Po)
    q = np.zeros((G.shape[0], n_c))
    np.add.at(q.T, cols, (u[:, rows] * c).T)
    dx = rnd(rnd(q) @ Pi.T)
    dc = s * np.sum(u[:, rows] * z[:, cols], axis=0)
    return y, dx, dc


# (n, rho_in, m, rho_out, nnz, T): the fused 128-wide shapes of the GPU tests, one of them with a
# single token, and a narrow-block one
CASES = [(4096, 64, 4096, 64, 10000, 13), (1024, 16, 2048, 32, 3000, 1), (256, 16, 512, 32, 700, 100)]


@pytest.fixture(scope="module", params=CASES, ids=lambda c: "n%d_m%d_nnz%d_T%d" % (c[0], c[2], c[4], c[5]))
def problem(request):
    n, rn, m, rm, nnz, T = request.param
    g = inputs.rng(n + m + nnz + T)
    rows, cols = inputs.support(g, m, n, nnz)
    vals = inputs.gaussian(g, (nnz,), std=0.02).astype(np.float64)
    X = inputs.gaussian(g, (T, n), dtype="bf16").astype(np.float64)
    G = inputs.gaussian(g, (T, m), dtype="bf16").astype(np.float64)
    P_in, P_out = oracle_frame(n // rn, rn, n), oracle_frame(m // rm, rm, m)
    s = 0.173
    fb = FwdBounds(P_in, P_out, rows, cols, vals, s, X, "bf16", n // rn, m // rm)
    bb = BwdBounds(P_in, P_out, rows, cols, vals, s, X, G, "bf16", n // rn, m // rm)
    return dict(P_in=P_in, P_out=P_out, rows=rows, cols=cols, vals=vals, X=X, G=G, s=s, fb=fb, bb=bb)


def test_bf16_emulation_inside_bounds(problem):
    p = problem
    y, dx, dc = _emulate(p["P_in"], p["P_out"], p["rows"], p["cols"], p["vals"], p["s"], p["X"], p["G"], _bf16)
    fb, bb = p["fb"], p["bb"]
    checks = {
        "y": within(y, fb.y, fb.by), "v": within(fb.coef(y), fb.v, fb.bv),
        "dX": within(dx, bb.dx, bb.bdx), "q": within(bb.coef(dx), bb.q, bb.bq),
        "dC": within(dc, bb.dc, bb.bdc),
    }
    assert all(ok for ok, _ in checks.values()), checks
    # the bound is not vacuous: the emulated errors use a visible part of it
    assert max(w for _, w in checks.values()) > 0.02, checks
    # and the usual normwise figures stay well inside 2e-2
    assert max_rel(y, fb.y) < 2e-2 and max_rel(dc, bb.dc) < 2e-2


def test_dropped_or_misrouted_entry_is_caught(problem):
    p = problem
    if p["X"].shape[0] == 1:
        pytest.skip("with one token a single entry's loss is caught only in the proportion "
                    "test_single_entry_detection_rate measures")
    rows, cols, vals = p["rows"], p["cols"], p["vals"]
    fb, bb = p["fb"], p["bb"]
    # an entry of median coefficient magnitude, dropped from the forward and backward streams
    e = int(np.argsort(np.abs(vals))[len(vals) // 2])
    keep = np.arange(len(rows)) != e
    y, dx, dc = _emulate(p["P_in"], p["P_out"], rows[keep], cols[keep], vals[keep], p["s"], p["X"], p["G"], _bf16)
    assert not within(fb.coef(y), fb.v, fb.bv)[0], "a dropped forward entry passed the coefficient-space check"
    assert not within(bb.coef(dx), bb.q, bb.bq)[0], "a dropped backward entry passed the coefficient-space check"
    # the same entry routed to the wrong input coefficient
    bad = cols.copy()
    bad[e] = (bad[e] + 1) % p["P_in"].shape[1]
    while np.any((rows == rows[e]) & (bad == bad[e]) & keep):
        bad[e] = (bad[e] + 1) % p["P_in"].shape[1]
    y2, dx2, dc2 = _emulate(p["P_in"], p["P_out"], rows, bad, vals, p["s"], p["X"], p["G"], _bf16)
    assert not within(fb.coef(y2), fb.v, fb.bv)[0]
    assert not within(bb.coef(dx2), bb.q, bb.bq)[0]
    assert not within(dc2, bb.dc, bb.bdc)[0]


def test_single_entry_detection_rate(problem):
    """Over every support entry: the fraction whose loss the element-wise checks would see.
    In coefficient space a lost forward entry e = (a, b) moves v_t[a] by s c_e z_t[b] for each
    token; a lost dC entry is off by dC_e itself."""
    p = problem
    fb, bb = p["fb"], p["bb"]
    rows, cols, vals, s = p["rows"], p["cols"], p["vals"], p["s"]
    Z = np.asarray(p["P_in"].T @ p["X"].T).T
    Uc = np.asarray(p["P_out"].T @ p["G"].T).T
    hit_v = np.any(np.abs(s * vals[None, :] * Z[:, cols]) > fb.bv[:, rows], axis=0)
    hit_q = np.any(np.abs(s * vals[None, :] * Uc[:, rows]) > bb.bq[:, cols], axis=0)
    hit_dc = np.abs(bb.dc) > bb.bdc
    T = p["X"].shape[0]
    print(f"T={T}: forward-entry detection {hit_v.mean():.3f}, backward-entry {hit_q.mean():.3f}, "
          f"dC-entry {hit_dc.mean():.3f}")
    # with one token the loss hides behind rounding whenever c_e z_b happens to be small; a fault
    # that loses several entries (a lane, a round, a pair of blocks) is caught almost surely
    want = {1: (0.3, 0.9), 13: (0.7, 0.8), 100: (0.9, 0.7)}[T]
    assert min(hit_v.mean(), hit_q.mean()) >= want[0]
    assert hit_dc.mean() >= want[1]


def test_split_bf16_product_error():
    """The bf16 merge forms u v as hi(u) hi(v) + hi(u) lo(v) + lo(u) hi(v) with hi = RNE_bf16(x) and
    lo = RNE_bf16(x - hi) (x - hi computed in fp32, exactly); each product is exact in fp32.  The
    per-term error bound that merged_bf16_ok(split=True) uses is 3.01 2^-16 |u v|: checked here on
    random fp32 factors over many binades, and found tight to within a factor of a few."""
    from paper_2608_26430_amd import inputs
    g = np.random.default_rng(7)
    u = (g.standard_normal(200000) * np.exp2(g.integers(-20, 20, 200000))).astype(np.float32)
    v = (g.standard_normal(200000) * np.exp2(g.integers(-20, 20, 200000))).astype(np.float32)

    def split(x):
        hi = inputs.bf16_round(x)
        lo = inputs.bf16_round((x - hi).astype(np.float32))
        return hi.astype(np.float64), lo.astype(np.float64)

    hu, lu = split(u)
    hv, lv = split(v)
    got = hu * hv + hu * lv + lu * hv
    exact = u.astype(np.float64) * v.astype(np.float64)
    rel = np.abs(got - exact) / np.abs(exact)
    assert rel.max() <= 3.01 * 2.0 ** -16
    assert rel.max() >= 0.5 * 2.0 ** -16      # the bound is not loose by orders of magnitude
