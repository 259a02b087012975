"""The paper's own subspace dimension rho = 2 (Sec. 4.1 and 4.2 configurations, k rho = n): each
frame is one dense realified DFT of size d/2, applied as two or three radix-4 stages in registers
and a dense DFT of at most 64 points on MFMA; the merge contracts the frame's single block pair on
MFMA.  Forward, backward and merge against the oracle element by element; the frame read back
against the oracle's frame."""
import numpy as np
import pytest

from oracle import frameft_oracle as O
from paper_2608_26430_amd import inputs
from tests.parity_util import (BwdBounds, FwdBounds, merge_abs_terms, merge_bound, oracle_frame, to_np, torch_act,
                               user_dc, within)

torch = pytest.importorskip("torch")
import paper_2608_26430_amd as ff  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    return torch.device("cuda:0")


def _ok(name, got, ref, bound):
    ok, worst = within(got, ref, bound)
    assert ok, f"{name}: element-wise bound exceeded (max err/bound {worst:.3g})"
    return worst


@pytest.mark.parametrize("d", [1024, 4096])
def test_rho2_frame_matches_oracle(dev, d):
    f = ff.framegen(d, d // 2, 2)
    ref = oracle_frame(d // 2, 2, d)
    cols = sorted(set([0, 1, 2, 3, d // 2, d - 1] + list(np.random.default_rng(d).integers(0, d, 20))))
    got = np.concatenate([f.export(c, 1) for c in cols], axis=1)
    np.testing.assert_allclose(got, ref[:, cols].toarray(), rtol=0, atol=3e-7)


# (d, nnz, T): the language-understanding runs use 1000 coefficients, the instruction-tuning runs
# 5000 (Sec. 4.1, 4.2); ragged token counts
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", [(1024, 1000, 33), (4096, 5000, 9)], ids=lambda c: "d%d_nnz%d_T%d" % c)
def test_rho2_fwd_bwd_parity(dev, case, dtype):
    d, nnz, T = case
    k = d // 2
    g = inputs.rng(d + nnz + T)
    rows, cols = inputs.support(g, d, d, nnz)
    vals = inputs.gaussian(g, (nnz,), std=0.02)
    X = inputs.gaussian(g, (T, d), dtype=dtype)
    G = inputs.gaussian(g, (T, d), dtype=dtype)
    s = 200.0 / d
    f = ff.framegen(d, k, 2)
    plan = ff.plan_create(f, f, rows, cols, max_tokens=T)
    assert plan.radix == (4, 4) and not plan.fast128
    Xd, Gd = torch_act(X, dtype, dev), torch_act(G, dtype, dev)
    c = torch.from_numpy(plan.to_plan(vals)).to(dev)
    Y = ff.adapter_fwd(plan, Xd, c, s)
    Y1 = Y.clone()
    ff.adapter_fwd(plan, Xd, c, s, Y=Y1, beta=1.0)
    dX, dC = ff.adapter_bwd(plan, Xd, Gd, c, s)
    torch.cuda.synchronize()
    P = oracle_frame(k, 2, d)
    fb = FwdBounds(P, P, rows, cols, vals, s, X, dtype, k, k)
    bb = BwdBounds(P, P, rows, cols, vals, s, X, G, dtype, k, k)
    y = to_np(Y)
    _ok("y", y, fb.y, fb.by)
    _ok("y coef", fb.coef(y), fb.v, fb.bv)
    fb2 = FwdBounds(P, P, rows, cols, vals, s, X, dtype, k, k, beta_y0=to_np(Y))
    _ok("y beta=1", to_np(Y1), fb2.y, fb2.by)
    dx = to_np(dX)
    _ok("dX", dx, bb.dx, bb.bdx)
    _ok("dX coef", bb.coef(dx), bb.q, bb.bq)
    _ok("dC", user_dc(plan, dC), bb.dc, bb.bdc)


def test_rho2_merge_large(dev):
    """d = 4096 (one 4096-wide block pair holding all 5000 entries): into an aligned fp32 array, a
    misaligned fp32 view with an odd leading dimension (element-wise accesses) and in place into a
    bf16 weight (split bf16 products); sampled rows against the oracle."""
    from tests.parity_util import merged_bf16_ok
    d, nnz = 4096, 5000
    k = d // 2
    g = inputs.rng(11)
    rows, cols = inputs.support(g, d, d, nnz)
    vals = inputs.gaussian(g, (nnz,), std=0.02)
    s = 200.0 / d
    f = ff.framegen(d, k, 2)
    plan = ff.plan_create(f, f, rows, cols, max_tokens=1)
    c = torch.from_numpy(plan.to_plan(vals)).to(dev)
    Wd = ff.merge_delta(plan, c, s, torch.full((d, d), float("nan"), device=dev), beta=0.0)
    buf = torch.zeros(d * (d + 1) + 1, device=dev)
    Wu = buf[1:].view(d, d + 1)[:, :d]                 # 4 bytes off 16-byte alignment, odd ldw
    Wu.copy_(Wd)
    ff.merge_delta(plan, c, -s, Wu, beta=1.0)          # unmerge: back to zero
    W0 = inputs.weight(inputs.rng(12), d, d, "bf16")
    Wb = ff.merge_delta(plan, c, s, torch_act(W0, "bf16", dev), beta=1.0)
    torch.cuda.synchronize()
    P = oracle_frame(k, 2, d)
    r = np.unique(np.concatenate([[0, 1, 2047, 2048, d - 1], np.random.default_rng(3).integers(0, d, 11)]))
    dw = O.merge_delta_rows(P, P, rows, cols, vals, s, r)
    dW_abs, depth = merge_abs_terms(P, P, rows, cols, vals, s, 2, 2, r)
    _ok("dW", to_np(Wd[r]), dw, merge_bound(dW_abs, depth))
    _ok("unmerged", to_np(Wu[r]), np.zeros_like(dw), 2 * merge_bound(dW_abs, depth))
    assert merged_bf16_ok(to_np(Wb[r]), W0[r], dw, dW_abs, depth, split=True)
    nrm = float(torch.linalg.vector_norm(Wd.double()))   # orthogonal frames: ||dW||_F = |s| ||C||_F
    assert abs(nrm - abs(s) * np.linalg.norm(vals.astype(np.float64))) <= 1e-5 * nrm


def test_rho2_merge_parity(dev):
    d, nnz = 1024, 1000
    k = d // 2
    g = inputs.rng(7)
    rows, cols = inputs.support(g, d, d, nnz)
    vals = inputs.gaussian(g, (nnz,), std=0.02)
    s = 200.0 / d
    f = ff.framegen(d, k, 2)
    plan = ff.plan_create(f, f, rows, cols, max_tokens=1)
    c = torch.from_numpy(plan.to_plan(vals)).to(dev)
    Wd = ff.merge_delta(plan, c, s, torch.empty((d, d), device=dev), beta=0.0)
    torch.cuda.synchronize()
    P = oracle_frame(k, 2, d)
    dw = O.merge_delta(P, P, rows, cols, vals, s)
    dW_abs, depth = merge_abs_terms(P, P, rows, cols, vals, s, 2, 2)
    _ok("dW", to_np(Wd), dw, merge_bound(dW_abs, depth))
