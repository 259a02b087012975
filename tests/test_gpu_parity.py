"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Tolerances (normwise relative error per output tensor): 1e-5 for fp32
activations, 2e-2 for bf16 activations with fp32 accumulation.  The merge is
fp32 arithmetic: 1e-5 for the dense delta; merged into a bf16 weight, the result
is within one bf16 ulp of the correctly rounded W0 + dW, widened by the fp32
rounding of the sum (visible only where W0 and dW nearly cancel).
"""
import numpy as np
import pytest

from oracle import frameft_oracle as O
from paper_2608_26430_amd import inputs
from tests.parity_util import (TOL, U32, BwdBounds, FwdBounds, guarded, guards_intact, max_rel, merge_abs_terms, merge_bound,
                               merged_bf16_ok, oracle_frame, plan_c, rel, to_np, torch_act, user_dc, within)

torch = pytest.importorskip("torch")
import paper_2608_26430_amd as ff  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    return torch.device("cuda:0")


@pytest.mark.parametrize("d,k,rho", [(256, 16, 16), (4096, 64, 64), (768, 12, 64), (2304, 36, 64),
                                     (2752, 172, 16), (3584, 224, 16), (64, 4, 16)])
def test_framegen_matches_oracle(dev, d, k, rho):
    f = ff.framegen(d, k, rho)
    ref = oracle_frame(k, rho, d)
    cols = sorted(set([0, 1, rho - 1, rho, k * rho - 1] + list(np.random.default_rng(d).integers(0, k * rho, 24))))
    got = np.concatenate([f.export(c, 1) for c in cols], axis=1)
    np.testing.assert_allclose(got, ref[:, cols].toarray(), rtol=0, atol=3e-7)


# (n, rho_in, m, rho_out, nnz, T): block widths 2k of 8, 16, 24, 32, 72, 128, 344 and 448,
# ragged token counts, a single token, an empty and a fully dense coefficient matrix.
SHAPES = [
    (256, 16, 256, 16, 512, 64),
    (256, 16, 256, 16, 512, 1),
    (256, 16, 512, 32, 700, 100),
    (768, 64, 2304, 64, 3000, 37),
    (1024, 16, 256, 16, 2000, 19),
    (2752, 16, 1024, 16, 4000, 9),
    (3584, 16, 256, 32, 5000, 5),
    (64, 16, 64, 16, 4096, 23),
    (256, 16, 256, 16, 0, 10),
    # both blocks 128 wide: the fused 128-wide kernels serve bf16
    (4096, 64, 4096, 64, 10000, 13),
    (1024, 16, 2048, 32, 3000, 1),
    (2048, 32, 1024, 16, 5000, 29),
    (1024, 16, 1024, 16, 0, 9),
    # the 8-token fused backward: an output side too wide for the 16-token array, and backward
    # streams too long for its registers
    (1024, 16, 8192, 128, 6000, 21),
    (1024, 16, 1024, 16, 40000, 11),
    # input side in chunks of blocks (dense support, 256-wide factored input blocks): fewer
    # tokens than a tile, and a single token
    (8192, 64, 2048, 64, 42000, 5),
    (8192, 64, 2048, 64, 42000, 1),
    # an output side too wide for four tokens per tile (factored 448-wide blocks): bf16 tiles stay
    # token-major
    (256, 16, 28672, 128, 5000, 7),
]


def _problem(shape, dtype, seed):
    n, rn, m, rm, nnz, T = shape
    g = inputs.rng(seed)
    rows, cols = inputs.support(g, m, n, nnz)
    vals = inputs.gaussian(g, (nnz,), std=0.02)
    X = inputs.gaussian(g, (T, n), dtype=dtype)
    G = inputs.gaussian(g, (T, m), dtype=dtype)
    return rows, cols, vals, X, G


def _adapter_rms_like(g, shape, ref, dtype):
    """Random N(0, rms(ref)^2) values (bf16-rounded for bf16): an existing Y or dX of the adapter
    term's own magnitude, so that a beta epilogue which dropped the adapter term would fail."""
    r = float(np.sqrt(np.mean(np.square(ref)))) if np.size(ref) else 1.0
    return inputs.gaussian(g, shape, std=max(r, 1e-6), dtype=dtype)


def _check(name, got, ref, bound, report):
    ok, worst = within(got, ref, bound)
    report[name] = (round(worst, 4), round(max_rel(got, ref), 6))
    assert ok, f"{name}: element-wise bound exceeded (max err/bound {worst:.3g}); {report}"


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "n%d_m%d_nnz%d_T%d" % (s[0], s[2], s[4], s[5]))
def test_small_parity(dev, shape, dtype):
    """Every output against the oracle element by element (token space, and for y / dX also
    coefficient space, where a single lost support entry stands out), with inputs and outputs in
    views whose leading dimension exceeds their width: the padding columns of X and G hold NaN
    patterns that must not leak into any result, and the padding and guard regions around Y, dX,
    dC and W must come back untouched."""
    n, rn, m, rm, nnz, T = shape
    rows, cols, vals, X, G = _problem(shape, dtype, seed=n * 7 + m + nnz + T)
    s = 0.173
    k_in, k_out = n // rn, m // rm
    P_in, P_out = oracle_frame(k_in, rn, n), oracle_frame(k_out, rm, m)
    f_in, f_out = ff.framegen(n, k_in, rn), ff.framegen(m, k_out, rm)
    plan = ff.plan_create(f_in, f_out, rows, cols, max_tokens=T)
    assert plan.fast128 == (k_in == 64 and k_out == 64 and (n // 128) % 2 == 0 and (m // 128) % 2 == 0)
    if plan.fast128:
        assert plan.bwd_tile_tokens == (8 if m > 4096 or nnz > 20000 else 16)
    # blocks wider than 128 (k = 172, 224) are applied as a radix-4 stage plus a DFT of size k/4
    assert plan.radix == (4 if 2 * k_in > 128 else 1, 4 if 2 * k_out > 128 else 1)
    # the generic kernels chunk the input side only for the wide, dense-support shapes
    assert (plan.gen_chunks > 1) == (n == 8192)
    # bf16 tiles keep four tokens per coefficient together (whole multiples of four tokens per
    # tile) unless not even four tokens fit
    assert plan.gen_token_groups == (m != 28672)
    if plan.gen_token_groups:
        assert plan.gen_tile_tokens("bf16") % 4 == 0 and plan.gen_tile_tokens("bf16") >= 4
    else:
        assert plan.gen_tile_tokens("bf16") < 4
    pad = 8 if dtype == "bf16" else 4
    xbuf, Xd = guarded(T, n, n + pad, dtype, dev, X)
    gbuf, Gd = guarded(T, m, m + 2 * pad, dtype, dev, G)
    c = plan_c(plan, vals, dev)
    order = plan.order
    assert np.array_equal(np.sort(order[order >= 0]), np.arange(nnz))
    assert plan.coef_slots == order.size >= nnz
    L = plan.coef_slots

    fb = FwdBounds(P_in, P_out, rows, cols, vals, s, X, dtype, k_in, k_out)
    bb = BwdBounds(P_in, P_out, rows, cols, vals, s, X, G, dtype, k_in, k_out)
    Y0 = _adapter_rms_like(inputs.rng(3), (T, m), fb.y, dtype)
    dX0 = _adapter_rms_like(inputs.rng(4), (T, n), bb.dx, dtype)
    fbb = FwdBounds(P_in, P_out, rows, cols, vals, s, X, dtype, k_in, k_out, beta_y0=0.75 * Y0)
    bbb = BwdBounds(P_in, P_out, rows, cols, vals, s, X, G, dtype, k_in, k_out, beta_dx0=-1.5 * dX0)

    # forward: overwrite a contiguous Y, and beta-accumulate into a padded, guarded one
    Y = ff.adapter_fwd(plan, Xd, c, s)
    ybuf, Yb = guarded(T, m, m + pad, dtype, dev, Y0)
    ff.adapter_fwd(plan, Xd, c, s, Y=Yb, beta=0.75)
    # backward: overwrite, then beta / accumulate into padded, guarded outputs
    dX, dC = ff.adapter_bwd(plan, Xd, Gd, c, s, dC=torch.full((L,), float("nan"), device=dev))
    dxbuf, dXb = guarded(T, n, n + 3 * pad, dtype, dev, dX0)
    dC0 = inputs.gaussian(inputs.rng(5), (nnz,)).astype(np.float32)
    dC_init = plan.to_plan(dC0)
    dC_init[order < 0] = 5.0            # accumulating calls leave padding slots alone
    dcbuf, dCb2 = guarded(1, L, L, "f32", dev, dC_init[None, :])
    dCb = dCb2[0]
    ff.adapter_bwd(plan, Xd, Gd, c, s, dX=dXb, beta_dx=-1.5, dC=dCb, accumulate_dc=True)
    _, dC2 = ff.adapter_bwd(plan, Xd, Gd, c, s, want_dx=False)
    # merge: dense delta into a padded fp32 array, and in place into a bf16 weight
    dw_ref = O.merge_delta(P_in, P_out, rows, cols, vals, s)
    wbuf, Wd = guarded(m, n, n + 4, "f32", dev)
    ff.merge_delta(plan, c, s, Wd, beta=0.0)
    W0 = inputs.weight(inputs.rng(6), m, n, "bf16")
    Wb = ff.merge_delta(plan, c, s, torch_act(W0, "bf16", dev), beta=1.0)
    torch.cuda.synchronize()

    for name, buf, rr, ww, ld, dt in (("Y", ybuf, T, m, m + pad, dtype), ("dX", dxbuf, T, n, n + 3 * pad, dtype),
                                      ("dC", dcbuf, 1, L, L, "f32"), ("W", wbuf, m, n, n + 4, "f32"),
                                      ("X", xbuf, T, n, n + pad, dtype), ("G", gbuf, T, m, m + 2 * pad, dtype)):
        assert guards_intact(buf, rr, ww, ld, dt), f"{name}: padding or guard region overwritten"
    rep = {}
    if nnz == 0:
        assert np.all(to_np(Y) == 0) and np.all(to_np(dX) == 0) and np.all(to_np(Wd) == 0)
        assert dC.numel() == L and np.all(to_np(dC) == 0)   # padding only
        _check("y beta", to_np(Yb), fbb.y, fbb.by, rep)
        _check("dX beta", to_np(dXb), bbb.dx, bbb.bdx, rep)
        return
    _check("y", to_np(Y), fb.y, fb.by, rep)
    _check("y coef", fb.coef(to_np(Y)), fb.v, fb.bv, rep)
    _check("y beta", to_np(Yb), fbb.y, fbb.by, rep)
    _check("y beta coef", fbb.coef(to_np(Yb)), fbb.v, fbb.bv, rep)
    _check("dX", to_np(dX), bb.dx, bb.bdx, rep)
    _check("dX coef", bb.coef(to_np(dX)), bb.q, bb.bq, rep)
    _check("dX beta", to_np(dXb), bbb.dx, bbb.bdx, rep)
    _check("dX beta coef", bbb.coef(to_np(dXb)), bbb.q, bbb.bq, rep)
    _check("dC", user_dc(plan, dC), bb.dc, bb.bdc, rep)
    assert np.all(to_np(dCb)[order < 0] == 5.0)
    _check("dC acc", plan.to_user(to_np(dCb)), dC0 + bb.dc,
           bb.bdc + 2 * U32 * (np.abs(dC0) + np.abs(bb.dc)), rep)
    assert torch.equal(dC, dC2), "dC is not deterministic"
    dW_abs, depth = merge_abs_terms(P_in, P_out, rows, cols, vals, s, rn, rm)
    _check("dW", to_np(Wd), dw_ref, merge_bound(dW_abs, depth), rep)
    assert merged_bf16_ok(to_np(Wb), W0, dw_ref, dW_abs, depth, split=True)
    # the normwise figures of the tolerance statement, for the record
    assert rel(to_np(Y), fb.y) <= TOL[dtype] and rel(user_dc(plan, dC), bb.dc) <= TOL[dtype]
    print(f"\n{shape} {dtype}: (max err/bound, max-abs/max|ref|) {rep}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [SHAPES[0], SHAPES[9], SHAPES[10], SHAPES[11], SHAPES[12]],
                         ids=lambda s: "n%d_m%d_nnz%d_T%d" % (s[0], s[2], s[4], s[5]))
def test_saved_copy_matches_plain_calls(dev, shape, dtype):
    """adapter_fwd(save=) / adapter_bwd(saved=) give bitwise the results of the plain calls,
    also when the copy was written by a forward with no tokens or overwritten by a later one."""
    n, rn, m, rm, nnz, T = shape
    rows, cols, vals, X, G = _problem(shape, dtype, seed=n + 3 * m + nnz + T)
    f_in, f_out = ff.framegen(n, n // rn, rn), ff.framegen(m, m // rm, rm)
    plan = ff.plan_create(f_in, f_out, rows, cols, max_tokens=T)
    assert plan.saved_floats == (plan.query(6) if plan.fast128 else 0)
    assert (plan.saved_floats > 0) == plan.fast128
    saved = plan.new_saved(dev)
    if saved is None:
        saved = torch.empty((0,), device=dev)   # accepted and ignored where no copy is needed
    Xd, Gd = torch_act(X, dtype, dev), torch_act(G, dtype, dev)
    c = plan_c(plan, vals, dev)
    other = plan_c(plan, inputs.gaussian(inputs.rng(9), (nnz,), std=0.02), dev)
    s = 0.31
    Y = ff.adapter_fwd(plan, Xd, c, s)
    dX, dC = ff.adapter_bwd(plan, Xd, Gd, c, s)
    dX0 = torch_act(inputs.gaussian(inputs.rng(4), (T, n), dtype=dtype), dtype, dev)
    dXb, _ = ff.adapter_bwd(plan, Xd, Gd, c, s, dX=dX0.clone(), beta_dx=0.5, want_dc=False)
    ff.adapter_fwd(plan, Xd, other, s, save=saved)               # overwritten below
    Ys = ff.adapter_fwd(plan, Xd, c, s, save=saved)
    dXs, dCs = ff.adapter_bwd(plan, Xd, Gd, c, s, saved=saved)
    dXbs, _ = ff.adapter_bwd(plan, Xd, Gd, c, s, dX=dX0.clone(), beta_dx=0.5, want_dc=False, saved=saved)
    ff.adapter_fwd(plan, Xd[:0], c, s, save=saved)               # no tokens: the copy alone
    dXe, _ = ff.adapter_bwd(plan, Xd, Gd, c, s, want_dc=False, saved=saved)
    torch.cuda.synchronize()
    assert torch.equal(Y, Ys)
    assert torch.equal(dX, dXs) and torch.equal(dC, dCs)
    assert torch.equal(dXb, dXbs)
    assert torch.equal(dX, dXe)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_batched_matches_single_calls(dev, dtype):
    n, m, nnz, T, count = 4096, 4096, 4000, 21, 3
    g = inputs.rng(77)
    rows, cols = inputs.support(g, m, n, nnz)
    f = ff.framegen(4096, 64, 64)
    plan = ff.plan_create(f, f, rows, cols, max_tokens=T, max_batch=count)
    P = oracle_frame(64, 64, 4096)
    s = 0.05
    vals = [inputs.gaussian(g, (nnz,), std=0.02) for _ in range(count)]
    Xs = [inputs.gaussian(g, (T, n), dtype=dtype) for _ in range(count)]
    Gs = [inputs.gaussian(g, (T, m), dtype=dtype) for _ in range(count)]
    Xd = [torch_act(x, dtype, dev) for x in Xs]
    Gd = [torch_act(x, dtype, dev) for x in Gs]
    cd = [plan_c(plan, v, dev) for v in vals]
    Yd = [torch.empty((T, m), dtype=Xd[0].dtype, device=dev) for _ in range(count)]
    dXd = [torch.empty((T, n), dtype=Xd[0].dtype, device=dev) for _ in range(count)]
    dCd = [torch.full((plan.coef_slots,), float("nan"), device=dev) for _ in range(count)]
    ff.adapter_fwd_batched(plan, Xd, cd, s, Yd)
    ff.adapter_bwd_batched(plan, Xd, Gd, cd, s, dXd, dCd)
    torch.cuda.synchronize()
    tol = TOL[dtype]
    for i in range(count):
        y_ref = O.adapter_fwd(P, P, rows, cols, vals[i], s, Xs[i])
        dx_ref, dc_ref = O.adapter_bwd(P, P, rows, cols, vals[i], s, Xs[i], Gs[i])
        assert rel(to_np(Yd[i]), y_ref) <= tol
        assert rel(to_np(dXd[i]), dx_ref) <= tol
        assert rel(user_dc(plan, dCd[i]), dc_ref) <= tol


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(2752, 16, 1024, 16, 3000), (768, 64, 2304, 64, 3000)],
                         ids=["factored_in", "direct_vit"])
def test_generic_backward_many_tiles_per_workgroup(dev, dtype, shape):
    """The generic backward runs at most one workgroup per CU, looping over tiles: with several
    tiles per workgroup, a dX-only call (no dC rows to accumulate into), a dC-only call and a
    call with both match the oracle, and dC is deterministic.  Shapes: a factored input frame,
    and directly applied frames (token-grouped tiles in bf16)."""
    n, rn, m, rm, nnz = shape
    f_in, f_out = ff.framegen(n, n // rn, rn), ff.framegen(m, m // rm, rm)
    g = inputs.rng(4242)
    rows, cols = inputs.support(g, m, n, nnz)
    probe = ff.plan_create(f_in, f_out, rows, cols, max_tokens=1)
    tt = probe.tile_tokens(dtype)
    ncu = torch.cuda.get_device_properties(dev).multi_processor_count
    T = tt * (2 * ncu + 3) + 1   # two to three tiles per workgroup, a ragged last tile
    vals = inputs.gaussian(g, (nnz,), std=0.02)
    X = inputs.gaussian(g, (T, n), dtype=dtype)
    G = inputs.gaussian(g, (T, m), dtype=dtype)
    plan = ff.plan_create(f_in, f_out, rows, cols, max_tokens=T)
    assert plan.radix == ((4, 1) if n == 2752 else (1, 1)) and not plan.fast128
    assert plan.gen_token_groups
    Xd, Gd = torch_act(X, dtype, dev), torch_act(G, dtype, dev)
    c = plan_c(plan, vals, dev)
    s = -0.7
    dXo, _ = ff.adapter_bwd(plan, Xd, Gd, c, s, want_dc=False)
    _, dCo = ff.adapter_bwd(plan, Xd, Gd, c, s, want_dx=False)
    dX, dC = ff.adapter_bwd(plan, Xd, Gd, c, s)
    torch.cuda.synchronize()
    P_in, P_out = oracle_frame(n // rn, rn, n), oracle_frame(m // rm, rm, m)
    tok = _sample_tokens(T, 64, 11)
    dx_ref, _ = O.adapter_bwd(P_in, P_out, rows, cols, vals, s, X[tok], G[tok])
    dc_ref = O.coeff_grad_entries(P_in, P_out, rows, cols, s, X, G)
    tol = TOL[dtype]
    assert rel(to_np(dXo[tok]), dx_ref) <= tol
    assert rel(to_np(dX[tok]), dx_ref) <= tol
    assert rel(user_dc(plan, dCo), dc_ref) <= tol
    assert torch.equal(dC, dCo), "dC is not deterministic"


def test_grouped_tiles_several_walk_passes(dev):
    """bf16 token-grouped tiles of more than 20 tokens, whose sparse walks take several passes (in
    the backward the later passes add into the dC partial rows), with two tiles per backward
    workgroup: a 256 x 256 layer at 30,720 tokens, for which a call takes 60-token tiles.  y and dX
    on sampled tokens, dC over all tokens."""
    n = m = 256
    rn = 16
    nnz, T = 512, 30720
    f = ff.framegen(n, n // rn, rn)
    g = inputs.rng(7171)
    rows, cols = inputs.support(g, m, n, nnz)
    vals = inputs.gaussian(g, (nnz,), std=0.02)
    X = inputs.gaussian(g, (T, n), dtype="bf16")
    G = inputs.gaussian(g, (T, m), dtype="bf16")
    plan = ff.plan_create(f, f, rows, cols, max_tokens=T)
    assert plan.gen_token_groups and plan.gen_tile_tokens("bf16") >= 60 and not plan.fast128
    Xd, Gd = torch_act(X, "bf16", dev), torch_act(G, "bf16", dev)
    c = plan_c(plan, vals, dev)
    s = 0.37
    Y = ff.adapter_fwd(plan, Xd, c, s)
    dX, dC = ff.adapter_bwd(plan, Xd, Gd, c, s)
    _, dC2 = ff.adapter_bwd(plan, Xd, Gd, c, s, want_dx=False)
    torch.cuda.synchronize()
    P = oracle_frame(n // rn, rn, n)
    tok = _sample_tokens(T, 64, 12)
    y_ref = O.adapter_fwd(P, P, rows, cols, vals, s, X[tok])
    dx_ref, _ = O.adapter_bwd(P, P, rows, cols, vals, s, X[tok], G[tok])
    dc_ref = O.coeff_grad_entries(P, P, rows, cols, s, X, G)
    tol = TOL["bf16"]
    assert rel(to_np(Y[tok]), y_ref) <= tol
    assert rel(to_np(dX[tok]), dx_ref) <= tol
    assert rel(user_dc(plan, dC), dc_ref) <= tol
    assert torch.equal(dC, dC2), "dC is not deterministic"


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_generic_input_chunks(dev, dtype):
    """An input side too wide to sit whole next to the output side for 8 tokens (factored
    256-wide blocks) and a dense enough support (nnz >= 4 (n + m)): the generic kernels take the
    input side a chunk of blocks at a time.  The forward (v summed over chunks; also with beta)
    matches the oracle; with several tiles per workgroup, a dX-only call, a dC-only call and a
    call with both match the oracle, dC is deterministic, and beta accumulates into dX."""
    n, rn, m, rm, nnz = 8192, 64, 2048, 64, 42000
    f_in, f_out = ff.framegen(n, n // rn, rn), ff.framegen(m, m // rm, rm)
    g = inputs.rng(5151)
    rows, cols = inputs.support(g, m, n, nnz)
    probe = ff.plan_create(f_in, f_out, rows, cols, max_tokens=1)
    assert probe.gen_chunks > 1 and probe.radix == (4, 1) and not probe.fast128
    tt = probe.gen_tile_tokens(dtype)
    assert tt > probe.tile_tokens(dtype)
    ncu = torch.cuda.get_device_properties(dev).multi_processor_count
    T = tt * (ncu + 2) + 1   # more tiles than workgroups, a ragged last tile
    vals = inputs.gaussian(g, (nnz,), std=0.02)
    X = inputs.gaussian(g, (T, n), dtype=dtype)
    G = inputs.gaussian(g, (T, m), dtype=dtype)
    plan = ff.plan_create(f_in, f_out, rows, cols, max_tokens=T)
    Xd, Gd = torch_act(X, dtype, dev), torch_act(G, dtype, dev)
    c = plan_c(plan, vals, dev)
    s = 0.9
    Y = ff.adapter_fwd(plan, Xd, c, s)
    Y2 = Y.clone()
    ff.adapter_fwd(plan, Xd, c, s, Y=Y2, beta=1.0)
    dXo, _ = ff.adapter_bwd(plan, Xd, Gd, c, s, want_dc=False)
    _, dCo = ff.adapter_bwd(plan, Xd, Gd, c, s, want_dx=False)
    dX, dC = ff.adapter_bwd(plan, Xd, Gd, c, s)
    dX2 = dX.clone()
    ff.adapter_bwd(plan, Xd, Gd, c, s, dX=dX2, beta_dx=1.0, want_dc=False)
    torch.cuda.synchronize()
    P_in, P_out = oracle_frame(n // rn, rn, n), oracle_frame(m // rm, rm, m)
    tok = _sample_tokens(T, 48, 12)
    y_ref = O.adapter_fwd(P_in, P_out, rows, cols, vals, s, X[tok])
    dx_ref, _ = O.adapter_bwd(P_in, P_out, rows, cols, vals, s, X[tok], G[tok])
    dc_ref = O.coeff_grad_entries(P_in, P_out, rows, cols, s, X, G)
    tol = TOL[dtype]
    assert rel(to_np(Y[tok]), y_ref) <= tol
    assert rel(to_np(Y2[tok]), 2.0 * y_ref) <= tol
    assert rel(to_np(dXo[tok]), dx_ref) <= tol
    assert rel(to_np(dX[tok]), dx_ref) <= tol
    assert rel(to_np(dX2[tok]), 2.0 * dx_ref) <= tol
    assert rel(user_dc(plan, dCo), dc_ref) <= tol
    assert torch.equal(dC, dCo), "dC is not deterministic"


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(256, 16, 512, 32, 700, 37), (4096, 64, 4096, 64, 10000, 13)],
                         ids=lambda s: "n%d_m%d" % (s[0], s[2]))
def test_dc_only_without_coefficients(dev, shape, dtype):
    """A backward that asks only for dC needs no coefficients: with c_vals NULL (single call) and a
    NULL pointer array (batched call) dC still matches the oracle element by element, on the
    generic kernels (every fp32 call, and bf16 on the 256 -> 512 layer) and the fused ones."""
    n, rn, m, rm, nnz, T = shape
    rows, cols, vals, X, G = _problem(shape, dtype, seed=n + m + T + 17)
    k_in, k_out = n // rn, m // rm
    f_in, f_out = ff.framegen(n, k_in, rn), ff.framegen(m, k_out, rm)
    plan = ff.plan_create(f_in, f_out, rows, cols, max_tokens=T, max_batch=2)
    s = -0.37
    Xd, Gd = torch_act(X, dtype, dev), torch_act(G, dtype, dev)
    _, dC = ff.adapter_bwd(plan, Xd, Gd, None, s, want_dx=False)
    dCs = [torch.full((plan.coef_slots,), float("nan"), device=dev) for _ in range(2)]
    ff.adapter_bwd_batched(plan, [Xd, Xd], [Gd, Gd], None, s, None, dCs)
    torch.cuda.synchronize()
    P_in, P_out = oracle_frame(k_in, rn, n), oracle_frame(k_out, rm, m)
    bb = BwdBounds(P_in, P_out, rows, cols, vals, s, X, G, dtype, k_in, k_out)
    rep = {}
    _check("dC", user_dc(plan, dC), bb.dc, bb.bdc, rep)
    for i in range(2):
        assert torch.equal(dCs[i], dC)


@pytest.mark.parametrize("shape", [(256, 16, 512, 32, 700, 37), (4096, 64, 4096, 64, 10000, 13)],
                         ids=lambda s: "n%d_m%d" % (s[0], s[2]))
def test_coef_layout_conversion(dev, shape):
    """ff_coef_to_plan / ff_coef_to_user (Algorithm 1 step 4 on the device): a training step kept
    entirely in the caller's support order -- C converted to the plan layout, forward and
    backward, dC converted back (overwrite and accumulate) -- matches the oracle in user order;
    the conversions equal the host permutation exactly and write nothing outside their arrays."""
    n, rn, m, rm, nnz, T = shape
    dtype = "bf16"
    rows, cols, vals, X, G = _problem(shape, dtype, seed=n + 2 * m + T)
    k_in, k_out = n // rn, m // rm
    f_in, f_out = ff.framegen(n, k_in, rn), ff.framegen(m, k_out, rm)
    plan = ff.plan_create(f_in, f_out, rows, cols, max_tokens=T)
    L = plan.coef_slots
    s = 0.21
    cubuf, cu2 = guarded(1, nnz, nnz, "f32", dev, vals[None, :])
    cpbuf, cp2 = guarded(1, L, L, "f32", dev)
    ff.coef_to_plan(plan, cu2[0], cp2[0])
    Xd, Gd = torch_act(X, dtype, dev), torch_act(G, dtype, dev)
    Y = ff.adapter_fwd(plan, Xd, cp2[0], s)
    _, dCp = ff.adapter_bwd(plan, Xd, Gd, cp2[0], s, want_dx=False)
    dubuf, du2 = guarded(1, nnz, nnz, "f32", dev)
    ff.coef_to_user(plan, dCp, du2[0])
    acc = torch.from_numpy(np.arange(nnz, dtype=np.float32)).to(dev)
    ff.coef_to_user(plan, dCp, acc, accumulate=True)
    torch.cuda.synchronize()
    assert np.array_equal(to_np(cp2[0]), plan.to_plan(vals).astype(np.float64))
    assert np.array_equal(to_np(du2[0]), plan.to_user(to_np(dCp)))
    assert np.array_equal(to_np(acc), (np.arange(nnz, dtype=np.float32) + plan.to_user(to_np(dCp)).astype(np.float32)))
    for buf, w in ((cubuf, nnz), (cpbuf, L), (dubuf, nnz)):
        assert guards_intact(buf, 1, w, w, "f32")
    P_in, P_out = oracle_frame(k_in, rn, n), oracle_frame(k_out, rm, m)
    fb = FwdBounds(P_in, P_out, rows, cols, vals, s, X, dtype, k_in, k_out)
    bb = BwdBounds(P_in, P_out, rows, cols, vals, s, X, G, dtype, k_in, k_out)
    rep = {}
    _check("y coef", fb.coef(to_np(Y)), fb.v, fb.bv, rep)
    _check("dC user order", to_np(du2[0]), bb.dc, bb.bdc, rep)
    with pytest.raises(ff.FrameFTError):            # overlapping arrays are refused
        ff.coef_to_user(plan, dCp, dCp[:nnz])


def test_empty_batch_is_noop_and_zeroes_dc(dev):
    n = m = 256
    rows, cols, vals, X, G = _problem((n, 16, m, 16, 100, 4), "f32", 1)
    f = ff.framegen(256, 16, 16)
    plan = ff.plan_create(f, f, rows, cols, max_tokens=4)
    c = plan_c(plan, vals, dev)
    Xe = torch.zeros((0, n), device=dev)
    Ge = torch.zeros((0, m), device=dev)
    Y = ff.adapter_fwd(plan, Xe, c, 1.0)
    dC = torch.full((plan.coef_slots,), 7.0, device=dev)
    dX, dC = ff.adapter_bwd(plan, Xe, Ge, c, 1.0, dC=dC)
    torch.cuda.synchronize()
    assert Y.shape == (0, m) and dX.shape == (0, n)
    assert torch.all(dC == 0)


def test_argument_errors_write_nothing(dev):
    f = ff.framegen(256, 16, 16)
    rows, cols, vals, X, G = _problem((256, 16, 256, 16, 50, 8), "f32", 2)
    with pytest.raises(ff.FrameFTError) as ei:
        ff.plan_create(f, f, np.array([1, 1]), np.array([2, 2]), max_tokens=8)
    assert ei.value.name == "FF_EINVAL"
    with pytest.raises(ff.FrameFTError):
        ff.plan_create(f, f, np.array([256]), np.array([0]), max_tokens=8)
    plan = ff.plan_create(f, f, rows, cols, max_tokens=8)
    c = plan_c(plan, vals, dev)
    Y = torch.full((9, 256), 3.0, device=dev)
    with pytest.raises(ff.FrameFTError) as ei:       # T above max_tokens
        ff.adapter_fwd(plan, torch.zeros((9, 256), device=dev), c, 1.0, Y=Y)
    assert ei.value.name == "FF_EINVAL"
    Xb = torch.zeros((8, 256), device=dev, dtype=torch.bfloat16)
    Yb = torch.full((8, 256), 3.0, device=dev, dtype=torch.bfloat16)
    with pytest.raises(ff.FrameFTError):              # misaligned view
        ff.adapter_fwd(plan, Xb[:, 1:], c, 1.0, Y=Yb[:, 1:])
    torch.cuda.synchronize()
    assert torch.all(Y == 3.0) and torch.all(Yb == 3.0)


# ------------------------------------------------------------------ full-size configurations

def _sample_tokens(T, k, seed):
    g = np.random.default_rng(seed)
    extra = g.choice(T, size=min(k, T), replace=False)
    return np.unique(np.concatenate([[0, 1, T // 2, T - 1], extra]))


def _full_size_check(dev, wl_name, adapter_index=0, n_tok=48, n_nnz=384, n_rows=6, bwd_chunked=None):
    wl = inputs.WORKLOADS[wl_name]
    ad = wl.adapters[adapter_index]
    data = inputs.adapter_data(wl, ad, seed=wl.seed + adapter_index)
    T, dtype = wl.tokens, wl.dtype
    P_in = oracle_frame(ad.k_in, ad.rho_in, ad.d_in)
    P_out = oracle_frame(ad.k_out, ad.rho_out, ad.d_out)
    f_in = ff.framegen(ad.d_in, ad.k_in, ad.rho_in)
    f_out = ff.framegen(ad.d_out, ad.k_out, ad.rho_out)
    plan = ff.plan_create(f_in, f_out, data.rows, data.cols, max_tokens=T)
    if bwd_chunked is not None:
        assert (plan.gen_chunks > 1) == bwd_chunked
    Xd, Gd = torch_act(data.X, dtype, dev), torch_act(data.G, dtype, dev)
    c = plan_c(plan, data.vals, dev)
    Y = ff.adapter_fwd(plan, Xd, c, data.scale)
    dX, dC = ff.adapter_bwd(plan, Xd, Gd, c, data.scale)
    W0 = inputs.weight(inputs.rng(wl.seed + 99), ad.d_out, ad.d_in, "bf16")
    Wb = ff.merge_delta(plan, c, data.scale, torch_act(W0, "bf16", dev), beta=1.0)
    Wd = ff.merge_delta(plan, c, data.scale, torch.empty((ad.d_out, ad.d_in), device=dev), beta=0.0)
    torch.cuda.synchronize()
    tol = TOL[dtype]
    tok = _sample_tokens(T, n_tok, wl.seed)
    y_ref = O.adapter_fwd(P_in, P_out, data.rows, data.cols, data.vals, data.scale, data.X[tok])
    dx_ref, _ = O.adapter_bwd(P_in, P_out, data.rows, data.cols, data.vals, data.scale, data.X[tok],
                              data.G[tok])
    assert rel(to_np(Y[tok]), y_ref) <= tol
    assert rel(to_np(dX[tok]), dx_ref) <= tol
    ent = np.random.default_rng(wl.seed + 1).choice(ad.nnz, size=min(n_nnz, ad.nnz), replace=False)
    dc_ref = O.coeff_grad_entries(P_in, P_out, data.rows[ent], data.cols[ent], data.scale, data.X, data.G)
    assert rel(user_dc(plan, dC)[ent], dc_ref) <= tol
    r = np.unique(np.concatenate([[0, ad.d_out - 1], np.random.default_rng(wl.seed + 2).integers(0, ad.d_out, n_rows)]))
    dw_ref = O.merge_delta_rows(P_in, P_out, data.rows, data.cols, data.vals, data.scale, r)
    assert rel(to_np(Wd[r]), dw_ref) <= 1e-5
    assert merged_bf16_ok(to_np(Wb[r]), W0[r], dw_ref,
                          *merge_abs_terms(P_in, P_out, data.rows, data.cols, data.vals, data.scale,
                                          ad.rho_in, ad.rho_out, r), split=True)
    # the frames are orthogonal, so ||dW||_F = |s| ||C||_F for the whole matrix
    nrm = float(torch.linalg.vector_norm(Wd.double()))
    assert abs(nrm - abs(data.scale) * np.linalg.norm(data.vals.astype(np.float64))) <= 1e-5 * nrm


def test_cfg1_full(dev):
    _full_size_check(dev, "cfg1_256_fp32", n_tok=64, n_nnz=512, n_rows=256)


def test_cfg2_llama7b_qproj_full(dev):
    _full_size_check(dev, "cfg2_llama7b_qproj")


def test_cfg3_llama7b_mlp_up_full(dev):
    _full_size_check(dev, "cfg3_llama7b_mlp", adapter_index=0, n_tok=24, n_nnz=256, n_rows=4)


def test_cfg3_llama7b_mlp_down_full(dev):
    _full_size_check(dev, "cfg3_llama7b_mlp", adapter_index=1, n_tok=24, n_nnz=256, n_rows=4, bwd_chunked=False)


def test_cfg5_llama70b_down_full(dev):
    _full_size_check(dev, "cfg5_llama70b_down", n_tok=12, n_nnz=192, n_rows=3, bwd_chunked=True)


def test_cfg5_vitb16_qkv_full(dev):
    _full_size_check(dev, "cfg5_vitb16_qkv", n_tok=48, n_nnz=384, n_rows=8)


@pytest.mark.parametrize("group", [("q_proj", "k_proj", "v_proj", "o_proj"), ("gate_proj", "up_proj"),
                                   ("down_proj",)])
def test_cfg4_stack_batched_full(dev, group):
    """The 32-layer stack: one plan per projection shape (support shared across layers and
    projections), one batched call over layers {0, 31} x the group's projections at full
    per-adapter size (2048 tokens); every adapter checked on sampled tokens and entries."""
    wl = inputs.WORKLOADS["cfg4_llama7b_stack"]
    ads = [a for a in wl.adapters if a.name in group]
    ad0 = ads[0]
    layers = (0, wl.layers - 1)
    datas = [inputs.adapter_data(wl, ad, seed=wl.seed + 1000 * layer + 10 * i, support_seed=wl.seed + 10 * i)
             for layer in layers for i, ad in enumerate(ads)]
    # one support per group (the first adapter's draw), shared by every layer and projection
    rows, cols = datas[0].rows, datas[0].cols
    T, dtype = wl.tokens, wl.dtype
    f_in = ff.framegen(ad0.d_in, ad0.k_in, ad0.rho_in)
    f_out = ff.framegen(ad0.d_out, ad0.k_out, ad0.rho_out)
    count = len(datas)
    plan = ff.plan_create(f_in, f_out, rows, cols, max_tokens=T, max_batch=count)
    Xd = [torch_act(d.X, dtype, dev) for d in datas]
    Gd = [torch_act(d.G, dtype, dev) for d in datas]
    cd = [plan_c(plan, d.vals, dev) for d in datas]
    Yd = [torch.empty((T, ad0.d_out), dtype=Xd[0].dtype, device=dev) for _ in datas]
    dXd = [torch.empty((T, ad0.d_in), dtype=Xd[0].dtype, device=dev) for _ in datas]
    dCd = [torch.full((plan.coef_slots,), float("nan"), device=dev) for _ in datas]
    s = datas[0].scale
    ff.adapter_fwd_batched(plan, Xd, cd, s, Yd)
    ff.adapter_bwd_batched(plan, Xd, Gd, cd, s, dXd, dCd)
    torch.cuda.synchronize()
    P_in = oracle_frame(ad0.k_in, ad0.rho_in, ad0.d_in)
    P_out = oracle_frame(ad0.k_out, ad0.rho_out, ad0.d_out)
    tol = TOL[dtype]
    for i, d in enumerate(datas):
        tok = _sample_tokens(T, 16, wl.seed + i)
        y_ref = O.adapter_fwd(P_in, P_out, rows, cols, d.vals, s, d.X[tok])
        dx_ref, _ = O.adapter_bwd(P_in, P_out, rows, cols, d.vals, s, d.X[tok], d.G[tok])
        assert rel(to_np(Yd[i][tok]), y_ref) <= tol
        assert rel(to_np(dXd[i][tok]), dx_ref) <= tol
        ent = np.random.default_rng(wl.seed + i).choice(len(rows), size=128, replace=False)
        dc_ref = O.coeff_grad_entries(P_in, P_out, rows[ent], cols[ent], s, d.X, d.G)
        assert rel(user_dc(plan, dCd[i])[ent], dc_ref) <= tol


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(256, 16, 256, 16, 512, 64), (4096, 64, 4096, 64, 10_000, 40),
                                   (768, 64, 768, 64, 3_000, 37)],
                         ids=lambda s: "n%d_m%d_nnz%d_T%d" % (s[0], s[2], s[4], s[5]))
def test_block_diagonal_support(dev, shape, dtype):
    """C = diag(C_1..C_k) with the nonzeros spread uniformly over the diagonal blocks (Sec. 3.1,
    Sec. 3.3): forward, backward and merge against the oracle."""
    n, rn, m, rm, nnz, T = shape
    k = n // rn
    g = inputs.rng(n + nnz + T)
    rows, cols = inputs.support_block_diagonal(g, k, rm, rn, nnz)
    vals = inputs.gaussian(g, (nnz,), std=0.02)
    X = inputs.gaussian(g, (T, n), dtype=dtype)
    G = inputs.gaussian(g, (T, m), dtype=dtype)
    s = 0.31
    P_in, P_out = oracle_frame(k, rn, n), oracle_frame(m // rm, rm, m)
    f_in = ff.framegen(n, k, rn)
    f_out = f_in if (m, rm) == (n, rn) else ff.framegen(m, m // rm, rm)
    plan = ff.plan_create(f_in, f_out, rows, cols, max_tokens=T)
    c = plan_c(plan, vals, dev)
    Xd, Gd = torch_act(X, dtype, dev), torch_act(G, dtype, dev)
    Y = ff.adapter_fwd(plan, Xd, c, s)
    dX, dC = ff.adapter_bwd(plan, Xd, Gd, c, s)
    Wd = ff.merge_delta(plan, c, s, torch.zeros((m, n), device=dev), beta=0.0)
    torch.cuda.synchronize()
    tol = TOL[dtype]
    dx_ref, dc_ref = O.adapter_bwd(P_in, P_out, rows, cols, vals, s, X, G)
    assert rel(to_np(Y), O.adapter_fwd(P_in, P_out, rows, cols, vals, s, X)) <= tol
    assert rel(to_np(dX), dx_ref) <= tol
    assert rel(user_dc(plan, dC), dc_ref) <= tol
    assert rel(to_np(Wd), O.merge_delta(P_in, P_out, rows, cols, vals, s)) <= 1e-5


def test_hot_swap_merge_then_unmerge(dev):
    """Merging s P_out C P_in^T into W and then merging with -s (the hot swap of Sec. 3.4, "Storage efficiency") gives
    back W up to fp32 rounding, and the merged weight reproduces W0 x + adapter forward."""
    n = m = 4096
    rows, cols, vals, X, _ = _problem((n, 64, m, 64, 10_000, 16), "f32", 77)
    f = ff.framegen(n, 64, 64)
    plan = ff.plan_create(f, f, rows, cols, max_tokens=16)
    c = plan_c(plan, vals, dev)
    s = 200.0 / 4096.0
    W0 = torch.from_numpy(inputs.weight(inputs.rng(8), m, n, "f32")).to(dev)
    W = W0.clone()
    ff.merge_delta(plan, c, s, W, beta=1.0)
    Xd = torch.from_numpy(X).to(dev)
    y_merged = Xd @ W.T
    y_split = Xd @ W0.T + ff.adapter_fwd(plan, Xd, c, s)
    ff.merge_delta(plan, c, -s, W, beta=1.0)
    torch.cuda.synchronize()
    assert rel(to_np(y_merged), to_np(y_split)) <= 1e-5
    assert torch.max(torch.abs(W - W0)).item() <= 2.0 ** -20
