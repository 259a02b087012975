"""Plan groups: adapters over one frame pair, each with its own support (per-layer random masks,
tenants), in one launch per kernel; optionally each on its own number of tokens.

Every adapter is checked element by element against the oracle on its own support and tokens;
on the fused 128-wide kernels the group's results are also bitwise those of the single calls
(same kernels, same order of operations)."""
import numpy as np
import pytest

from oracle import frameft_oracle as O
from paper_2608_26430_amd import inputs
from tests.parity_util import (BwdBounds, FwdBounds, guarded, guards_intact, oracle_frame, to_np, torch_act,
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


# (n, rho_in, m, rho_out, nnz, dtype, T): fused 128-wide blocks, generic narrow blocks, and
# factored 344-wide input blocks
CASES = [(1024, 16, 2048, 32, 3000, "bf16", 45), (256, 16, 512, 32, 700, "f32", 37),
         (256, 16, 512, 32, 700, "bf16", 37), (2752, 16, 1024, 16, 4000, "bf16", 23)]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "n%d_m%d_%s" % (c[0], c[2], c[5]))
@pytest.mark.parametrize("ragged", [False, True], ids=["same_tokens", "per_adapter_tokens"])
def test_group_of_supports(dev, case, ragged):
    n, rn, m, rm, nnz, dtype, T = case
    k_in, k_out = n // rn, m // rm
    count = 4
    f_in, f_out = ff.framegen(n, k_in, rn), ff.framegen(m, k_out, rm)
    P_in, P_out = oracle_frame(k_in, rn, n), oracle_frame(k_out, rm, m)
    g = inputs.rng(n + m + nnz + T + ragged)
    sups = [inputs.support(g, m, n, nnz) for _ in range(count)]          # one random mask per adapter
    plans = [ff.plan_create(f_in, f_out, r, c, max_tokens=T) for r, c in sups]
    group = ff.plan_group(plans)
    vals = [inputs.gaussian(g, (nnz,), std=0.02) for _ in range(count)]
    Xs = [inputs.gaussian(g, (T, n), dtype=dtype) for _ in range(count)]
    Gs = [inputs.gaussian(g, (T, m), dtype=dtype) for _ in range(count)]
    toks = [T, 5, 0, T - 3] if ragged else [T] * count
    tokens = torch.tensor(toks, dtype=torch.int32, device=dev) if ragged else None
    s = 0.27
    Xd = [torch_act(x, dtype, dev) for x in Xs]
    Gd = [torch_act(x, dtype, dev) for x in Gs]
    cd = [torch.from_numpy(p.to_plan(v)).to(dev) for p, v in zip(plans, vals)]
    ybufs = [guarded(T, m, m + 8, dtype, dev) for _ in range(count)]
    dxbufs = [guarded(T, n, n + 8, dtype, dev) for _ in range(count)]
    Yd, dXd = [b[1] for b in ybufs], [b[1] for b in dxbufs]
    dCd = [torch.full((p.coef_slots,), float("nan"), device=dev) for p in plans]
    ff.adapter_fwd_group(group, Xd, cd, s, Yd, tokens=tokens)
    ff.adapter_bwd_group(group, Xd, Gd, cd, s, dXd, dCd, tokens=tokens)
    single = None
    if plans[0].fast128 and not ragged:
        single = [(ff.adapter_fwd(p, x, c, s), *ff.adapter_bwd(p, x, gg, c, s))
                  for p, x, gg, c in zip(plans, Xd, Gd, cd)]
    torch.cuda.synchronize()
    for i in range(count):
        t = toks[i]
        rows, cols = sups[i]
        # rows past the adapter's tokens (and every padding / guard element) are untouched
        assert guards_intact(ybufs[i][0], t, m, m + 8, dtype), f"adapter {i}: Y written past its tokens"
        assert guards_intact(dxbufs[i][0], t, n, n + 8, dtype), f"adapter {i}: dX written past its tokens"
        if t == 0:
            assert np.all(user_dc(plans[i], dCd[i]) == 0)
            continue
        fb = FwdBounds(P_in, P_out, rows, cols, vals[i], s, Xs[i][:t], dtype, k_in, k_out)
        bb = BwdBounds(P_in, P_out, rows, cols, vals[i], s, Xs[i][:t], Gs[i][:t], dtype, k_in, k_out)
        y, dx = to_np(Yd[i][:t]), to_np(dXd[i][:t])
        _ok(f"y[{i}]", y, fb.y, fb.by)
        _ok(f"y coef[{i}]", fb.coef(y), fb.v, fb.bv)
        _ok(f"dX[{i}]", dx, bb.dx, bb.bdx)
        _ok(f"dX coef[{i}]", bb.coef(dx), bb.q, bb.bq)
        _ok(f"dC[{i}]", user_dc(plans[i], dCd[i]), bb.dc, bb.bdc)
        if single is not None:
            assert torch.equal(single[i][0], Yd[i]) and torch.equal(single[i][1], dXd[i])
            assert torch.equal(single[i][2], dCd[i])


def test_group_mixes_fused_backward_tile_sizes(dev):
    """A sparse support runs the 16-token fused backward, a dense one (streams too long for its
    registers) the 8-token one; a group of both runs each adapter on its own kind, bitwise as the
    single calls, with per-adapter token counts."""
    n = m = 1024
    f = ff.framegen(n, 64, 16)
    g = inputs.rng(99)
    sups = [inputs.support(g, m, n, nnz) for nnz in (3000, 40000, 3000)]
    T = 40
    plans = [ff.plan_create(f, f, r, c, max_tokens=T) for r, c in sups]
    assert [p.bwd_tile_tokens for p in plans] == [16, 8, 16]
    group = ff.plan_group(plans)
    toks = [T, 19, 7]
    tokens = torch.tensor(toks, dtype=torch.int32, device=dev)
    X = [torch_act(inputs.gaussian(g, (T, n), dtype="bf16"), "bf16", dev) for _ in plans]
    G = [torch_act(inputs.gaussian(g, (T, m), dtype="bf16"), "bf16", dev) for _ in plans]
    c = [torch.from_numpy(p.to_plan(inputs.gaussian(g, (len(r),), std=0.02))).to(dev) for p, (r, _) in zip(plans, sups)]
    dX = [torch.zeros((T, n), dtype=torch.bfloat16, device=dev) for _ in plans]
    dC = [torch.empty((p.coef_slots,), device=dev) for p in plans]
    ff.adapter_bwd_group(group, X, G, c, 0.3, dX, dC, tokens=tokens)
    torch.cuda.synchronize()
    for i, p in enumerate(plans):
        t = toks[i]
        rx, rc = ff.adapter_bwd(p, X[i][:t], G[i][:t], c[i], 0.3)
        torch.cuda.synchronize()
        assert torch.equal(rx, dX[i][:t]) and torch.all(dX[i][t:] == 0)
        assert torch.equal(rc, dC[i])


def test_group_rejects_mismatched_plans(dev):
    f16, f32_ = ff.framegen(256, 16, 16), ff.framegen(512, 16, 32)
    r, c = inputs.support(inputs.rng(1), 256, 256, 300)
    a = ff.plan_create(f16, f16, r, c, max_tokens=8)
    r2, c2 = inputs.support(inputs.rng(2), 512, 256, 300)
    b = ff.plan_create(f16, f32_, r2, c2, max_tokens=8)
    with pytest.raises(ff.FrameFTError) as ei:        # other frames
        ff.plan_group([a, b])
    assert ei.value.name == "FF_EINVAL"
    with pytest.raises(ff.FrameFTError):              # the same plan twice
        ff.plan_group([a, a])


def test_group_zero_tokens_clear_dc(dev):
    f = ff.framegen(1024, 16, 64)
    plans = [ff.plan_create(f, f, *inputs.support(inputs.rng(i), 1024, 1024, 2000), max_tokens=16) for i in range(3)]
    group = ff.plan_group(plans)
    X = [torch.zeros((16, 1024), dtype=torch.bfloat16, device=dev)] * 3
    dCs = [torch.full((p.coef_slots,), 7.0, device=dev) for p in plans]
    ff.adapter_bwd_group(group, X, X, None, 1.0, None, dCs, T=0)
    torch.cuda.synchronize()
    assert all(torch.all(d == 0) for d in dCs)
