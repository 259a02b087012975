"""AdamW on the coefficient values (ff_adamw_step, ff_adamw_step_batched) against the fp64
optimizer oracle, one step at a time from the GPU's own previous state, element by element.

Bound per element (fp32 arithmetic, u = 2^-24): the decay and the moment updates round a few
times each, the step lr m_hat / (sqrt(v_hat) + eps) about eight times relative to itself."""
import numpy as np
import pytest

from oracle import optim_oracle as OO
from paper_2608_26430_amd import inputs
from tests.parity_util import to_np

torch = pytest.importorskip("torch")
import paper_2608_26430_amd as ff  # noqa: E402

pytestmark = pytest.mark.gpu
U = 2.0 ** -24
HP = dict(beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    return torch.device("cuda:0")


def _f32(x):
    return float(np.float32(x))


def _check_step(c0, g, m0, v0, t, lr, c1, m1, v1):
    b1, b2, eps, wd = (_f32(HP[k]) for k in ("beta1", "beta2", "eps", "weight_decay"))
    lr = _f32(lr)
    rc, rm, rv = OO.adamw_step(c0, g, m0, v0, t, lr, b1, b2, eps, wd)
    step = np.abs(rc - np.asarray(c0, dtype=np.float64) * (1 - lr * wd))
    assert np.all(np.abs(c1 - rc) <= 8 * U * np.abs(c0) + 24 * U * step + 1e-30)
    assert np.all(np.abs(m1 - rm) <= 4 * U * (b1 * np.abs(m0) + (1 - b1) * np.abs(g)) + 1e-38)
    assert np.all(np.abs(v1 - rv) <= 4 * U * (b2 * np.abs(v0) + (1 - b2) * g * g) + 1e-38)


@pytest.mark.parametrize("n,offset", [(10007, 0), (4096, 1), (3, 0)])
def test_adamw_matches_oracle_over_a_schedule(dev, n, offset):
    """Five steps with the warmup schedule's rates, 16-byte aligned vectors with a ragged tail and
    vectors only 4-byte aligned (the scalar path)."""
    g = inputs.rng(n + offset)
    base = [torch.zeros(n + offset, device=dev) for _ in range(4)]
    c, gr, m, v = (b[offset:] for b in base)
    c.copy_(torch.from_numpy(inputs.gaussian(g, (n,), std=0.02)))
    total, warm = 20, OO.warmup_steps(20, 0.06)
    for t in range(1, 6):
        gt = inputs.gaussian(g, (n,), std=10.0 ** -t)
        gr.copy_(torch.from_numpy(gt))
        lr = OO.linear_warmup_lr(t, warm, total, 0.12)
        assert ff.lr_linear_warmup(t, warm, total, 0.12) == pytest.approx(lr, rel=1e-15, abs=0)
        c0, m0, v0 = to_np(c), to_np(m), to_np(v)
        ff.adamw_step(c, gr, m, v, lr, t, **HP)
        torch.cuda.synchronize()
        _check_step(c0, gt.astype(np.float64), m0, v0, t, lr, to_np(c), to_np(m), to_np(v))


def test_adamw_batched_matches_single_calls(dev):
    count, n = 5, 10000
    g = inputs.rng(77)
    cs = [torch.from_numpy(inputs.gaussian(g, (n,), std=0.02)).to(dev) for _ in range(count)]
    gs = [torch.from_numpy(inputs.gaussian(g, (n,))).to(dev) for _ in range(count)]
    ms = [torch.zeros(n, device=dev) for _ in range(count)]
    vs = [torch.zeros(n, device=dev) for _ in range(count)]
    ref = [(c.clone(), m.clone(), v.clone()) for c, m, v in zip(cs, ms, vs)]
    for t in (1, 2, 3):
        ff.adamw_step_batched(cs, gs, ms, vs, 0.1, t, **HP)
        for (c, m, v), gr in zip(ref, gs):
            ff.adamw_step(c, gr, m, v, 0.1, t, **HP)
    torch.cuda.synchronize()
    for (c, m, v), c2, m2, v2 in zip(ref, cs, ms, vs):
        assert torch.equal(c, c2) and torch.equal(m, m2) and torch.equal(v, v2)


def test_adamw_keeps_plan_padding_zero_and_rejects_bad_arguments(dev):
    """Stepping a plan-layout coefficient array with its plan-layout gradient leaves the padding
    slots at zero; step 0 and a negative rate are refused and write nothing."""
    n = m = 1024
    rows, cols = inputs.support(inputs.rng(3), m, n, 3000)
    f = ff.framegen(n, 16, 64)
    plan = ff.plan_create(f, f, rows, cols, max_tokens=8)
    g = inputs.rng(4)
    c = torch.from_numpy(plan.to_plan(inputs.gaussian(g, (3000,), std=0.02))).to(dev)
    X = torch.from_numpy(inputs.gaussian(g, (8, n), dtype="bf16")).to(dev, torch.bfloat16)
    G = torch.from_numpy(inputs.gaussian(g, (8, m), dtype="bf16")).to(dev, torch.bfloat16)
    _, dC = ff.adapter_bwd(plan, X, G, c, 0.2, want_dx=False)
    mm, vv = torch.zeros_like(c), torch.zeros_like(c)
    ff.adamw_step(c, dC, mm, vv, 0.1, 1, **HP)
    torch.cuda.synchronize()
    pad = plan.order < 0
    assert np.all(to_np(c)[pad] == 0) and np.all(to_np(mm)[pad] == 0)
    keep = c.clone()
    for bad in (dict(lr=0.1, step=0), dict(lr=-1.0, step=2)):
        with pytest.raises(ff.FrameFTError):
            ff.adamw_step(c, dC, mm, vv, bad["lr"], bad["step"], **HP)
    torch.cuda.synchronize()
    assert torch.equal(c, keep)
