"""Pins for the optimizer oracle (oracle/optim_oracle.py), each against something other than
itself: torch's AdamW and transformers' linear warmup schedule (library routines), the closed
form of Adam's first step, and pure decay under a zero gradient."""
import math

import numpy as np
import pytest

from oracle import optim_oracle as OO


def test_adamw_matches_torch_adamw_over_several_steps():
    torch = pytest.importorskip("torch")
    g = np.random.default_rng(0)
    c0 = g.standard_normal(257) * 0.02
    grads = [g.standard_normal(257) * s for s in (1.0, 0.3, 3.0, 0.01, 1.0, 0.5)]
    lrs = [0.12, 0.1, 0.05, 0.33, 0.2, 0.01]
    hp = dict(betas=(0.9, 0.999), eps=1e-8, weight_decay=0.01)
    p = torch.nn.Parameter(torch.tensor(c0, dtype=torch.float64))
    opt = torch.optim.AdamW([p], lr=lrs[0], **hp)
    c, m, v = c0.copy(), np.zeros_like(c0), np.zeros_like(c0)
    for t, (gr, lr) in enumerate(zip(grads, lrs), start=1):
        for group in opt.param_groups:
            group["lr"] = lr
        p.grad = torch.tensor(gr, dtype=torch.float64)
        opt.step()
        c, m, v = OO.adamw_step(c, gr, m, v, t, lr, 0.9, 0.999, 1e-8, 0.01)
        np.testing.assert_allclose(c, p.detach().numpy(), rtol=1e-13, atol=1e-16)
        st = opt.state[p]
        np.testing.assert_allclose(m, st["exp_avg"].numpy(), rtol=1e-13, atol=1e-18)
        np.testing.assert_allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-13, atol=1e-20)


def test_first_step_closed_form():
    """At t = 1 without decay the bias corrections undo the averaging exactly:
    m_hat = g and v_hat = g^2, so the step is lr g / (|g| + eps)."""
    g = np.array([3.0, -2.0, 1e-3, 0.0, -5e-9])
    c0 = np.array([0.5, 0.5, -0.1, 0.2, 0.0])
    c, m, v = OO.adamw_step(c0, g, np.zeros(5), np.zeros(5), 1, 0.1, 0.9, 0.999, 1e-8, 0.0)
    np.testing.assert_allclose(c, c0 - 0.1 * g / (np.abs(g) + 1e-8), rtol=1e-14, atol=1e-17)
    np.testing.assert_allclose(m, 0.1 * g, rtol=1e-15)
    np.testing.assert_allclose(v, 0.001 * g * g, rtol=1e-12)


def test_zero_gradient_is_pure_decay():
    c0 = np.array([1.0, -2.0, 0.25])
    c, m, v = c0.copy(), np.zeros(3), np.zeros(3)
    for t in range(1, 8):
        c, m, v = OO.adamw_step(c, np.zeros(3), m, v, t, 0.1, weight_decay=0.05)
    np.testing.assert_allclose(c, c0 * (1 - 0.1 * 0.05) ** 7, rtol=1e-14)
    assert np.all(m == 0) and np.all(v == 0)


@pytest.mark.parametrize("total,ratio", [(1000, 0.06), (217, 0.03), (50, 0.06)])
def test_linear_warmup_matches_transformers_schedule(total, ratio):
    torch = pytest.importorskip("torch")
    tr = pytest.importorskip("transformers")
    warm = OO.warmup_steps(total, ratio)
    assert warm == math.ceil(total * ratio)
    p = torch.nn.Parameter(torch.zeros(1))
    opt = torch.optim.SGD([p], lr=0.12)
    sch = tr.get_linear_schedule_with_warmup(opt, num_warmup_steps=warm, num_training_steps=total)
    for step in range(total + 3):
        assert OO.linear_warmup_lr(step, warm, total, 0.12) == pytest.approx(opt.param_groups[0]["lr"], abs=1e-15)
        opt.step()
        sch.step()
    assert OO.linear_warmup_lr(0, warm, total, 0.12) == 0.0
    assert OO.linear_warmup_lr(warm, warm, total, 0.12) == pytest.approx(0.12)
    assert OO.linear_warmup_lr(total, warm, total, 0.12) == 0.0
