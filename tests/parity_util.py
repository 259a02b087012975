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


def merged_bf16_ok(got, W0, dW, dW_abs=None, depth=0):
    """bf16 merge check: within one bf16 ulp of RNE(W0 + dW), widened by the fp32 rounding of
    W0 + dW (2^-22 (|W0| + |dW|)), which matters only where the two nearly cancel.

    With dW_abs (the sum of the absolute values of the terms of each dW element, i.e. the
    merge of |P_out| |C| |P_in|^T) and depth (the largest number of support entries summed into
    one element), also by the recursive-summation bound of the kernel's fp32 arithmetic,
    (depth + 4) 2^-24 dW_abs: each term is a product of four fp32-rounded factors and each fused
    multiply-add rounds the running sum once.  Near W0 + dW = 0 that error is not small next to
    the bf16 spacing of the result."""
    from paper_2608_26430_amd import inputs
    exact = W0.astype(np.float64) + dW
    want = inputs.bf16_round(exact.astype(np.float32)).astype(np.float64)
    bound = bf16_ulp(want) + 2.0 ** -22 * (np.abs(W0) + np.abs(dW)) + 1e-30
    if dW_abs is not None:
        bound = bound + (depth + 4) * 2.0 ** -24 * 1.01 * np.asarray(dW_abs, dtype=np.float64)
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
