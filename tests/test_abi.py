"""CPU-side checks of the C ABI: the library loads, exports what include/frameft.h
declares, validates arguments, and its host frame construction equals the oracle's."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2608_26430_amd as ff
from paper_2608_26430_amd import binding
from oracle import frameft_oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "frameft.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ff_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(binding.library_path())
    names = _declared()
    assert len(names) >= 17, names
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings_and_version():
    lib = binding._load()
    assert lib.ff_abi_version() == 1
    for code, name in [(0, "FF_OK"), (1, "FF_EINVAL"), (2, "FF_ENOTFF"), (3, "FF_EUNSUPPORTED"),
                       (4, "FF_ENOMEM"), (5, "FF_EDEVICE"), (99, "FF_UNKNOWN")]:
        assert lib.ff_status_string(code).decode() == name


@pytest.mark.parametrize("k,rho,d", [(6, 6, 22), (2, 4, 8), (1, 8, 8), (4, 12, 48), (5, 8, 40),
                                     (16, 16, 256), (3, 10, 30), (12, 64, 768), (36, 64, 2304),
                                     (64, 64, 4096)])
def test_host_frame_equals_oracle(k, rho, d):
    ref = O.tight_fusion_frame(k, rho, d).toarray()
    got = ff.tff_host(d, k, rho)
    assert got.shape == ref.shape
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-13)


def test_host_frame_column_window():
    ref = O.tight_fusion_frame(172, 64, 11008)
    cols = [0, 1, 2, 63, 64, 5000, 11007]
    got = np.stack([ff.tff_host(11008, 172, 64, c, 1)[:, 0] for c in cols], axis=1)
    np.testing.assert_allclose(got, ref[:, cols].toarray(), rtol=0, atol=1e-13)


@pytest.mark.parametrize("args,status", [((10, 2, 4), "FF_ENOTFF"), ((12, 4, 3), "FF_EINVAL"),
                                         ((11, 2, 4), "FF_EINVAL"), ((0, 1, 2), "FF_EINVAL"),
                                         ((6, 1, 8), "FF_ENOTFF")])
def test_host_frame_rejects(args, status):
    d, k, rho = args
    with pytest.raises(ff.FrameFTError) as ei:
        ff.tff_host(d, k, rho)
    assert ei.value.name == status


def test_host_frame_rejects_bad_column_range():
    with pytest.raises(ff.FrameFTError) as ei:
        ff.tff_host(8, 2, 4, 6, 4)
    assert ei.value.name == "FF_EINVAL"


def test_framegen_shape_checks_precede_device_use():
    # block widths the kernels do not take (2k not a multiple of 8 with k rho = d, not a multiple of
    # 4 for a redundant frame) and frames that are not tight are rejected on the host
    for (d, k, rho), status in [((22, 7, 6), "FF_EUNSUPPORTED"), ((16, 2, 8), "FF_EUNSUPPORTED"),
                                ((10, 2, 4), "FF_ENOTFF"), ((22, 4, 6), "FF_ENOTFF")]:
        with pytest.raises(ff.FrameFTError) as ei:
            ff.framegen(d, k, rho)
        assert ei.value.name == status


def test_null_handles_are_rejected_without_a_device():
    lib = binding._load()
    assert binding._STATUS[lib.ff_adapter_fwd(None, 1, 0, None, 0, None, 1.0, 0.0, None, 0, None)] == "FF_EINVAL"
    assert binding._STATUS[lib.ff_adapter_bwd(None, 1, 0, None, 0, None, 0, None, 1.0, 0.0, None, 0, 0, None,
                                              None)] == "FF_EINVAL"
    assert binding._STATUS[lib.ff_merge_delta(None, None, 1.0, 0, 0.0, None, 0, None)] == "FF_EINVAL"
    assert binding._STATUS[lib.ff_plan_create(None, None, 0, None, None, 1, 1, None)] == "FF_EINVAL"
    assert binding._STATUS[lib.ff_time_next_kernel(ctypes.c_void_p(1), None)] == "FF_EINVAL"
    assert lib.ff_last_error().decode() != ""
    lib.ff_frame_destroy(None)
    lib.ff_plan_destroy(None)


def test_framegen_without_device_reports_device_error():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    with pytest.raises(ff.FrameFTError) as ei:
        ff.framegen(256, 16, 16)
    assert ei.value.name == "FF_EDEVICE"


def test_lr_schedule_host_function_matches_oracle():
    from oracle import optim_oracle as OO
    for total, ratio in ((1000, 0.06), (217, 0.03), (5, 0.5)):
        warm = OO.warmup_steps(total, ratio)
        for step in list(range(0, total + 2, max(1, total // 37))) + [warm - 1, warm, warm + 1, total - 1]:
            want = OO.linear_warmup_lr(step, warm, total, 0.33)
            assert ff.lr_linear_warmup(step, warm, total, 0.33) == pytest.approx(want, rel=1e-14, abs=1e-300)
