"""Host tests of the guarded-dispatch policy (no GPU): a variant goes to
libkf355 only when the call is supported, agrees with eager within the dtype
tolerance and is measured faster, each decision carries its reason, is made
once per variant, survives a save / load round trip, and install() /
uninstall() restore PyTorch's functions exactly.  The two paths are stand-in
callables and the timer is injected, so nothing touches a device."""
import os

import pytest
import torch
import torch.nn.functional as F

from paper_2607_24762_amd import dispatch, kf355


def fixed_timer(times):
    def timer(fn, reps):
        return times[fn.__name__]
    return timer


def kf_fn():
    return torch.tensor([1.0, 2.0])


def eager_fn():
    return torch.tensor([1.0, 2.0])


def test_faster_and_valid_goes_to_kf355():
    d = dispatch.GuardedDispatcher(timer=fixed_timer({"kf_fn": 1.0, "eager_fn": 5.0}))
    y = d.call("op", (torch.zeros(2),), kf_fn, eager_fn)
    (dec,) = d.decisions.values()
    assert dec.backend == "kf355" and dec.reason.startswith("faster") and dec.kf_us == 1.0
    assert torch.equal(y, kf_fn())


def test_slower_stays_on_eager():
    d = dispatch.GuardedDispatcher(timer=fixed_timer({"kf_fn": 9.0, "eager_fn": 5.0}))
    d.call("op", (torch.zeros(2),), kf_fn, eager_fn)
    (dec,) = d.decisions.values()
    assert dec.backend == "eager" and dec.reason.startswith("slower")


def test_invalid_result_stays_on_eager():
    d = dispatch.GuardedDispatcher(timer=fixed_timer({"kf_fn": 1.0, "bad": 1.0, "eager_fn": 5.0}))

    def bad():
        return torch.tensor([1.0, 2.5])
    d.call("op", (torch.zeros(2),), bad, eager_fn)
    (dec,) = d.decisions.values()
    assert dec.backend == "eager" and dec.reason.startswith("invalid") and dec.max_abs_diff == pytest.approx(0.5)


def test_tolerance_follows_output_dtype():
    d = dispatch.GuardedDispatcher(timer=fixed_timer({"near": 1.0, "ref": 5.0}))

    def ref():
        return torch.tensor([1.0, 0.5], dtype=torch.bfloat16)

    def near():   # one bf16 ulp away from ref at 1.0
        return torch.tensor([1.0078125, 0.5], dtype=torch.bfloat16)
    d.call("op", (torch.zeros(2, dtype=torch.bfloat16),), near, ref)
    assert next(iter(d.decisions.values())).backend == "kf355"


def test_unsupported_call_stays_on_eager_and_other_errors_propagate():
    d = dispatch.GuardedDispatcher(timer=fixed_timer({}))

    def unsupported():
        raise kf355.KfError(5, "only dense row-major tensors are supported")
    y = d.call("op", (torch.zeros(3),), unsupported, eager_fn)
    (dec,) = d.decisions.values()
    assert dec.backend == "eager" and dec.reason.startswith("unsupported") and torch.equal(y, eager_fn())

    def hip_failure():
        raise kf355.KfError(7, "launch failed")
    with pytest.raises(kf355.KfError):
        d.call("op", (torch.zeros(4),), hip_failure, eager_fn)


def test_decision_is_made_once_per_variant():
    calls = {"n": 0}

    def counted():
        calls["n"] += 1
        return torch.tensor([1.0, 2.0])
    d = dispatch.GuardedDispatcher(timer=lambda fn, reps: 1.0 if fn is counted else 2.0)
    for _ in range(5):
        d.call("op", (torch.zeros(2),), counted, eager_fn)
    assert len(d.decisions) == 1 and calls["n"] == 5   # one run while deciding, then 4 routed calls
    d.call("op", (torch.zeros(3),), counted, eager_fn)      # new shape: a new variant
    assert len(d.decisions) == 2


def test_save_and_load_round_trip(tmp_path):
    d = dispatch.GuardedDispatcher(timer=fixed_timer({"kf_fn": 1.0, "eager_fn": 5.0}))
    d.call("op", (torch.zeros(2), 3, 1e-5), kf_fn, eager_fn)
    path = os.path.join(tmp_path, "decisions.json")
    d.save(path)
    e = dispatch.GuardedDispatcher()
    e.load(path)
    assert e.report() == d.report()


def test_variant_key_distinguishes_layouts_and_arguments():
    x = torch.zeros(4, 6)
    k = dispatch.variant_key
    assert k("softmax", (x, -1)) != k("softmax", (x.t(), -1))            # strides
    assert k("softmax", (x, -1)) != k("softmax", (x, 0))                 # dim
    assert k("softmax", (x, -1)) != k("softmax", (x.bfloat16(), -1))     # dtype


def test_install_restores_and_passes_cpu_tensors_through():
    if not os.path.exists(kf355.LIB_PATH):
        pytest.skip("libkf355.so not built")
    originals = (torch.softmax, torch.Tensor.softmax, F.softmax, F.layer_norm, F.group_norm, F.adaptive_avg_pool2d,
                 F.max_pool2d)
    x = torch.randn(2, 8, 4, 4)
    with dispatch.installed() as d:
        assert torch.softmax is not originals[0]
        # CPU tensors are not eligible: the original functions run, nothing is decided.
        assert torch.equal(torch.softmax(x, -1), originals[0](x, -1))
        assert torch.equal(x.softmax(1), originals[1](x, 1))
        assert torch.equal(F.group_norm(x, 2), originals[4](x, 2))
        assert torch.equal(F.layer_norm(x, (4,)), originals[3](x, (4,)))
        assert torch.equal(F.adaptive_avg_pool2d(x, 1), originals[5](x, 1))
        y, i = F.max_pool2d(x, 2, return_indices=True)
        ty, ti = originals[6](x, 2, return_indices=True)
        assert torch.equal(y, ty) and torch.equal(i, ti)
        assert d.decisions == {}
    assert (torch.softmax, torch.Tensor.softmax, F.softmax, F.layer_norm, F.group_norm,
            F.adaptive_avg_pool2d, F.max_pool2d) == originals


def test_agree_scales_with_the_output_and_checks_specials():
    ref = torch.tensor([4.0, 0.0002670, -3.0], dtype=torch.bfloat16)
    near = torch.tensor([4.0, 0.00122, -3.0], dtype=torch.bfloat16)     # 2^-10 of the scale off near zero
    far = torch.tensor([4.0, 0.25, -3.0], dtype=torch.bfloat16)
    assert dispatch.agree(near, ref)[0]
    assert not dispatch.agree(far, ref)[0]
    nan = torch.tensor([float("nan"), 1.0])
    assert dispatch.agree(nan, nan.clone())[0]
    assert not dispatch.agree(torch.tensor([1.0, 1.0]), nan)[0]
    inf = torch.tensor([float("inf"), 1.0])
    assert dispatch.agree(inf, inf.clone())[0]
    assert not dispatch.agree(torch.tensor([-float("inf"), 1.0]), inf)[0]
    assert not dispatch.agree(torch.zeros(2), torch.zeros(3))[0]
    assert not dispatch.agree(torch.zeros(2), torch.zeros(2, dtype=torch.float64))[0]
    assert dispatch.agree(torch.zeros(0), torch.zeros(0))[0]


def test_agree_on_tuples_and_integer_outputs():
    y = torch.tensor([1.0, 2.0])
    i = torch.tensor([3, 4])
    assert dispatch.agree((y, i), (y.clone(), i.clone()))[0]
    assert not dispatch.agree((y, i), (y, torch.tensor([3, 5])))[0]     # indices must be equal
    assert not dispatch.agree((y,), (y, i))[0]
    assert not dispatch.agree(y, (y, i))[0]
