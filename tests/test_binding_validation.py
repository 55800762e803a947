"""The Python binding rejects tensors the C ABI would misread, before any
library call: wrong dtypes (an int64 index tensor read as int32 pairs),
wrong shapes, row strides that differ from the logits' (the kernels address
every row-strided array at the logits' ld), non-contiguous cache arrays, and
tensors off the GPU.  Runs on the CPU: each case has exactly one defect, and
the binding raises ValueError before it would pass a pointer on."""
import pytest
import torch

import paper_2606_24143_amd as opd

N, V, K = 6, 64, 4


def loss_args(est="rkl_mc", **over):
    """Well-formed CPU arguments of loss_fwd_bwd (only the device is wrong)."""
    a = dict(logits=torch.zeros(N, V, dtype=torch.bfloat16))
    if est in opd.TOPK:
        a.update(idx=torch.zeros(N, K, dtype=torch.int32),
                 teacher_logp=torch.zeros(N, K, dtype=torch.float32))
    elif est in opd.DENSE:
        a.update(teacher_logits=torch.zeros(N, V, dtype=torch.bfloat16))
    else:
        a.update(sampled_ids=torch.zeros(N, K, dtype=torch.int32),
                 teacher_logp=torch.zeros(N, K, dtype=torch.float32),
                 behav_logp=torch.zeros(N, K, dtype=torch.float32))
    a.update(over)
    return a


def call(est, **over):
    a = loss_args(est, **over)
    logits = a.pop("logits")
    return opd.loss_fwd_bwd(logits, est, **a)


def test_well_formed_cpu_tensors_are_refused_for_the_device_only():
    for est in ("rkl_mc", "fkl_topk", "rkl_dense"):
        with pytest.raises(ValueError, match="GPU tensor"):
            call(est)


CASES = {
    "int64 idx (torch.topk's index dtype)":
        ("fkl_topk", dict(idx=torch.zeros(N, K, dtype=torch.int64)), "int32"),
    "int64 sampled ids": ("rkl_mc", dict(sampled_ids=torch.zeros(N, K, dtype=torch.int64)),
                          "int32"),
    "float64 teacher log-probs":
        ("rkl_mc", dict(teacher_logp=torch.zeros(N, K, dtype=torch.float64)), "float32"),
    "teacher log-probs of another width":
        ("rkl_mc", dict(teacher_logp=torch.zeros(N, K + 1)), "shape"),
    "behaviour log-probs of fewer rows":
        ("rkl_mc", dict(behav_logp=torch.zeros(N - 1, K)), "shape"),
    "transposed (non-contiguous) sampled ids":
        ("rkl_mc", dict(sampled_ids=torch.zeros(K, N, dtype=torch.int32).t()), "contiguous"),
    "mask of int32": ("rkl_mc", dict(mask=torch.ones(N, dtype=torch.int32)), "dtype"),
    "mask of another length": ("rkl_mc", dict(mask=torch.ones(N + 1, dtype=torch.uint8)),
                               "shape"),
    "teacher logits of another dtype":
        ("rkl_dense", dict(teacher_logits=torch.zeros(N, V, dtype=torch.float32)), "dtype"),
    "teacher logits with padded rows (another row stride)":
        ("fkl_dense", dict(teacher_logits=torch.zeros(N, V + 8, dtype=torch.bfloat16)[:, :V]),
         "row stride"),
    "missing teacher logits": ("fkl_dense", dict(teacher_logits=None), "teacher_logits"),
    "missing ids": ("rkl_topk", dict(idx=None), "idx"),
    "dlogits contiguous while the logits are padded":
        ("rkl_mc", dict(logits=torch.zeros(N, V + 8, dtype=torch.bfloat16)[:, :V],
                        out={"loss": torch.zeros(N), "dlogits": torch.zeros(N, V)}),
         "row stride"),
    "bf16 dlogits buffer with fp32 output requested":
        ("rkl_mc", dict(out={"loss": torch.zeros(N),
                             "dlogits": torch.zeros(N, V, dtype=torch.bfloat16)}), "dtype"),
    "dlogits narrower than V":
        ("rkl_mc", dict(out={"loss": torch.zeros(N), "dlogits": torch.zeros(N, V - 4)}),
         "shape"),
    "loss of float64": ("rkl_mc", dict(out={"loss": torch.zeros(N, dtype=torch.float64),
                                            "dlogits": torch.zeros(N, V)}), "float32"),
    "workspace of float32": ("rkl_mc", dict(workspace=torch.zeros(16)), "uint8"),
    "float16 logits": ("rkl_mc", dict(logits=torch.zeros(N, V, dtype=torch.float16)), "float32"),
}


@pytest.mark.parametrize("case", list(CASES))
def test_malformed_tensors_are_rejected(case):
    est, over, pattern = CASES[case]
    with pytest.raises((ValueError, TypeError), match=pattern):
        call(est, **over)


def test_unknown_estimator_and_gradient_dtype():
    with pytest.raises(ValueError, match="estimator"):
        opd.loss_fwd_bwd(torch.zeros(N, V), "kl_everything")
    with pytest.raises(ValueError, match="dlogits_dtype"):
        call("rkl_mc", dlogits_dtype=torch.float16)


def test_cache_builders_and_diagnostics_check_their_tensors():
    logits = torch.zeros(N, V, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="shape"):
        opd.sample_actions(logits, torch.zeros(N + 1, K))
    with pytest.raises(ValueError, match="float32"):
        opd.sample_actions(logits, torch.zeros(N, K, dtype=torch.float64))
    with pytest.raises(ValueError, match="int32"):
        opd.score_actions(logits, torch.zeros(N, K, dtype=torch.int64))
    with pytest.raises(ValueError, match="dtype"):
        opd.topk_support(logits, 4, mask=torch.ones(N, dtype=torch.float32))
    with pytest.raises(ValueError, match="GPU tensor"):
        opd.topk_support(logits, 4)
    f = torch.zeros(N, K)
    with pytest.raises(ValueError, match="lse"):
        opd.mc_diagnostics(torch.zeros(N + 1), f, f, f)
    with pytest.raises(ValueError, match="contiguous"):
        opd.mc_diagnostics(torch.zeros(N), f, torch.zeros(K, N).t(), f)
    with pytest.raises(ValueError, match="int32"):
        opd.validate_cache("rkl_topk", V, idx=torch.zeros(N, K, dtype=torch.int64),
                           teacher_logp=f)
