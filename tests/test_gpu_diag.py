"""GPU parity of opd_mc_diagnostics (Sec. 5.2, Fig. 5; App. E, Table 6)
against the oracle, through the C ABI, on the same fp32 inputs.

Tolerances.  The device forms rho = exp(log p - beta) and X = -rho A in fp32
(relative error ~1e-6 each):
  row_mean     |gpu - ref| <= 1e-5 (|ref| + s), s = mean_i |X_i| + 1
  row_var      |gpu - ref| <= 1e-4 (ref + s^2)
  row_rho_max, rho_quantile   relative 1e-5 (an order statistic moves no
               more than the values it orders)
  clip_frac    may differ only by entries whose |rho - 1| lies within 1e-5
               relative of clip_eps
  ratio_local, ratio_seq      relative 1e-3
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_24143_amd as opd
import synth
from gpu_common import say, to_dev

pytestmark = pytest.mark.gpu


def inputs(N, M, V=4000, seed=21, ragged=False):
    """fp32 lse / gathered from the oracle on generated rows, plus the cache."""
    w = synth.MC16.replace(N=N, V=V, M=M, seed=seed, dtype=synth.F32)
    d = synth.generate(w)
    ref = oracle.rows("rkl_mc", oracle.F32, d["logits"], V, ids=d["mc_ids"], tau=d["mc_tau"],
                      beta=d["mc_beta"], want_grad=False)
    lse = ref["lse"].astype(np.float32)
    gathered = ref["gathered"].astype(np.float32)
    mask = None
    if ragged:
        mask = (np.random.default_rng(seed).random(N) < 0.7).astype(np.uint8)
        mask[: min(N, 64)] = 0  # a whole masked sequence when seq_len <= 64
    return lse, gathered, d["mc_tau"], d["mc_beta"], mask


def compare(got, ref, tau, beta, lse, gathered, mask, eps):
    g = {k: v.cpu().numpy().astype(np.float64) for k, v in got.items()}
    valid = np.ones(lse.size, bool) if mask is None else mask == 1
    lp = gathered.astype(np.float64) - lse.astype(np.float64)[:, None]
    rho = np.exp(lp - beta.astype(np.float64))
    X = -rho * (tau.astype(np.float64) - lp)
    s = np.abs(X).mean(1) + 1.0
    if "row_mean" in g:
        err = np.abs(g["row_mean"] - ref["mean"])
        assert np.all(err[valid] <= 1e-5 * (np.abs(ref["mean"]) + s)[valid])
        assert np.all(g["row_mean"][~valid] == 0)
    if "row_var" in g and gathered.shape[1] >= 2:
        err = np.abs(g["row_var"] - ref["var"])
        assert np.all(err[valid] <= 1e-4 * (ref["var"] + s ** 2)[valid])
    if "row_rho_max" in g:
        err = np.abs(g["row_rho_max"] - ref["rho_max"])
        assert np.all(err[valid] <= 1e-5 * ref["rho_max"][valid] + 1e-30)
    if "rho_quantile" in g:
        assert abs(g["rho_quantile"][0] - ref["rho_quantile"]) <= 1e-5 * ref["rho_quantile"]
    if "clip_frac" in g:
        r = rho[valid].ravel()
        edge = np.sum(np.abs(np.abs(r - 1) - eps) <= 1e-5 * r)
        # plus the rounding of the fp32 output
        assert abs(g["clip_frac"][0] - ref["clip_frac"]) <= edge / r.size + 1e-7 * ref["clip_frac"]
    for k in ("ratio_local", "ratio_seq"):
        if k in g:
            assert np.allclose(g[k], ref[k], rtol=1e-3, atol=0), (k, g[k], ref[k])


@pytest.mark.parametrize("N,M,groups,seq,ragged", [
    (300, 16, (2, 4, 8), 0, False),
    (300, 16, (1, 2, 4, 8), 32, True),
    (64, 256, (1, 2, 128), 16, False),   # 256 draws: up to four groups per lane
    (257, 5, (), 0, True),               # M not a power of two, no groups
    (10, 1, (), 0, False),               # one draw: no variance
])
@pytest.mark.parametrize("q", [0.99, 0.5, 1.0])
def test_diag_parity(N, M, groups, seq, ragged, q):
    say("diag N=%d M=%d groups=%s seq=%d ragged=%s q=%g" % (N, M, groups, seq, ragged, q))
    lse, gathered, tau, beta, mask = inputs(N, M, ragged=ragged)
    eps = 0.2
    got = opd.mc_diagnostics(to_dev(lse), to_dev(gathered), to_dev(tau), to_dev(beta),
                             mask=None if mask is None else to_dev(mask), quantile=q,
                             clip_eps=eps, group_sizes=groups, seq_len=seq)
    torch.cuda.synchronize()
    # the ABI takes the quantile and clip range as fp32: the oracle gets those values
    ref = oracle.mc_diagnostics(lse, gathered, tau, beta, mask=mask, q=float(np.float32(q)),
                                eps=float(np.float32(eps)), group_sizes=groups, seq_len=seq)
    compare(got, ref, tau, beta, lse, gathered, mask, float(np.float32(eps)))
    if M == 1:
        assert np.all(np.isnan(got["row_var"].cpu().numpy()))


def test_diag_is_deterministic():
    lse, gathered, tau, beta, mask = inputs(500, 16, ragged=True)
    args = (to_dev(lse), to_dev(gathered), to_dev(tau), to_dev(beta))
    kw = dict(mask=to_dev(mask), group_sizes=(2, 4), seq_len=50)
    a = opd.mc_diagnostics(*args, **kw)
    b = opd.mc_diagnostics(*args, **kw)
    torch.cuda.synchronize()
    for k in a:
        assert torch.equal(a[k], b[k]), k


@pytest.mark.slow
def test_diag_full_size_after_the_loss_call():
    # the loss call's own lse_out and gathered_out feed the diagnostics
    w = synth.MC16
    say("diag full size %s" % w.name)
    d = synth.generate(w)
    logits = to_dev(d["logits"])
    ids, tau, beta = (to_dev(d[k]) for k in ("mc_ids", "mc_tau", "mc_beta"))
    out = opd.loss_fwd_bwd(logits, "rkl_mc", sampled_ids=ids, teacher_logp=tau, behav_logp=beta,
                           want_lse=True, want_gathered=True)
    groups = (2, 4, 8)
    got = opd.mc_diagnostics(out["lse"], out["gathered"].contiguous(), tau, beta,
                             group_sizes=groups, seq_len=2048)
    torch.cuda.synchronize()
    lse = out["lse"].cpu().numpy()
    gathered = out["gathered"].cpu().numpy()
    ref = oracle.mc_diagnostics(lse, gathered, d["mc_tau"], d["mc_beta"], group_sizes=groups,
                                seq_len=2048, q=float(np.float32(0.99)),
                                eps=float(np.float32(0.2)))
    compare(got, ref, d["mc_tau"], d["mc_beta"], lse, gathered, None, float(np.float32(0.2)))
    # the row means are the loss values themselves
    assert torch.allclose(got["row_mean"], out["loss"], rtol=1e-5, atol=1e-6)
    # iid draws: the fixed-prefix ratios follow 1/m (Table 6's column does too)
    r = got["ratio_local"].cpu().numpy()
    assert np.all(np.abs(r * np.array(groups) - 1) < 0.05), r
