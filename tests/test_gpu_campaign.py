"""GPU fault-injection campaigns (Sec. III-A) against the oracle: the
library's fault-site list equals the oracle's, and sampled (fault, image)
inferences of a campaign give the oracle's accumulated-checksum value,
critical label and detection flag (outside the documented rounding band).
"""

import numpy as np
import pytest

import oracle
from workloads import by_name, config, gen

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

RTOL = {"f32": 1e-4, "f16": 2e-2}


def _say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module")
def P():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_16742_amd as P
    return P


@pytest.mark.parametrize("label", ["tiny_f32_b1", "resnet20_f32_b128",
                                   "mobilenetv2_f16_b128", "vgg16_f16_b32"])
def test_fault_sites_match_oracle(P, label):
    net = config(label)
    params = gen.make_params(net)
    _say("fault sites", label)
    cn = P.CtcNet(net.layers, net.in_shape, net.classes, net.dtype, params,
                  protect=True, max_batch=2)
    got = [tuple(int(v) for v in s) for s in cn.fault_sites(with_acts=True)]
    want = [tuple(int(v) for v in s) for s in
            oracle.fault_sites(net, oracle.protect_params(net, params))]
    assert got == want


def _band_flag(S, ref, tau, rtol):
    if not np.isfinite(S):
        return False
    return abs(abs(S - ref) - tau) <= 4 * rtol * max(abs(S), abs(ref))


def _band_crit(logits, rtol):
    if not np.all(np.isfinite(logits)):
        return False
    t = np.sort(logits)[-2:]
    return t[1] - t[0] <= 4 * rtol * np.max(np.abs(logits))


def _check_sample(net, S_gpu, top_gpu, out_or, gold_or, ref, tau, rtol):
    S_or = float(out_or[-1])
    if np.isfinite(S_or):
        assert abs(float(S_gpu) - S_or) <= rtol * max(abs(S_or), 1e-30) \
            or abs(float(S_gpu) - S_or) <= rtol * abs(ref), (S_gpu, S_or)
    else:
        assert not np.isfinite(S_gpu)
    from paper_2609_16742_amd import campaign as C
    fl_gpu = bool(C.flags_at([S_gpu], ref, tau)[0])
    fl_or = bool(oracle.verify([S_or], ref, tau)[0])
    if not _band_flag(S_or, ref, tau, rtol):
        assert fl_gpu == fl_or
    crit_gpu = top_gpu < 0 or top_gpu != oracle.top1(gold_or[:-1])
    crit_or = oracle.is_critical(out_or[:-1], gold_or[:-1])
    if not (_band_crit(out_or[:-1], rtol) or _band_crit(gold_or[:-1], rtol)):
        assert crit_gpu == crit_or


@pytest.mark.parametrize("label,nf,ns", [("tiny_f32_b1", 64, 64),
                                         ("resnet20_f32_b128", 24, 24)])
def test_param_campaign_matches_oracle(P, label, nf, ns):
    from paper_2609_16742_amd import campaign as C
    net = config(label)
    params = gen.make_params(net)
    B = max(net.batch, 4)
    run = C.Runner(net, params, max_batch=B)
    dp = oracle.protect_params(net, params)
    sites = run.cn.fault_sites(with_acts=False)
    faults = gen.sample_faults(sites, nf, 77, stream=gen.S_FAULTS)
    x = gen.make_inputs(net, 2 * B)
    xd = torch.from_numpy(x).cuda()
    _say("campaign", label, nf, "faults x", B, "images")
    S, top, img = run.param_campaign(faults, xd, chunk=16)
    g = np.random.default_rng(5)
    picks = [(int(g.integers(nf)), int(g.integers(B))) for _ in range(ns)]
    cal = oracle.forward_batch(net, dp, gen.make_inputs(
        net, 256, stream=gen.S_CALIB), threads=8)[:, -1]
    ref, tau = oracle.calibrate(cal, 0.01)
    rtol = RTOL[net.dtype]
    gold = {}
    for fi, r in picks:
        i = int(img[fi, r])
        if i not in gold:
            gold[i] = oracle.forward_image(net, dp, x[i], keep=True)
        T = gold[i]
        f = faults[fi]
        oracle.apply_param_fault(net, dp, f["site"], f["layer"], f["index"],
                                 f["bit"])
        out_or = oracle.forward_image(net, dp, x[i], start=int(f["layer"]),
                                      acts=T)
        oracle.apply_param_fault(net, dp, f["site"], f["layer"], f["index"],
                                 f["bit"])
        _check_sample(net, S[fi, r], int(top[fi, r]), out_or,
                      T[-1].reshape(-1), ref, tau, rtol)


def test_act_campaign_matches_oracle(P):
    from paper_2609_16742_amd import campaign as C
    net = config("resnet20_f32_b128")
    params = gen.make_params(net)
    run = C.Runner(net, params, max_batch=16)
    dp = oracle.protect_params(net, params)
    sites = [s for s in run.cn.fault_sites(with_acts=True)
             if s[0] == gen.SITE_ACT]
    faults = gen.sample_faults(sites, 40, 78, stream=gen.S_FAULTS)
    x = gen.make_inputs(net, 24)
    xd = torch.from_numpy(x).cuda()
    _say("activation campaign resnet20", len(faults))
    S, top, img = run.act_campaign(faults, xd)
    cal = oracle.forward_batch(net, dp, gen.make_inputs(
        net, 256, stream=gen.S_CALIB), threads=8)[:, -1]
    ref, tau = oracle.calibrate(cal, 0.01)
    nl = len(net.layers)
    for j in range(0, 40, 3):
        f = faults[j]
        i = int(img[j])
        T = oracle.forward_image(net, dp, x[i], keep=True)
        t = int(f["layer"])
        if t == 0:
            out_or = oracle.forward_image(net, dp, x[i], act_faults=[
                (0, int(f["index"]), int(f["bit"]))])
        else:
            acts = list(T)
            acts[t] = T[t].copy()
            oracle.core._flip(acts[t], int(f["index"]), int(f["bit"]),
                              oracle.stored_f32(net, t))
            out_or = (acts[t].reshape(-1) if t == nl else
                      oracle.forward_image(net, dp, None, start=t, acts=acts))
        _check_sample(net, S[j], int(top[j]), out_or, T[-1].reshape(-1),
                      ref, tau, RTOL[net.dtype])


def test_host_decision_equals_fused_detector(P):
    """flags_at (used to sweep thresholds offline) takes the same fp32
    decision as the detector fused in the classifier epilogue."""
    from paper_2609_16742_amd import campaign as C
    net = config("resnet20_f32_b128")
    params = gen.make_params(net)
    run = C.Runner(net, params, max_batch=128)
    x = torch.from_numpy(gen.make_inputs(net, 128)).cuda()
    out = run.cn.forward(x).cpu().numpy()
    S = out[:, -1].astype(np.float64)
    ref = float(np.mean(S))
    for tau in np.quantile(np.abs(S - ref), [0.5, 0.9, 0.99]):
        run.cn.set_threshold(ref, float(tau))
        fl = torch.zeros(128, dtype=torch.uint8, device="cuda")
        o2 = torch.empty_like(torch.from_numpy(out)).cuda()
        from paper_2609_16742_amd import ctc
        ctc.ctc_network_forward(run.cn.h, 128, x, o2, fl,
                                ctc.CTC_REEXEC_SYNC, None)
        torch.cuda.synchronize()
        assert np.array_equal(fl.cpu().numpy().astype(bool),
                              C.flags_at(out[:, -1], ref, tau))


def test_study_small_end_to_end(P):
    """The whole study on the tiny net at small sizes: thresholds ordered by
    alpha, FI-based false-positive rate on its own calibration campaign
    below alpha, rates in [0, 1], overhead measured."""
    from paper_2609_16742_amd import campaign as C
    res = C.study("tiny_f32_b1", n_faults=300, n_act=300, n_cal=500,
                  eval_images=8, cal_images=8, overhead_passes=20,
                  log=_say)
    d, f = res["thresholds"]["distribution"], res["thresholds"]["fi"]
    assert d["0.001"]["tau"] >= d["0.01"]["tau"] >= d["0.05"]["tau"]
    assert f["0.001"]["tau"] >= f["0.01"]["tau"] >= f["0.05"]["tau"]
    for camp in ("parameter_campaign", "activation_campaign"):
        for m in ("distribution", "fi"):
            for a in ("0.001", "0.01", "0.05"):
                r = res[camp][m][a]
                assert 0 <= r["FPR"] <= 1
                assert r["critical"] + r["noncritical"] > 0
    o = res["overhead_under_fi"]
    assert o["protected_s"] > 0 and o["unprotected_s"] > 0
