"""GPU fault-injection campaigns (Sec. III-A) against the oracle, on every
workload: the library's fault-site list equals the oracle's; a weight fault
writes exactly the oracle's flipped pattern into the deployed device weight
(binary16 patterns included, NaN payloads kept) and clearing restores it;
sampled (fault, image) inferences of parameter and activation campaigns
give the oracle's accumulated-checksum value S, the oracle's critical label
and -- read from the flag byte the detector fused in the classifier wrote
-- the oracle's detection flag.

Decision parity.  The detector compares |S - ref| with tau in fp32 on each
side's own S.  The two S values differ by at most the value tolerance, so
the flags can only legitimately differ where the oracle's deviation lies
within that discrepancy of tau: a flag is compared strictly whenever
| |S_or - ref| - tau | exceeds |S_gpu - S_or| plus two fp32 rounding units
of max(|S|, |ref|), and counted in the band otherwise.  Likewise a critical
label is compared whenever the oracle's top-2 logit gap exceeds twice the
largest logit discrepancy of that inference.  Band counts are printed and
must stay below 1% of the compared inferences.
"""

import os
import zlib
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle
from workloads import config, gen

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

RTOL = {"f32": 1e-4, "f16": 2e-2}
THREADS = min(16, os.cpu_count() or 1)
EPS32 = 2.0 ** -23


def _say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module")
def P():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_16742_amd as P
    return P


@pytest.mark.parametrize("label", ["tiny_f32_b1", "resnet20_f32_b128",
                                   "resnet18_f16_b64", "resnet18_f32_b64",
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


@pytest.mark.parametrize("label", ["resnet18_f16_b64", "mobilenetv2_f16_b128",
                                   "vgg16_f16_b32", "resnet20_f32_b128"])
def test_weight_faults_write_the_oracles_pattern(P, label):
    """Sampled weight faults plus two on one element that make a binary16
    signalling-NaN pattern (1.0 = 0x3c00, bits 14 then 0: 0x7c01): after
    inject, the deployed device element holds exactly the oracle's flipped
    pattern; after clear, the original one (XOR involution, Sec. III-A)."""
    net = config(label)
    params = gen.make_params(net)
    dp = oracle.protect_params(net, params)
    cn = P.CtcNet(net.layers, net.in_shape, net.classes, net.dtype, params,
                  protect=True, max_batch=2)
    f16 = net.dtype == "f16"
    sites = [s for s in oracle.fault_sites(net, dp) if s[0] == gen.SITE_WEIGHT]
    faults = [tuple(int(v) for v in (f["site"], f["layer"], f["index"],
                                     f["bit"], 0))
              for f in gen.sample_faults(sites, 40, 91)]
    # the carry-through filter of the first protected conv: a weight of 1.0
    L0 = next(i for i, p in enumerate(dp) if p is not None
              and net.layers[i]["op"] == "conv")
    w0 = dp[L0]["w"]
    ct = int(np.ravel_multi_index((w0.shape[0] - 1, 0, w0.shape[2] // 2,
                                   w0.shape[3] // 2), w0.shape))
    assert w0.reshape(-1)[ct] == 1.0
    groups = [[f] for f in faults] + [[(gen.SITE_WEIGHT, L0, ct, 14, 0),
                                       (gen.SITE_WEIGHT, L0, ct, 0, 0)]]

    def stored(layer, index):
        v = dp[layer]["w"].reshape(-1)[index:index + 1]
        if f16:
            return int(oracle.core.f16_pattern_of_stored(v)[0])
        return int(v.view(np.uint32)[0])

    _say("weight fault patterns", label, len(groups))
    for g in groups:
        before = [cn.weight_bits(f[1], f[2]) for f in g]
        assert before == [stored(f[1], f[2]) for f in g]
        cn.inject(g)
        for f in g:
            oracle.apply_param_fault(net, dp, f[0], f[1], f[2], f[3])
        after = [cn.weight_bits(f[1], f[2]) for f in g]
        assert after == [stored(f[1], f[2]) for f in g], (g, before, after)
        cn.clear_faults()
        for f in g[::-1]:
            oracle.apply_param_fault(net, dp, f[0], f[1], f[2], f[3])
        assert [cn.weight_bits(f[1], f[2]) for f in g] == before
    if f16:   # the signalling-NaN pattern reached the device unquieted
        cn.inject(groups[-1])
        assert cn.weight_bits(L0, ct) == 0x7c01
        cn.clear_faults()
        assert cn.weight_bits(L0, ct) == 0x3c00


# ------------------------------------------------------- campaign parity

def _oracle_fault_run(net, dp, x, T, f):
    """The oracle's output row under one fault, recomputed from the
    faulted layer on the golden activations T of image x."""
    site, layer, index, bit = (int(f[0]), int(f[1]), int(f[2]), int(f[3]))
    if site == gen.SITE_ACT:
        if layer == 0:
            return oracle.forward_image(net, dp, x, act_faults=[
                (0, index, bit)])
        acts = list(T)
        acts[layer] = T[layer].copy()
        oracle.core._flip(acts[layer], index, bit,
                          oracle.stored_f32(net, layer))
        if layer == len(net.layers):
            return acts[layer].reshape(-1).copy()
        return oracle.forward_image(net, dp, None, start=layer, acts=acts)
    ldp = list(dp)
    ldp[layer] = {k: v.copy() for k, v in dp[layer].items()}
    oracle.apply_param_fault(net, ldp, site, layer, index, bit)
    return oracle.forward_image(net, ldp, x, start=layer, acts=T)


class _Tally:
    def __init__(self):
        self.n = self.band_flag = self.band_crit = 0
        self.flagged = self.critical = 0
        self.max_rel_s = 0.0


def _check(net, tally, out_gpu, flag_gpu, out_or, gold_gpu, gold_or, ref,
           tau):
    """One (fault, image) inference: S within the value tolerance, the
    fused detector's flag byte equal to the decision on the GPU's own S and
    to the oracle's decision, the critical label (each side against its own
    golden run) equal to the oracle's, outside the data-derived bands of
    the module docstring."""
    rtol = RTOL[net.dtype]
    S_g, S_o = float(out_gpu[-1]), float(out_or[-1])
    tally.n += 1
    # the fused detector decides on its own S exactly (fp32 comparison)
    assert bool(flag_gpu) == bool(oracle.verify([S_g], ref, tau)[0])
    f_or = bool(oracle.verify([S_o], ref, tau)[0])
    if np.isfinite(S_o):
        assert np.isfinite(S_g), (S_g, S_o)
        d = abs(S_g - S_o)
        assert d <= rtol * abs(S_o), (S_g, S_o)
        tally.max_rel_s = max(tally.max_rel_s, d / max(abs(S_o), 1e-30))
        margin = d + 2 * EPS32 * max(abs(S_o), abs(S_g), abs(ref))
        if abs(abs(S_o - ref) - tau) <= margin:
            tally.band_flag += 1
        else:
            assert bool(flag_gpu) == f_or, (S_g, S_o, ref, tau)
    else:
        assert not np.isfinite(S_g), (S_g, S_o)
        assert bool(flag_gpu) and f_or
    tally.flagged += f_or
    crit_or = oracle.is_critical(out_or[:-1], gold_or[:-1])
    crit_g = oracle.is_critical(out_gpu[:-1], gold_gpu[:-1])
    tally.critical += crit_or
    near = False
    for lg, lo in ((out_gpu[:-1], out_or[:-1]), (gold_gpu[:-1], gold_or[:-1])):
        if np.all(np.isfinite(lo)):
            assert np.all(np.isfinite(lg)), (lg, lo)
            dl = np.max(np.abs(lg - lo))
            assert dl <= rtol * np.max(np.abs(lo)), (dl, np.max(np.abs(lo)))
            top2 = np.sort(lo)[-2:]
            near = near or top2[1] - top2[0] <= 2 * dl
        else:
            assert not np.all(np.isfinite(lg)), (lg, lo)
    if near:
        tally.band_crit += 1
        return
    assert crit_g == crit_or, (out_gpu, out_or)


# label, parameter faults, activation faults, sampled inferences of each
CAMPAIGNS = [
    ("tiny_f32_b1", 64, 64, 40),
    ("resnet20_f32_b128", 24, 128, 16),
    ("resnet18_f16_b64", 12, 64, 10),
    ("resnet18_f32_b64", 8, 64, 6),
    ("mobilenetv2_f16_b128", 16, 128, 12),
    ("vgg16_f16_b32", 6, 32, 5),
]


def _planted(net, dp):
    """Two faults every campaign carries, so that detected and critical
    inferences occur: bit 14 (fp16) / 30 (fp32) of the first protected
    conv's carry-through weight 1.0 (Inf, then NaN downstream: critical and
    flagged), and bit 30 of S in the final output row (flagged, never
    critical)."""
    L0 = next(i for i, p in enumerate(dp) if p is not None
              and net.layers[i]["op"] == "conv")
    w0 = dp[L0]["w"]
    ct = int(np.ravel_multi_index((w0.shape[0] - 1, 0, w0.shape[2] // 2,
                                   w0.shape[3] // 2), w0.shape))
    top = 14 if net.dtype == "f16" else 30
    return ((gen.SITE_WEIGHT, L0, ct, top, 0),
            (gen.SITE_ACT, len(net.layers), net.classes, 30, 0))


@pytest.mark.parametrize("label,nf,na,ns", CAMPAIGNS)
def test_campaign_flags_and_labels_match_oracle(P, label, nf, na, ns):
    """A parameter campaign (each fault on the whole batch) and an
    activation campaign (one fault per batch row) on the GPU through
    ctc_inject_bitflip; ns sampled inferences of each, the batch's first
    and last images always among them, recomputed by the oracle from the
    faulted layer.  Threshold: ref = the oracle's mean fault-free S of the
    sampled images, tau between their middle deviations from it (one
    image: 1% of |ref|), so that both decisions occur."""
    from paper_2609_16742_amd import campaign as C
    net = config(label)
    params = gen.make_params(net)
    dp = oracle.protect_params(net, params)
    B = net.batch
    run = C.Runner(net, params, max_batch=B)
    x = gen.make_inputs(net, B, offset=3 * B)
    xd = torch.from_numpy(x).cuda()
    g = np.random.default_rng(zlib.crc32(label.encode()))
    rows = sorted({0, B - 1} | {int(v) for v in g.integers(0, B, 2)})
    with ThreadPoolExecutor(THREADS) as ex:
        gold = dict(zip(rows, ex.map(lambda i: oracle.forward_image(
            net, dp, x[i], keep=True), rows)))
    S_gold = np.array([gold[i][-1].reshape(-1)[-1] for i in rows], np.float64)
    ref = float(S_gold.mean())
    dev = np.sort(np.abs(S_gold - ref))
    k = len(dev)
    # between the middle deviations of the sampled rows: faults that leave
    # S alone keep half the rows unflagged, the others flagged
    tau = 0.5 * (dev[k // 2 - 1] + dev[k // 2]) if k > 1 else 0.01 * abs(ref)
    run.cn.set_threshold(ref, tau)
    gold_gpu = run.cn.forward(xd).cpu().numpy()

    sites = oracle.fault_sites(net, dp)
    psites = [s for s in sites if s[0] != gen.SITE_ACT]
    asites = [s for s in sites if s[0] == gen.SITE_ACT]
    pf = gen.sample_faults(psites, nf, 201, stream=gen.S_FAULTS)
    af = gen.sample_faults(asites, na, 202, stream=gen.S_FAULTS)
    pw, pa = _planted(net, dp)
    pf[-1] = pw
    af[-1] = (pa[0], pa[1], pa[2], pa[3], 0)
    _say("campaign", label, nf, "parameter faults x", B, "images,", na,
         "activation faults")
    S1, t1, i1, f1 = run.param_campaign(pf, xd, chunk=8)
    S2, t2, i2, f2 = run.act_campaign(af, xd)
    # sampled inferences: (kind, fault index, batch row); the planted ones
    # on the first sampled row
    picks = {("p", nf - 1, rows[0])}
    while len(picks) < ns:
        picks.add(("p", int(g.integers(nf)), rows[len(picks) % len(rows)]))
    acand = [j for j in range(na) if j % B in rows and j != na - 1]
    g.shuffle(acand)
    apicks = {("a", na - 1, (na - 1) % B)} | {("a", j, j % B)
                                             for j in acand[:ns - 1]}
    picks = sorted(picks) + sorted(apicks)
    # the GPU's full output rows of the sampled inferences, rerun one by
    # one; they equal the campaign loops' S and image bookkeeping
    cols = net.classes + 1
    gpu_rows = {}
    out = torch.empty((B, cols), dtype=torch.float32, device="cuda")
    for kind, fi, r in picks:
        if (kind, fi) in gpu_rows:
            continue
        f = pf[fi] if kind == "p" else af[fi]
        run.cn.inject([(int(f["site"]), int(f["layer"]), int(f["index"]),
                        int(f["bit"]), r if kind == "a" else 0)])
        run.cn.forward(xd, out=out)
        run.cn.clear_faults()
        gpu_rows[(kind, fi)] = out.cpu().numpy().copy()
    for kind, fi, r in picks:
        s_run = gpu_rows[(kind, fi)][r, -1]
        s_camp = S1[fi, r] if kind == "p" else S2[fi]
        assert s_run == s_camp or (np.isnan(s_run) and np.isnan(s_camp))
        assert int(i1[fi, r] if kind == "p" else i2[fi]) == r

    def orun(p):
        kind, fi, r = p
        f = pf[fi] if kind == "p" else af[fi]
        ff = (int(f["site"]), int(f["layer"]), int(f["index"]), int(f["bit"]))
        return _oracle_fault_run(net, dp, x[r], gold[r], ff)

    with ThreadPoolExecutor(THREADS) as ex:
        ors = list(ex.map(orun, picks))
    tally = _Tally()
    for (kind, fi, r), o_or in zip(picks, ors):
        flag = f1[fi, r] if kind == "p" else f2[fi]
        _check(net, tally, gpu_rows[(kind, fi)][r], flag, o_or, gold_gpu[r],
               gold[r][-1].reshape(-1), ref, tau)
    _say("  compared", tally.n, "flag band", tally.band_flag, "critical band",
         tally.band_crit, "flagged", tally.flagged, "critical",
         tally.critical, "max rel S err %.3g" % tally.max_rel_s)
    assert tally.band_flag + tally.band_crit <= max(1, 0.01 * tally.n)
    assert 0 < tally.flagged < tally.n and tally.critical > 0


def test_fault_free_flags_match_oracle_mobilenetv2(P):
    """A 224x224 network at a calibrated threshold: tau from the oracle's
    own calibration (Sec. II-C, 256 fault-free inputs, alpha 5%); the flag
    bytes the fused detector writes for 128 fresh images equal the
    oracle's decisions outside the decision band."""
    net = config("mobilenetv2_f16_b128")
    params = gen.make_params(net)
    dp = oracle.protect_params(net, params)
    cal = oracle.forward_batch(net, dp, gen.make_inputs(
        net, 256, stream=gen.S_CALIB), threads=THREADS)[:, -1]
    ref, tau = oracle.calibrate(cal, 0.05)
    B = net.batch
    x = gen.make_inputs(net, B)
    ref_out = oracle.forward_batch(net, dp, x, threads=THREADS)
    cn = P.CtcNet(net.layers, net.in_shape, net.classes, net.dtype, params,
                  protect=True, max_batch=B)
    cn.set_threshold(ref, tau)
    fl = torch.zeros(B, dtype=torch.uint8, device="cuda")
    out = cn.forward(torch.from_numpy(x).cuda(), flags=fl)
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    f = fl.cpu().numpy()
    tally = _Tally()
    for i in range(B):
        _check(net, tally, o[i], f[i], ref_out[i], o[i], ref_out[i], ref,
               tau)
    _say("fault-free mobilenetv2: compared", tally.n, "band",
         tally.band_flag, "flagged", tally.flagged, "max rel S err %.3g"
         % tally.max_rel_s)
    assert tally.band_flag <= max(1, 0.01 * tally.n)
    assert 0 < tally.flagged < B


def test_detector_verify_equals_fused_detector(P):
    """The study's decisions at every (method, alpha) come from ctc_verify;
    at the deployed threshold they equal the flag bytes of the detector
    fused in the classifier, bit for bit."""
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
        fused = fl.cpu().numpy().astype(bool)
        assert np.array_equal(fused, C.detector_flags(out[:, -1], ref, tau))
        assert np.array_equal(fused, oracle.verify(out[:, -1], ref, tau))


def test_study_small_end_to_end(P):
    """The whole study on the tiny net at small sizes: thresholds ordered by
    alpha, FI-based false-positive rate on its own calibration campaign
    below alpha, rates in [0, 1], the fused detector agreeing with
    ctc_verify at the deployed threshold, overhead measured."""
    from paper_2609_16742_amd import campaign as C
    res = C.study("tiny_f32_b1", n_faults=300, n_act=300, n_cal=500,
                  eval_images=8, cal_images=8, overhead_passes=20,
                  log=_say)
    d, f = res["thresholds"]["distribution"], res["thresholds"]["fi"]
    assert d["0.001"]["tau"] >= d["0.01"]["tau"] >= d["0.05"]["tau"]
    assert f["0.001"]["tau"] >= f["0.01"]["tau"] >= f["0.05"]["tau"]
    for camp in ("parameter_campaign", "activation_campaign"):
        assert res[camp]["fused_detector_agrees"]
        for m in ("distribution", "fi"):
            for a in ("0.001", "0.01", "0.05"):
                r = res[camp][m][a]
                assert 0 <= r["FPR"] <= 1
                assert r["critical"] + r["noncritical"] > 0
    o = res["overhead_under_fi"]
    assert o["protected_s"] > 0 and o["unprotected_s"] > 0
