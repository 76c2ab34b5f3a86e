"""Fault-injection campaigns on the GPU and the detection-threshold study
(Sec. II-C, Sec. III-A and III-B).

A campaign injects single-bit flips through the library's own hook
(``ctc_inject_bitflip``), runs the protected network on the device and
records, per (fault, image) inference, the accumulated-checksum neuron S
and whether the fault was critical (the faulty top-1 class differs from
the same network's fault-free top-1; a NaN logit counts as a change).
From those records:

* distribution-based thresholds (Sec. II-C): ref = mean fault-free S over
  the calibration (training-analogue) inputs, tau = the order statistic
  that flags fewer than alpha of them (``ctc_threshold_from_samples``);
* FI-based thresholds (Sec. II-C): a campaign on the calibration inputs,
  tau = the order statistic over the non-critical faulty inferences at the
  fault-free ref, so that their false-positive rate stays below alpha
  (``ctc_threshold_at_ref``);
* TPR, FPR and Youden's J (Sec. III-A) of both methods for every alpha, on
  an independent campaign over the evaluation inputs;
* the fault-free flag rate of the distribution-based thresholds on a
  large set of further evaluation images (``--ff-images``), which should
  sit near alpha;
* the run-time overhead of detection + re-execution under injected faults
  (Sec. III-B): protected deferred-re-execution passes, each under a fresh
  parameter fault, against unprotected passes under the same faults.

Parameter faults (the paper's fault model) apply to a whole batch: one
sampled fault is evaluated on one batch of B images, i.e. B (fault, image)
inferences per forward pass.  Activation faults (one stored element of one
image) go one per batch row.  The number of parameter faults defaults to
the statistical fault-injection size for the network's parameter bits
(95% confidence, 1% margin: about 9604).

    python -m paper_2609_16742_amd.campaign --workload resnet20_f32_b128 \\
        --out results/campaign_resnet20_f32_b128.json
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np
import torch

from . import ctc
from .runtime import CtcNet

ALPHAS = (0.001, 0.01, 0.05)


# ------------------------------------------------------------ decisions

def detector_flags(S, ref, tau, device="cuda"):
    """The library's detector (``ctc_verify``, Sec. II-B) on accumulated-
    checksum values: flag = not(|S - ref| <= tau) in fp32, NaN and Inf
    flagged.  S is copied to the device as fp32 and verified there in
    chunks of the kernel's maximum batch; returns a bool array of S's
    shape."""
    shape = np.shape(S)
    S = np.ascontiguousarray(np.asarray(S, np.float32).reshape(-1))
    n = S.size
    if n == 0:
        return np.zeros(shape, bool)
    Sd = torch.from_numpy(S).to(device)
    fl = torch.empty(n, dtype=torch.uint8, device=device)
    cnt = torch.empty(1, dtype=torch.int32, device=device)
    for s in range(0, n, 4096):
        m = min(4096, n - s)
        ctc.ctc_verify(Sd[s:s + m], m, 1, ref, tau, fl[s:s + m], cnt, None)
    return fl.cpu().numpy().astype(bool).reshape(shape)


def top1_rows(logits):
    """Top-1 class per row (lowest index on ties), -1 for a row with a NaN
    logit."""
    logits = np.asarray(logits)
    t = np.argmax(logits, axis=-1)
    t[np.isnan(logits).any(axis=-1)] = -1
    return t


def rates(flags, critical):
    """TPR, FPR, Youden's J and the counts behind them."""
    flags = np.asarray(flags, bool).ravel()
    critical = np.asarray(critical, bool).ravel()
    nc, nn = int(critical.sum()), int((~critical).sum())
    det, fa = int((flags & critical).sum()), int((flags & ~critical).sum())
    tpr = det / nc if nc else float("nan")
    fpr = fa / nn if nn else float("nan")
    return {"TPR": tpr, "FPR": fpr, "J": tpr - fpr, "critical": nc,
            "noncritical": nn, "detected": det, "false_alarms": fa}


# ------------------------------------------------------------ the runner

class Runner:
    """A protected network bound on the device plus campaign loops."""

    def __init__(self, net, params, max_batch=None, device="cuda"):
        self.net = net
        self.B = int(max_batch or net.batch)
        self.cols = net.classes + 1
        self.device = device
        self.cn = CtcNet(net.layers, net.in_shape, net.classes, net.dtype,
                         params, protect=True, max_batch=self.B,
                         device=device)
        self.params = params

    # fault-free outputs of a host image set, chunks of B
    def forward_all(self, x):
        out = np.empty((len(x), self.cols), np.float32)
        for s in range(0, len(x), self.B):
            xd = torch.from_numpy(np.ascontiguousarray(x[s:s + self.B])) \
                .to(self.device)
            out[s:s + len(xd)] = self.cn.forward(xd).cpu().numpy()
        return out

    def param_campaign(self, faults, x_dev, chunk=64, progress=None):
        """Each parameter fault i runs on image batch i mod (E / B) of the
        device image set x_dev [E, C, H, W].  Returns S [n, B] (fp32), the
        top-1 [n, B], the image index [n, B] of every inference and the
        flag bytes the detector fused in the classifier wrote [n, B] (at
        the threshold set on the net)."""
        B, n = self.B, len(faults)
        nb = len(x_dev) // B
        if nb < 1:
            raise ValueError("need at least one batch of images")
        S = np.empty((n, B), np.float32)
        top = np.empty((n, B), np.int64)
        img = np.empty((n, B), np.int64)
        flags = np.empty((n, B), bool)
        buf = torch.empty((chunk, B, self.cols), dtype=torch.float32,
                          device=self.device)
        fbuf = torch.empty((chunk, B), dtype=torch.uint8, device=self.device)
        h = self.cn.h
        st = torch.cuda.current_stream().cuda_stream
        one = (ctc.ctc_fault * 1)()
        for c0 in range(0, n, chunk):
            c1 = min(n, c0 + chunk)
            for i in range(c0, c1):
                f = faults[i]
                one[0] = ctc.ctc_fault(int(f["site"]), int(f["layer"]),
                                       int(f["index"]), int(f["bit"]), 0)
                b = i % nb
                ctc._check(ctc._lib.ctc_inject_bitflip(h, one, 1, st))
                ctc.ctc_network_forward(h, B, x_dev[b * B:(b + 1) * B],
                                        buf[i - c0], fbuf[i - c0],
                                        ctc.CTC_REEXEC_NONE, st)
                ctc._check(ctc._lib.ctc_clear_faults(h, st))
                img[i] = b * B + np.arange(B)
            o = buf[:c1 - c0].cpu().numpy()
            S[c0:c1] = o[:, :, -1]
            top[c0:c1] = top1_rows(o[:, :, :-1])
            flags[c0:c1] = fbuf[:c1 - c0].cpu().numpy().astype(bool)
            if progress:
                progress(c1, n)
        return S, top, img, flags

    def act_campaign(self, faults, x_dev, progress=None):
        """Activation faults, one per batch row: fault j runs in row
        j mod B of pass j // B on image j mod E.  Returns S [n], top-1 [n],
        image index [n] and the fused detector's flag bytes [n]."""
        B, n, E = self.B, len(faults), len(x_dev)
        S = np.empty(n, np.float32)
        top = np.empty(n, np.int64)
        img = np.empty(n, np.int64)
        flags = np.empty(n, bool)
        out = torch.empty((B, self.cols), dtype=torch.float32,
                          device=self.device)
        fout = torch.empty(B, dtype=torch.uint8, device=self.device)
        xb = torch.empty((B,) + tuple(x_dev.shape[1:]), dtype=x_dev.dtype,
                         device=self.device)
        h = self.cn.h
        st = torch.cuda.current_stream().cuda_stream
        arr = (ctc.ctc_fault * B)()
        for p0 in range(0, n, B):
            p1 = min(n, p0 + B)
            ids = np.arange(p0, p1)
            src = torch.from_numpy(ids % E).to(self.device)
            xb[:p1 - p0] = x_dev[src]
            for r, j in enumerate(ids):
                f = faults[j]
                arr[r] = ctc.ctc_fault(int(f["site"]), int(f["layer"]),
                                       int(f["index"]), int(f["bit"]), r)
            ctc._check(ctc._lib.ctc_inject_bitflip(h, arr, p1 - p0, st))
            ctc.ctc_network_forward(h, p1 - p0, xb[:p1 - p0], out[:p1 - p0],
                                    fout[:p1 - p0], ctc.CTC_REEXEC_NONE, st)
            ctc._check(ctc._lib.ctc_clear_faults(h, st))
            o = out[:p1 - p0].cpu().numpy()
            S[p0:p1] = o[:, -1]
            top[p0:p1] = top1_rows(o[:, :-1])
            img[p0:p1] = ids % E
            flags[p0:p1] = fout[:p1 - p0].cpu().numpy().astype(bool)
            if progress:
                progress(p1, n)
        return S, top, img, flags

    def timed_overhead(self, faults, x_dev, ref, tau, passes, warmup=3):
        """Sec. III-B under FI: wall time of `passes` protected passes
        (deferred re-execution, detector at (ref, tau)) each under a fresh
        parameter fault, against the unprotected network under the same
        faults (same inject / clear calls).  Returns the two times and
        the number of re-executed images."""
        net, B = self.net, self.B
        un = CtcNet(net.layers, net.in_shape, net.classes, net.dtype,
                    self.params, protect=False, max_batch=B,
                    device=self.device)
        self.cn.set_threshold(ref, tau)
        st = torch.cuda.current_stream().cuda_stream
        nb = len(x_dev) // B
        outs_p = torch.empty((passes + warmup, B, self.cols),
                             dtype=torch.float32, device=self.device)
        flags = torch.zeros((passes + warmup, B), dtype=torch.uint8,
                            device=self.device)
        outs_u = torch.empty((B, net.classes), dtype=torch.float32,
                             device=self.device)
        one = (ctc.ctc_fault * 1)()

        def run(handle, k0, k, prot):
            for k_ in range(k0, k0 + k):
                f = faults[k_ % len(faults)]
                one[0] = ctc.ctc_fault(int(f["site"]), int(f["layer"]),
                                       int(f["index"]), int(f["bit"]), 0)
                b = k_ % nb
                ctc._check(ctc._lib.ctc_inject_bitflip(handle, one, 1, st))
                if prot:
                    ctc.ctc_network_forward(handle, B,
                                            x_dev[b * B:(b + 1) * B],
                                            outs_p[k_], flags[k_],
                                            ctc.CTC_REEXEC_DEFERRED, st)
                else:
                    ctc.ctc_network_forward(handle, B,
                                            x_dev[b * B:(b + 1) * B], outs_u,
                                            None, ctc.CTC_REEXEC_NONE, st)
                ctc._check(ctc._lib.ctc_clear_faults(handle, st))
            if prot:
                ctc.ctc_network_flush(handle, st)

        run(self.cn.h, 0, warmup, True)
        run(un.h, 0, warmup, False)
        torch.cuda.synchronize()
        times = {}
        for name, handle, prot in (("protected", self.cn.h, True),
                                   ("unprotected", un.h, False),
                                   ("protected_2", self.cn.h, True),
                                   ("unprotected_2", un.h, False)):
            if prot:
                flags[warmup:].zero_()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            run(handle, warmup, passes, prot)
            torch.cuda.synchronize()
            times[name] = time.perf_counter() - t0
        reexec = int(flags[warmup:].sum().item())
        tp = min(times["protected"], times["protected_2"])
        tu = min(times["unprotected"], times["unprotected_2"])
        del un
        return {"passes": passes, "images": passes * B,
                "protected_s": tp, "unprotected_s": tu,
                "overhead_pct": 100.0 * (tp / tu - 1.0),
                "flagged_images": reexec,
                "flag_rate": reexec / float(passes * B)}


# ------------------------------------------------------------ the study

def param_bits(sites):
    return int(sum(s[2] * s[3] for s in sites))


def study(workload, n_faults=None, n_act=None, n_cal=None, eval_images=None,
          cal_images=None, overhead_passes=200, seed=None, log=print,
          select="last", ff_images=8192):
    """Runs the full threshold study for one workload; returns a dict.
    ``select``: which channel of each layer the carry-through filter
    replaces -- "last" (the channel at the last index) or "l1" (the least
    important one by L1 norm, Sec. II-A, via ctc_select_channels_l1)."""
    from workloads import config, gen

    net = config(workload)
    params = gen.make_params(net)
    if select == "l1":
        params, _ = ctc.ctc_select_channels_l1(net.layers, params)
    elif select != "last":
        raise ValueError("select must be 'last' or 'l1'")
    run = Runner(net, params)
    B = run.B
    sites_p = run.cn.fault_sites(with_acts=False)
    sites_a = [s for s in run.cn.fault_sites(with_acts=True)
               if s[0] == ctc.CTC_SITE_ACT]
    nbits = param_bits(sites_p)
    n_faults = n_faults or gen.leveugle_sample_size(nbits)
    n_act = n_act or gen.leveugle_sample_size(param_bits(sites_a))
    # calibration set sizes as in the study plan: 10 000 fault-free
    # inputs for the 32x32 nets, 2000 for ResNet-18 / MobileNetV2, 500 VGG
    n_cal = n_cal or {"tiny": 10000, "resnet20": 10000,
                      "vgg16": 500}.get(net.name, 2000)
    eval_images = eval_images or 4 * B
    cal_images = cal_images or eval_images
    seed = gen.BASE_SEEDS[net.name] if seed is None else seed
    t_all = time.time()

    def prog(tag):
        last = [0.0]

        def f(i, n):
            if time.time() - last[0] > 20 or i == n:
                last[0] = time.time()
                log("  %s %d/%d" % (tag, i, n))
        return f

    # distribution-based thresholds from fault-free calibration inputs
    log("%s: fault-free calibration on %d images" % (workload, n_cal))
    xc = gen.make_inputs(net, max(n_cal, cal_images), stream=gen.S_CALIB)
    out_c = run.forward_all(xc)
    Sc = out_c[:n_cal, -1].astype(np.float64)
    dist = {}
    for a in ALPHAS:
        r, t = ctc.ctc_threshold_from_samples(Sc, a)
        dist[a] = {"ref": r, "tau": t}
    ref = dist[0.01]["ref"]

    # FI-based thresholds: campaign on the calibration inputs
    log("%s: calibration FI campaign, %d parameter faults x %d images"
        % (workload, n_faults, B))
    fc = gen.sample_faults(sites_p, n_faults, seed, stream=gen.S_FAULTS)
    xcd = torch.from_numpy(xc[:cal_images]).to(run.device)
    gold_c = top1_rows(out_c[:cal_images, :-1])
    S1, t1, i1, _ = run.param_campaign(fc, xcd, progress=prog("cal"))
    crit1 = t1 != gold_c[i1]
    fi = {}
    for a in ALPHAS:
        fi[a] = {"ref": ref,
                 "tau": ctc.ctc_threshold_at_ref(S1[~crit1], ref, a)}
    del xcd

    # evaluation: fault-free rate, parameter and activation campaigns
    log("%s: evaluation campaigns" % workload)
    xe = gen.make_inputs(net, eval_images)
    out_e = run.forward_all(xe)
    gold_e = top1_rows(out_e[:, :-1])
    xed = torch.from_numpy(xe).to(run.device)
    fe = gen.sample_faults(sites_p, n_faults, seed + 1, stream=gen.S_FAULTS)
    run.cn.set_threshold(dist[0.01]["ref"], dist[0.01]["tau"])
    S2, t2, i2, f2 = run.param_campaign(fe, xed, progress=prog("eval"))
    crit2 = t2 != gold_e[i2]
    fa = gen.sample_faults(sites_a, n_act, seed + 2, stream=gen.S_FAULTS)
    S3, t3, i3, f3 = run.act_campaign(fa, xed, progress=prog("act"))
    crit3 = t3 != gold_e[i3]

    def table(S, crit, fused):
        # every (method, alpha) decision by the library's detector; at the
        # deployed threshold (distribution-based, alpha 1%) it must equal
        # the flag bytes of the detector fused in the classifier
        t = {m: {str(a): dict(rates(detector_flags(S, th[a]["ref"],
                                                   th[a]["tau"], run.device),
                                    crit), tau=th[a]["tau"])
                 for a in ALPHAS}
             for m, th in (("distribution", dist), ("fi", fi))}
        same = detector_flags(S, dist[0.01]["ref"], dist[0.01]["tau"],
                              run.device)
        t["fused_detector_agrees"] = bool(np.array_equal(same, fused))
        return t

    # the fault-free flag rate again on a larger set of evaluation-stream
    # images (past the campaign's own few batches), so that it can be told
    # apart from alpha: the binomial standard error at n images is
    # sqrt(alpha (1 - alpha) / n)
    log("%s: fault-free flag rate on %d images" % (workload, ff_images))
    Sff = np.concatenate(
        [run.forward_all(x)[:, -1]
         for x in gen.input_chunks(net, ff_images, 1024, offset=eval_images)])
    res = {
        "workload": workload, "dtype": net.dtype, "batch": B,
        "channel_selection": select,
        "alphas": list(ALPHAS), "n_cal": n_cal,
        "calibration_images_fi": cal_images, "eval_images": eval_images,
        "parameter_bits": nbits,
        "parameter_faults": {"calibration": n_faults, "evaluation": n_faults},
        "inferences_per_parameter_fault": B,
        "activation_faults": n_act,
        "thresholds": {"distribution": {str(a): dist[a] for a in ALPHAS},
                       "fi": {str(a): fi[a] for a in ALPHAS}},
        "fault_free_flag_rate": {
            str(a): float(detector_flags(out_e[:, -1], dist[a]["ref"],
                                         dist[a]["tau"], run.device).mean())
            for a in ALPHAS},
        "fault_free_flag_rate_large": dict(
            {str(a): float(detector_flags(Sff, dist[a]["ref"], dist[a]["tau"],
                                          run.device).mean())
             for a in ALPHAS}, images=int(ff_images)) if ff_images else None,
        "parameter_campaign": dict(
            table(S2, crit2, f2),
            critical_fraction=float(crit2.mean())),
        "activation_campaign": dict(
            table(S3, crit3, f3),
            critical_fraction=float(crit3.mean())),
    }
    for m in ("distribution", "fi"):
        res["best_alpha_by_J_" + m] = max(
            ALPHAS, key=lambda a: res["parameter_campaign"][m][str(a)]["J"])
    if overhead_passes:
        log("%s: overhead under FI, %d passes" % (workload, overhead_passes))
        res["overhead_under_fi"] = run.timed_overhead(
            fe, xed, dist[0.01]["ref"], dist[0.01]["tau"], overhead_passes)
    res["seconds"] = time.time() - t_all
    res["seed"] = seed
    return res


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", default="resnet20_f32_b128")
    ap.add_argument("--faults", type=int, default=None,
                    help="parameter faults per campaign (default: the "
                         "95%%/1%% statistical size)")
    ap.add_argument("--act-faults", type=int, default=None)
    ap.add_argument("--ncal", type=int, default=None)
    ap.add_argument("--eval-images", type=int, default=None)
    ap.add_argument("--ff-images", type=int, default=8192,
                    help="images of the larger fault-free flag-rate set")
    ap.add_argument("--overhead-passes", type=int, default=200)
    ap.add_argument("--select", choices=("last", "l1"), default="last",
                    help="pruned channel: the last one, or the least "
                         "important by L1 norm")
    ap.add_argument("--out", default=None)
    a = ap.parse_args(argv)
    if not torch.cuda.is_available():
        sys.exit("campaigns run on the GPU")
    res = study(a.workload, a.faults, a.act_faults, a.ncal, a.eval_images,
                overhead_passes=a.overhead_passes,
                log=lambda s: print(s, flush=True), select=a.select,
                ff_images=a.ff_images)
    txt = json.dumps(res, indent=1)
    if a.out:
        os.makedirs(os.path.dirname(os.path.abspath(a.out)), exist_ok=True)
        with open(a.out, "w") as fh:
            fh.write(txt + "\n")
    print(json.dumps({k: res[k] for k in ("workload", "seconds")}))


if __name__ == "__main__":
    main()
