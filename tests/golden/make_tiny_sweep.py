"""Exhaustive single-bit fault sweep of the tiny net with the CPU oracle.

Writes tests/golden/tiny_sweep.npz and tiny_sweep.json: for every one of the
1,060,544 single-bit flips of one seeded input image (every bit of every
deployed parameter and of every stored activation element, Sec. III-A fault
model widened to activations) the detection flag (Sec. II-B) at the
distribution-based threshold (Sec. II-C, alpha = 1%, 2000 calibration
images), whether the flip is critical (changes the golden top-1), and
whether the flag or the critical label sits in the rounding band where a
different summation order may decide differently.  Uses only oracle/ and the
seeded workload generators.

    python tests/golden/make_tiny_sweep.py [--threads N]
"""

import argparse
import hashlib
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from workloads import config, gen  # noqa: E402

ALPHA = 0.01
N_CAL = 2000
RTOL = 1e-4


def fault_list(net, dp):
    return gen.enumerate_faults(oracle.fault_sites(net, dp), image=0)


def list_digest(faults):
    return hashlib.sha256(faults.tobytes()).hexdigest()[:16]


def band_flags(S, ref, tau):
    S = np.asarray(S, np.float64)
    dev = np.abs(S - ref)
    fin = np.isfinite(S)
    return fin & (np.abs(dev - tau) <= 4 * RTOL * np.maximum(np.abs(S),
                                                              abs(ref)))


def band_critical(logits):
    out = np.zeros(len(logits), bool)
    for i, lr in enumerate(logits):
        if np.all(np.isfinite(lr)):
            top2 = np.sort(lr)[-2:]
            out[i] = (top2[1] - top2[0]) <= 4 * RTOL * np.max(np.abs(lr))
    return out


def run(threads):
    net = config("tiny_f32_b1")
    params = gen.make_params(net)
    dp = oracle.protect_params(net, params)
    cal = oracle.forward_batch(net, dp, gen.make_inputs(
        net, N_CAL, stream=gen.S_CALIB), threads=threads)[:, -1]
    ref, tau = oracle.calibrate(cal, ALPHA)
    x = gen.make_inputs(net, 1)[0]
    T = oracle.forward_image(net, dp, x, keep=True)
    gold = T[-1].reshape(-1)
    faults = fault_list(net, dp)
    n = len(faults)
    outs = np.zeros((n, gold.size), np.float32)
    nl = len(net.layers)

    def work(lo, hi):
        ldp = [None if p is None else {k: v.copy() for k, v in p.items()}
               for p in dp]
        for i in range(lo, hi):
            f = faults[i]
            if f["site"] == gen.SITE_ACT:
                t = int(f["layer"])
                if t == 0:
                    outs[i] = oracle.forward_image(net, ldp, x, act_faults=[
                        (0, int(f["index"]), int(f["bit"]))])
                    continue
                acts = list(T)
                acts[t] = T[t].copy()
                oracle.core._flip(acts[t], int(f["index"]), int(f["bit"]),
                                  oracle.stored_f32(net, t))
                outs[i] = (acts[t].reshape(-1) if t == nl else
                           oracle.forward_image(net, ldp, None, start=t,
                                                acts=acts))
            else:
                oracle.apply_param_fault(net, ldp, f["site"], f["layer"],
                                         f["index"], f["bit"])
                outs[i] = oracle.forward_image(net, ldp, x,
                                               start=int(f["layer"]), acts=T)
                oracle.apply_param_fault(net, ldp, f["site"], f["layer"],
                                         f["index"], f["bit"])

    t0 = time.time()
    step = 4096
    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(lambda lo: work(lo, min(lo + step, n)),
                    range(0, n, step)))
    S = outs[:, -1]
    flag = oracle.verify(S, ref, tau)
    g1 = oracle.top1(gold[:-1])
    crit = np.array([oracle.is_critical(o[:-1], gold[:-1]) for o in outs])
    fband = band_flags(S, ref, tau)
    cband = band_critical(outs[:, :-1])
    dt = time.time() - t0

    groups = {}
    names = {gen.SITE_WEIGHT: "weight", gen.SITE_BIAS: "bias",
             gen.SITE_ACT: "activation"}
    for kind in (gen.SITE_WEIGHT, gen.SITE_BIAS, gen.SITE_ACT):
        m = faults["site"] == kind
        c, f_ = crit[m], flag[m]
        groups[names[kind]] = {
            "flips": int(m.sum()), "critical": int(c.sum()),
            "detected_critical": int((c & f_).sum()),
            "noncritical_flagged": int((~c & f_).sum()),
            "TPR": float((c & f_).sum() / max(c.sum(), 1)),
            "FPR": float((~c & f_).sum() / max((~c).sum(), 1))}
    summary = {
        "workload": "tiny_f32_b1", "image": "eval stream image 0",
        "alpha": ALPHA, "n_cal": N_CAL, "ref": ref, "tau": tau,
        "golden_S": float(gold[-1]), "golden_top1": g1,
        "flips": n, "fault_list_sha": list_digest(faults),
        "flagged": int(flag.sum()), "critical": int(crit.sum()),
        "detected_critical": int((crit & flag).sum()),
        "TPR": float((crit & flag).sum() / max(crit.sum(), 1)),
        "FPR": float((~crit & flag).sum() / max((~crit).sum(), 1)),
        "flag_band": int(fband.sum()), "critical_band": int(cband.sum()),
        "by_site": groups, "oracle_seconds": dt, "threads": threads,
        "command": "python tests/golden/make_tiny_sweep.py --threads %d"
                   % threads}
    np.savez_compressed(os.path.join(HERE, "tiny_sweep.npz"),
                        flag=np.packbits(flag), critical=np.packbits(crit),
                        flag_band=np.packbits(fband),
                        critical_band=np.packbits(cband),
                        n=np.int64(n), ref=np.float64(ref),
                        tau=np.float64(tau))
    with open(os.path.join(HERE, "tiny_sweep.json"), "w") as fh:
        json.dump(summary, fh, indent=1)
    print(json.dumps(summary, indent=1))


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--threads", type=int, default=os.cpu_count() or 1)
    run(ap.parse_args().threads)
