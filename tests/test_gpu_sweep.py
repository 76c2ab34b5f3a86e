"""Exhaustive single-bit fault sweep of the tiny net on the GPU, compared
flag by flag with the oracle's sweep (tests/golden/tiny_sweep.npz, written
by tests/golden/make_tiny_sweep.py from the oracle alone).

Every bit of every deployed parameter (one forward per flip) and of every
stored activation element (4096 flips per pass, one per batch row) of one
seeded image is flipped; the GPU detector's flag (fused in the classifier
epilogue) and the critical label must equal the oracle's except inside the
documented rounding band."""

import json
import os

import numpy as np
import pytest

import oracle
from workloads import config, gen

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
GOLD = os.path.join(HERE, "golden", "tiny_sweep.npz")


def _say(*a):
    print(*a, flush=True)


def test_tiny_exhaustive_sweep_matches_oracle():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_16742_amd as P
    from paper_2609_16742_amd import ctc
    g = np.load(GOLD)
    summ = json.load(open(os.path.join(HERE, "golden", "tiny_sweep.json")))
    n = int(g["n"])
    flag_or = np.unpackbits(g["flag"])[:n].astype(bool)
    crit_or = np.unpackbits(g["critical"])[:n].astype(bool)
    fband = np.unpackbits(g["flag_band"])[:n].astype(bool)
    cband = np.unpackbits(g["critical_band"])[:n].astype(bool)

    net = config("tiny_f32_b1")
    params = gen.make_params(net)
    dp = oracle.protect_params(net, params)
    faults = gen.enumerate_faults(oracle.fault_sites(net, dp), image=0)
    import hashlib
    assert len(faults) == n == 1060544
    assert hashlib.sha256(faults.tobytes()).hexdigest()[:16] == \
        summ["fault_list_sha"]

    B = 4096
    cn = P.CtcNet(net.layers, net.in_shape, net.classes, net.dtype, params,
                  protect=True, max_batch=B)
    cn.set_threshold(float(g["ref"]), float(g["tau"]))
    x1 = torch.from_numpy(gen.make_inputs(net, 1)).cuda()
    xb = x1.expand(B, -1, -1, -1).contiguous()
    gold = cn.forward(x1)[0].cpu().numpy()
    out = torch.empty((n, net.classes + 1), device="cuda")
    flags = torch.zeros(n, dtype=torch.uint8, device="cuda")

    is_act = faults["site"] == gen.SITE_ACT
    pidx = np.nonzero(~is_act)[0]
    aidx = np.nonzero(is_act)[0]
    _say("parameter flips", len(pidx), "activation flips", len(aidx))
    h, st = cn.h, torch.cuda.current_stream().cuda_stream
    one = (ctc.ctc_fault * 1)()
    for i in pidx:
        f = faults[i]
        one[0] = ctc.ctc_fault(int(f["site"]), int(f["layer"]),
                               int(f["index"]), int(f["bit"]), 0)
        ctc._check(ctc._lib.ctc_inject_bitflip(h, one, 1, st))
        ctc.ctc_network_forward(h, 1, x1, out[i], flags[i],
                                ctc.CTC_REEXEC_NONE, st)
        ctc._check(ctc._lib.ctc_clear_faults(h, st))
    torch.cuda.synchronize()
    _say("parameter flips done")
    arr = (ctc.ctc_fault * B)()
    for s in range(0, len(aidx), B):
        ids = aidx[s:s + B]
        for r, i in enumerate(ids):
            f = faults[i]
            arr[r] = ctc.ctc_fault(int(f["site"]), int(f["layer"]),
                                   int(f["index"]), int(f["bit"]), r)
        ctc._check(ctc._lib.ctc_inject_bitflip(h, arr, len(ids), st))
        ob = torch.empty((B, net.classes + 1), device="cuda")
        fb = torch.zeros(B, dtype=torch.uint8, device="cuda")
        ctc.ctc_network_forward(h, B, xb, ob, fb, ctc.CTC_REEXEC_NONE, st)
        ctc._check(ctc._lib.ctc_clear_faults(h, st))
        idx_t = torch.from_numpy(ids).cuda()
        out[idx_t] = ob[:len(ids)]
        flags[idx_t] = fb[:len(ids)]
    torch.cuda.synchronize()
    _say("activation flips done")
    o = out.cpu().numpy()
    flag_gpu = flags.cpu().numpy().astype(bool)
    # the detector's flags are the verify of the stored S
    assert np.array_equal(flag_gpu, oracle.verify(o[:, -1], g["ref"],
                                                  g["tau"]))
    assert oracle.top1(gold[:-1]) == summ["golden_top1"]
    crit_gpu = np.array([oracle.is_critical(r[:-1], gold[:-1]) for r in o])
    keep_f, keep_c = ~fband, ~cband
    mf = np.nonzero(keep_f & (flag_gpu != flag_or))[0]
    mc = np.nonzero(keep_c & (crit_gpu != crit_or))[0]
    _say("flagged gpu", int(flag_gpu.sum()), "oracle", int(flag_or.sum()),
         "critical gpu", int(crit_gpu.sum()), "oracle", int(crit_or.sum()),
         "band", int(fband.sum()), int(cband.sum()),
         "mismatch", len(mf), len(mc))
    assert len(mf) == 0, [tuple(faults[i]) for i in mf[:10]]
    assert len(mc) == 0, [tuple(faults[i]) for i in mc[:10]]
    assert fband.sum() + cband.sum() <= 0.01 * n
