"""HIP graph replay (ctc_graph_*): a captured run of one-pass inferences
gives the same bits as the same passes issued one call at a time, and stays
within tolerance of the oracle; flagged images are re-run by a re-executing
launch (Sec. II-B); parameter faults injected after capture are seen.

Every test replays its graph several times, with eager work and
synchronisations between the replays, and checks every replay.
"""

import os

import numpy as np
import pytest

import oracle
from workloads import config, gen

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

THREADS = min(16, os.cpu_count() or 1)
RTOL = {"f32": 1e-4, "f16": 2e-2}


@pytest.fixture(scope="module")
def P():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_16742_amd as pkg
    return pkg


def _say(*a):
    print(*a, flush=True)


def _net(P, net, params, protect=True, max_batch=None):
    return P.CtcNet(net.layers, net.in_shape, net.classes, net.dtype, params,
                    protect=protect, max_batch=max_batch or net.batch)


def _per_pass(cn, x, B, flags=None):
    """The same passes, one ctc_network_forward call each (CTC_REEXEC_NONE)."""
    n = x.shape[0]
    out = torch.empty((n, cn.out_cols), dtype=torch.float32, device=x.device)
    for k in range(0, n, B):
        cn.forward(x[k:k + B], out=out[k:k + B],
                   flags=None if flags is None else flags[k:k + B])
    return out


# (workload, images per pass, passes, max_batch, oracle rows or None)
CASES = [
    ("tiny_f32_b1", 1, 64, 1, list(range(64))),
    ("tiny_f32_b1", 4, 8, 8, list(range(32))),
    # first kernel = fused stem block staging the caller's images itself
    ("resnet20_f32_b128", 32, 3, 32, [0, 31, 32, 63, 95]),
    ("resnet18_f16_b64", 4, 2, 8, None),
]


@pytest.mark.parametrize("label,B,passes,maxb,rows", CASES)
def test_graph_replay_matches_forward(P, label, B, passes, maxb, rows):
    net = config(label)
    params = gen.make_params(net)
    cn = _net(P, net, params, max_batch=maxb)
    n = B * passes
    _say("graph", label, "B", B, "passes", passes)
    xh = gen.make_inputs(net, n)
    x = torch.from_numpy(xh).cuda()
    base = _per_pass(cn, x, B)
    S = base[:, -1].double().cpu().numpy()
    ref = float(np.median(S))
    tau = float(np.quantile(np.abs(S - ref), 0.75))
    cn.set_threshold(ref, tau)
    fl_ref = torch.zeros(n, dtype=torch.uint8, device="cuda")
    _per_pass(cn, x, B, fl_ref)
    out = torch.empty_like(base)
    fl = torch.zeros(n, dtype=torch.uint8, device="cuda")
    g = cn.graph(x, B, out=out, flags=fl)
    want_o, want_f = base.cpu().numpy(), fl_ref.cpu().numpy()
    assert 0 < want_f.sum() < n
    for rep in range(3):
        out.fill_(float("nan"))
        fl.fill_(7)
        assert g.launch() == 0
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy(), want_o), rep
        assert np.array_equal(fl.cpu().numpy(), want_f), rep
        cn.forward(x[:B])                     # eager work between replays
        torch.cuda.synchronize()
    if rows is not None:
        dp = oracle.protect_params(net, params)
        orc = oracle.forward_batch(net, dp, xh[rows], threads=THREADS)
        got = out.cpu().numpy()[rows]
        rt = RTOL[net.dtype]
        for gr, r in zip(got, orc):
            assert np.max(np.abs(gr[:-1] - r[:-1])) <= rt * np.max(np.abs(r[:-1]))
            assert abs(gr[-1] - r[-1]) <= rt * abs(r[-1])


def test_graph_sync_reexecutes_flagged_images(P):
    """tau = -1 flags every image: a re-executing launch re-runs all of them
    in max_batch-image passes (one input assembly each) and rewrites their
    rows with identical results; the threshold is the one at capture."""
    ctc = P.ctc
    net = config("tiny_f32_b1")
    params = gen.make_params(net)
    cn = _net(P, net, params, max_batch=8)
    B, passes = 4, 8
    n = B * passes
    x = torch.from_numpy(gen.make_inputs(net, n)).cuda()
    base = _per_pass(cn, x, B).cpu().numpy()
    cn.set_threshold(0.0, -1.0)
    out = torch.empty((n, cn.out_cols), device="cuda")
    fl = torch.zeros(n, dtype=torch.uint8, device="cuda")
    g = cn.graph(x, B, out=out, flags=fl)
    cn.set_threshold(0.0, float("inf"))       # not seen by the graph
    for rep in range(2):
        out.fill_(float("nan"))
        fl.zero_()
        torch.cuda.synchronize()
        ctc.ctc_net_profile(cn.h, 1)
        nf = g.launch(ctc.CTC_REEXEC_SYNC)
        launches, _ = ctc.ctc_net_profile_read(cn.h, len(net.layers))
        ctc.ctc_net_profile(cn.h, 0)
        torch.cuda.synchronize()
        assert nf == n
        assert int(launches[0]) == n // 8     # the re-run passes' assemblies
        assert fl.cpu().numpy().all()
        assert np.array_equal(out.cpu().numpy(), base)
        cn.forward(x[:B])
        torch.cuda.synchronize()
    # no flags: nothing re-run
    g2 = cn.graph(x, B, flags=fl)
    assert g2.launch(ctc.CTC_REEXEC_SYNC) == 0
    torch.cuda.synchronize()
    assert not fl.cpu().numpy().any()
    assert np.array_equal(g2.out.cpu().numpy(), base)


def test_graph_sees_parameter_faults(P):
    """A weight flip injected after capture reaches the replay (the graph
    reads the deployed parameters when it runs) and is gone after
    ctc_clear_faults."""
    net = config("tiny_f32_b1")
    params = gen.make_params(net)
    cn = _net(P, net, params, max_batch=1)
    n = 16
    x = torch.from_numpy(gen.make_inputs(net, n)).cuda()
    g = cn.graph(x, 1)
    g.launch()
    torch.cuda.synchronize()
    clean = g.out.cpu().numpy().copy()
    cn.inject([(gen.SITE_WEIGHT, 0, 5, 30, 0)])
    for rep in range(2):
        g.launch()
        torch.cuda.synchronize()
        faulty = _per_pass(cn, x, 1).cpu().numpy()
        torch.cuda.synchronize()
        got = g.out.cpu().numpy()
        assert np.array_equal(got, faulty, equal_nan=True), rep
        assert not np.array_equal(got, clean, equal_nan=True)
    cn.clear_faults()
    g.launch()
    torch.cuda.synchronize()
    assert np.array_equal(g.out.cpu().numpy(), clean)


def test_graph_rejects_bad_requests(P):
    ctc = P.ctc
    net = config("tiny_f32_b1")
    params = gen.make_params(net)
    cn = _net(P, net, params, max_batch=4)
    un = _net(P, net, params, protect=False, max_batch=4)
    x = torch.from_numpy(gen.make_inputs(net, 8)).cuda()
    out = torch.empty((8, cn.out_cols), device="cuda")

    def status(fn):
        with pytest.raises(ctc.CtcError) as e:
            fn()
        return e.value.status

    assert status(lambda: ctc.ctc_graph_create(cn.h, 0, 1, x, out)) == ctc.CTC_ERR_ARG
    assert status(lambda: ctc.ctc_graph_create(cn.h, 8, 1, x, out)) == ctc.CTC_ERR_ARG
    assert status(lambda: ctc.ctc_graph_create(cn.h, 4, 0, x, out)) == ctc.CTC_ERR_ARG
    assert status(lambda: ctc.ctc_graph_create(cn.h, 4, 2, None, out)) == ctc.CTC_ERR_ARG
    ctc.ctc_net_profile(cn.h, 1)
    assert status(lambda: ctc.ctc_graph_create(cn.h, 4, 2, x, out)) == ctc.CTC_ERR_STATE
    ctc.ctc_net_profile_read(cn.h, len(net.layers))
    ctc.ctc_net_profile(cn.h, 0)
    cn.inject([(ctc.CTC_SITE_ACT, 1, 0, 30, 0)])
    assert status(lambda: ctc.ctc_graph_create(cn.h, 4, 2, x, out)) == ctc.CTC_ERR_STATE
    cn.clear_faults()
    gu = un.graph(x, 4)
    assert status(lambda: gu.launch(ctc.CTC_REEXEC_SYNC)) == ctc.CTC_ERR_STATE
    assert status(lambda: gu.launch(ctc.CTC_REEXEC_DEFERRED)) == ctc.CTC_ERR_ARG
    assert gu.launch() == 0
    torch.cuda.synchronize()
    assert np.array_equal(gu.out.cpu().numpy(),
                          _per_pass(un, x, 4).cpu().numpy())
