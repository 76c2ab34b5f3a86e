"""Edge cases of the device path: empty, single-image and ragged batches,
the largest batch, batches that vary from call to call under deferred
re-execution, and arguments the library must reject without touching
state."""

import numpy as np
import pytest

import oracle
from workloads import config, gen

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module")
def P():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_16742_amd as P
    return P


@pytest.fixture(scope="module")
def r20(P):
    net = config("resnet20_f32_b128")
    params = gen.make_params(net)
    cn = P.CtcNet(net.layers, net.in_shape, net.classes, net.dtype, params,
                  protect=True, max_batch=128)
    x = gen.make_inputs(net, 128)
    return net, params, cn, x


def test_batch_sizes_agree_with_full_batch(P, r20):
    """Every row's output is independent of the batch it runs in (0, 1, 7,
    63, 128 images): bit-identical to the same image in a full batch."""
    net, params, cn, x = r20
    xd = torch.from_numpy(x).cuda()
    full = cn.forward(xd).cpu().numpy()
    out = torch.empty((1, net.classes + 1), device="cuda")
    P.ctc.ctc_network_forward(cn.h, 0, xd, out, None, P.ctc.CTC_REEXEC_NONE)
    for n in (1, 7, 63, 128):
        _say("batch", n)
        o = cn.forward(xd[-n:].contiguous()).cpu().numpy()
        assert np.array_equal(o.view(np.uint32), full[-n:].view(np.uint32)), n


def test_batch_above_max_is_rejected(P, r20):
    net, params, cn, x = r20
    big = torch.zeros((129,) + net.in_shape, device="cuda")
    with pytest.raises(P.ctc.CtcError):
        cn.forward(big)
    # the net still works afterwards
    xd = torch.from_numpy(x[:4]).cuda()
    o = cn.forward(xd).cpu().numpy()
    ref = oracle.forward_batch(net, oracle.protect_params(net, params), x[:1])
    assert abs(o[0, -1] - ref[0, -1]) <= 1e-4 * abs(ref[0, -1])


def test_deferred_calls_of_varying_size(P, r20):
    """Deferred re-execution with call sizes 1, 128, 5, 64, 0, 37 and a
    final flush: every output row equals the single-pass result (no faults,
    so re-executed rows are recomputed identically), every flag equals
    the fp32 decision on S."""
    net, params, cn, x = r20
    xd = torch.from_numpy(x).cuda()
    full = cn.forward(xd).cpu().numpy()
    S = full[:, -1].astype(np.float64)
    ref = float(np.mean(S))
    tau = float(np.quantile(np.abs(S - ref), 0.9))
    cn.set_threshold(ref, tau)
    sizes = [1, 128, 5, 64, 0, 37]
    outs, flags = [], []
    for k, n in enumerate(sizes):
        idx = (np.arange(n) * 7 + k * 13) % 128
        o = torch.full((max(n, 1), net.classes + 1), float("nan"), device="cuda")
        f = torch.full((max(n, 1),), 255, dtype=torch.uint8, device="cuda")
        xi = xd[torch.from_numpy(idx).cuda()].contiguous() if n else xd[:1]
        P.ctc.ctc_network_forward(cn.h, n, xi, o, f, P.ctc.CTC_REEXEC_DEFERRED)
        outs.append((idx, o))
        flags.append(f)
    cn.flush()
    torch.cuda.synchronize()
    for (idx, o), f in zip(outs, flags):
        if len(idx) == 0:
            continue
        got = o.cpu().numpy()
        assert np.array_equal(got.view(np.uint32), full[idx].view(np.uint32))
        assert np.array_equal(f.cpu().numpy()[:len(idx)].astype(bool),
                              oracle.verify(full[idx, -1], ref, tau))


def test_bad_faults_are_rejected_without_effect(P, r20):
    net, params, cn, x = r20
    xd = torch.from_numpy(x[:8]).cuda()
    before = cn.forward(xd).cpu().numpy()
    bad = [
        (gen.SITE_WEIGHT, 0, 10 ** 9, 0, 0),          # index past the layer
        (gen.SITE_WEIGHT, 0, 0, 32, 0),               # bit past fp32
        (gen.SITE_BIAS, 0, 0, 0, 0),                  # the stem has no bias
        (gen.SITE_ACT, 99, 0, 0, 0),                  # no such tensor
        (gen.SITE_ACT, 1, 0, 0, 128),                 # row past max_batch
    ]
    for f in bad:
        with pytest.raises(P.ctc.CtcError):
            cn.inject([f])
    # a good fault then a bad one in the same call: nothing applied
    with pytest.raises(P.ctc.CtcError):
        cn.inject([(gen.SITE_WEIGHT, 0, 0, 30, 0), bad[0]])
    after = cn.forward(xd).cpu().numpy()
    assert np.array_equal(before.view(np.uint32), after.view(np.uint32))


def test_conv2d_forward_empty_batch_is_a_no_op(P):
    ctc = P.ctc
    d = ctc.layer_desc(16, 16, 3, 3, 1, 1, 1, 0, 0)
    x = torch.zeros((1, 8, 8, 16), device="cuda")
    w = torch.zeros((16, 3, 3, 16), device="cuda")
    sc = torch.ones(16, device="cuda")
    sh = torch.zeros(16, device="cuda")
    y = torch.full((1, 8, 8, 16), 7.0, device="cuda")
    ctc.ctc_conv2d_forward(d, ctc.CTC_F32, 0, 8, 8, x, w, sc, sh, None, 1, y)
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())


def test_verify_extremes(P):
    """ctc_verify at batch 1 and at its 4096 maximum; beyond is rejected."""
    ctc = P.ctc
    for n in (1, 4096):
        S = torch.linspace(-2, 2, n, device="cuda")
        fl = torch.zeros(n, dtype=torch.uint8, device="cuda")
        cnt = torch.zeros(1, dtype=torch.int32, device="cuda")
        idx = torch.full((n,), -1, dtype=torch.int32, device="cuda")
        ctc.ctc_verify(S, n, 1, 0.0, 1.0, fl, cnt, idx)
        torch.cuda.synchronize()
        want = ~(np.abs(S.cpu().numpy()) <= 1.0)
        assert np.array_equal(fl.cpu().numpy().astype(bool), want)
        k = int(cnt.item())
        assert k == int(want.sum())
        assert sorted(idx.cpu().numpy()[:k].tolist()) == \
            np.nonzero(want)[0].tolist()
    S = torch.zeros(4097, device="cuda")
    with pytest.raises(ctc.CtcError):
        ctc.ctc_verify(S, 4097, 1, 0.0, 1.0, None,
                       torch.zeros(1, dtype=torch.int32, device="cuda"), None)
