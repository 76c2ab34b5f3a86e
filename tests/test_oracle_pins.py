"""Pins of the CPU oracle against facts that do not come from the oracle.

Every check here compares the oracle with something fixed independently of
it: a library routine (numpy's IEEE binary16 conversion, torch float64
convolution / pooling / linear), a closed form stated in Sec. II of the
paper (the carry-through filter yields the channel sum, the sum is
one-to-one for a 3x3/pad 1/stride 1 conv, the checksum never leaks into
normal channels, identity BN, the residual rule, the accumulated-checksum
neuron), an order-statistic definition checked by brute force, or an
exhaustively enumerated structural prediction on the tiny net.
"""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from workloads import by_name, config, gen
from workloads.nets import Net, _B

EPS = 1e-5


# ------------------------------------------------------------ binary16 (P11)

def _structured_f32_patterns():
    """Every sign, every binary32 exponent that lands near the binary16
    range, the top 10 mantissa bits exhaustively, and the 13 dropped bits at
    the rounding-critical values (0, 1, just below/at/above the half, max)."""
    sign = np.array([0, 1], np.uint32) << 31
    exp = np.arange(90, 160, dtype=np.uint32) << 23        # 2^-37 .. 2^32
    top = np.arange(1024, dtype=np.uint32) << 13
    low = np.array([0, 1, 0x0fff, 0x1000, 0x1001, 0x1fff, 0x0800, 0x17ff],
                   np.uint32)
    b = (sign[:, None, None, None] | exp[None, :, None, None]
         | top[None, None, :, None] | low[None, None, None, :]).reshape(-1)
    extra = np.array([0, 0x80000000, 0x7f800000, 0xff800000, 0x7fc00000,
                      0x7f800001, 0x00000001, 0x007fffff, 0x477fe000,
                      0x477fefff, 0x477ff000, 0x477fffff, 0x33000000,
                      0x33000001, 0x32ffffff, 0x387fc000, 0x38800000],
                     np.uint32)
    rnd = np.random.default_rng(7).integers(0, 2**32, 1 << 20,
                                            dtype=np.uint64).astype(np.uint32)
    return np.concatenate([b, extra, rnd]).view(np.float32)


def test_f16_rounding_matches_numpy_ieee_conversion():
    x = _structured_f32_patterns()
    mine = oracle.f32_to_f16_bits(x)
    with np.errstate(over="ignore", invalid="ignore"):
        ref = x.astype(np.float16).view(np.uint16)
    nan = np.isnan(x)
    assert np.array_equal(mine[~nan], ref[~nan])
    # NaN stays NaN (payload not compared)
    m = mine[nan]
    assert np.all(((m & 0x7c00) == 0x7c00) & ((m & 0x3ff) != 0))


def test_f16_widening_all_65536_patterns():
    h = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    mine = oracle.f16_bits_to_f32(h)
    ref = h.view(np.float16).astype(np.float32)
    nan = np.isnan(ref)
    assert np.array_equal(mine[~nan].view(np.uint32), ref[~nan].view(np.uint32))
    assert np.isnan(mine[nan]).all()


# ------------------------------------------- layer arithmetic vs torch f64

def _one_conv_net(c_in, c_out, k, stride, pad, groups=1, hw=9, **kw):
    b = _B()
    b.conv(0, c_in, c_out, k, stride, pad, groups=groups, bias=kw.get(
        "bias", False), bn=kw.get("bn", False), relu=kw.get("relu", False))
    return Net("t", (c_in, hw, hw), b.layers, 0, "f32", 1)


@pytest.mark.parametrize("c_in,c_out,k,stride,pad,groups", [
    (3, 8, 3, 1, 1, 1), (5, 4, 3, 2, 1, 1), (4, 6, 7, 2, 3, 1),
    (6, 4, 1, 2, 0, 1), (8, 8, 3, 1, 1, 8), (8, 8, 3, 2, 1, 8)])
def test_conv_matches_torch_float64(c_in, c_out, k, stride, pad, groups):
    rng = np.random.default_rng(1)
    x = rng.standard_normal((c_in, 11, 13)).astype(np.float32)
    w = rng.standard_normal((c_out, c_in // groups, k, k)).astype(np.float32)
    b = rng.standard_normal(c_out).astype(np.float32)
    P = (11 + 2 * pad - k) // stride + 1
    Q = (13 + 2 * pad - k) // stride + 1
    y = np.empty((c_out, P, Q), np.float32)
    oracle.lib().or_conv(x.ctypes.data, c_in, 11, 13, w.ctypes.data, c_out,
                         k, k, stride, pad, groups, b.ctypes.data, None, None,
                         None, None, EPS, None, 0, 0, y.ctypes.data)
    ref = F.conv2d(torch.from_numpy(x[None].astype(np.float64)),
                   torch.from_numpy(w.astype(np.float64)),
                   torch.from_numpy(b.astype(np.float64)), stride, pad,
                   groups=groups)[0].numpy()
    n = (c_in // groups) * k * k
    bound = 2 * n * np.finfo(np.float32).eps * F.conv2d(
        torch.from_numpy(np.abs(x[None]).astype(np.float64)),
        torch.from_numpy(np.abs(w).astype(np.float64)), None, stride, pad,
        groups=groups)[0].numpy() + 1e-7
    assert np.all(np.abs(y - ref) <= bound)
    # integer-valued operands: every partial sum is exact, so bit-exact
    xi = rng.integers(-4, 5, x.shape).astype(np.float32)
    wi = rng.integers(-3, 4, w.shape).astype(np.float32)
    oracle.lib().or_conv(xi.ctypes.data, c_in, 11, 13, wi.ctypes.data,
                         c_out, k, k, stride, pad, groups, None, None, None,
                         None, None, EPS, None, 0, 0, y.ctypes.data)
    ref = F.conv2d(torch.from_numpy(xi[None].astype(np.float64)),
                   torch.from_numpy(wi.astype(np.float64)), None, stride, pad,
                   groups=groups)[0].numpy()
    assert np.array_equal(y, ref.astype(np.float32))


def test_conv_bn_is_eq1_and_relu_residual():
    rng = np.random.default_rng(2)
    C, K = 4, 5
    x = rng.standard_normal((C, 6, 6)).astype(np.float32)
    w = rng.standard_normal((K, C, 3, 3)).astype(np.float32)
    mean, var = rng.standard_normal(K).astype(np.float32), rng.uniform(
        0.5, 2, K).astype(np.float32)
    gam, bet = rng.uniform(0.5, 1.5, K).astype(np.float32), \
        rng.standard_normal(K).astype(np.float32)
    res = rng.standard_normal((K, 6, 6)).astype(np.float32)
    y = np.empty((K, 6, 6), np.float32)
    oracle.lib().or_conv(x.ctypes.data, C, 6, 6, w.ctypes.data, K, 3, 3, 1, 1,
                         1, None, mean.ctypes.data, var.ctypes.data,
                         gam.ctypes.data, bet.ctypes.data, EPS,
                         res.ctypes.data, 1, 0, y.ctypes.data)
    c = F.conv2d(torch.from_numpy(x[None].astype(np.float64)),
                 torch.from_numpy(w.astype(np.float64)), None, 1, 1)[0].numpy()
    bn = ((c - mean[:, None, None]) / np.sqrt(var[:, None, None].astype(
        np.float64) + EPS) * gam[:, None, None] + bet[:, None, None])
    ref = np.maximum(bn + res, 0)
    assert np.allclose(y, ref, rtol=1e-5, atol=1e-5)


def test_pool_gap_fc_match_library():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((5, 9, 9)).astype(np.float32)
    for k, s, p in ((3, 2, 1), (2, 2, 0)):
        P = (9 + 2 * p - k) // s + 1
        y = np.empty((5, P, P), np.float32)
        oracle.lib().or_maxpool(x.ctypes.data, 5, 9, 9, k, s, p, 0,
                                y.ctypes.data)
        ref = F.max_pool2d(torch.from_numpy(x[None]), k, s, p)[0].numpy()
        assert np.array_equal(y, ref)
    xn = x.copy()
    xn[2, 4, 4] = np.nan
    y = np.empty((5, 4, 4), np.float32)
    oracle.lib().or_maxpool(xn.ctypes.data, 5, 9, 9, 2, 2, 0, 0, y.ctypes.data)
    ref = F.max_pool2d(torch.from_numpy(xn[None]), 2, 2, 0)[0].numpy()
    assert np.array_equal(np.isnan(y), np.isnan(ref))
    g = np.empty(5, np.float32)
    oracle.lib().or_gap(x.ctypes.data, 5, 9, 9, 0, g.ctypes.data)
    assert np.allclose(g, x.astype(np.float64).mean(axis=(1, 2)), rtol=1e-6,
                       atol=1e-7)
    W = rng.standard_normal((7, 45)).astype(np.float32)
    b = rng.standard_normal(7).astype(np.float32)
    v = rng.standard_normal(45).astype(np.float32)
    o = np.empty(7, np.float32)
    oracle.lib().or_fc(v.ctypes.data, 45, W.ctypes.data, 7, b.ctypes.data, 0,
                       0, o.ctypes.data)
    assert np.allclose(o, W.astype(np.float64) @ v + b, rtol=1e-5, atol=1e-5)


# ----------------------------------- the carry-through filter (P1, P2, P3)

def _two_conv_net(C, K1, K2, stride2=1, hw=8):
    b = _B()
    t = b.conv(0, C, K1, 3, 1, 1, bn=False, relu=False)
    b.conv(t, K1, K2, 3, stride2, 1, bn=False, relu=False)
    return Net("t", (C, hw, hw), b.layers, 0, "f32", 1)


def _int_params(net, rng):
    ps = []
    for L in net.layers:
        ps.append({"w": rng.integers(-3, 4, (L["c_out"], L["c_in"] //
                                              L["groups"], L["k"], L["k"])
                                     ).astype(np.float32)})
    return ps


@pytest.mark.parametrize("stride2", [1, 2])
def test_ct_channel_is_channel_sum_exact(stride2):
    """P1 (Sec. II-A): the carry-through output is the element-wise sum of
    the input feature maps over channels (including the incoming checksum),
    sampled at the output positions; bit-exact on integer data."""
    rng = np.random.default_rng(4)
    net = _two_conv_net(3, 6, 5, stride2)
    dp = oracle.protect_params(net, _int_params(net, rng))
    x = rng.integers(-5, 6, net.in_shape).astype(np.float32)
    T = oracle.forward_image(net, dp, x, keep=True)
    assert np.array_equal(T[1][-1], x.sum(axis=0))
    assert np.array_equal(T[2][-1], T[1].sum(axis=0)[::stride2, ::stride2])


def test_ct_sum_is_one_to_one_k3p1s1():
    """P2 (Sec. II-A): with kernel 3, padding 1, stride 1 every input
    element reaches exactly one carry-through output element."""
    rng = np.random.default_rng(5)
    net = _two_conv_net(4, 7, 3)
    dp = oracle.protect_params(net, _int_params(net, rng))
    x = rng.integers(-5, 6, net.in_shape).astype(np.float32)
    T = oracle.forward_image(net, dp, x, keep=True)
    assert T[1][-1].sum() == x.sum()
    assert T[2][-1].sum() == T[1].sum()


def test_checksum_does_not_leak_into_normal_channels():
    """P3 (Sec. II-A, input-channel level): changing the incoming checksum
    channel leaves every normal output channel bit-identical."""
    rng = np.random.default_rng(6)
    net = _two_conv_net(3, 6, 5)
    dp = oracle.protect_params(net, [
        {"w": rng.standard_normal((L["c_out"], L["c_in"], 3, 3)
                                  ).astype(np.float32)}
        for L in net.layers])
    x = rng.standard_normal(net.in_shape).astype(np.float32)
    T = oracle.forward_image(net, dp, x, keep=True)
    T2 = list(T)
    T2[1] = T[1].copy()
    T2[1][-1] += rng.standard_normal(T[1][-1].shape).astype(np.float32) * 100
    U = oracle.forward_image(net, dp, None, start=1, acts=T2, keep=True)
    assert np.array_equal(U[2][:-1].view(np.uint32), T[2][:-1].view(np.uint32))
    assert not np.array_equal(U[2][-1], T[2][-1])


# ---------------------- whole protected nets vs pruned nets in torch (P4)

def _pruned_forward_torch(net, params, x):
    """The network with every internal width reduced by one channel /
    neuron, run in float64 with torch.  Pruning the least-important channel
    and re-using its slot for the checksum (Sec. II-A) must leave the
    protected network's logits equal to this network's."""
    shp = net.shapes()
    T = [torch.from_numpy(x[None].astype(np.float64))]
    for L, p in zip(net.layers, params):
        a = T[L["inp"]]
        ck_in = L["inp"] != 0
        if L["op"] == "conv":
            K = L["c_out"] - 1
            if L["groups"] > 1:
                w = p["w"][:K]
                groups = K
            else:
                w = p["w"][:K, :(L["c_in"] - 1) if ck_in else L["c_in"]]
                groups = 1
            y = F.conv2d(a, torch.from_numpy(w.astype(np.float64)),
                         torch.from_numpy(p["b"][:K].astype(np.float64))
                         if "b" in p else None, L["stride"], L["pad"],
                         groups=groups)
            if "mean" in p:
                f = lambda v: torch.from_numpy(  # noqa: E731
                    v[:K].astype(np.float64))[None, :, None, None]
                y = (y - f(p["mean"])) / torch.sqrt(f(p["var"]) + EPS) \
                    * f(p["gamma"]) + f(p["beta"])
            if L["residual"] >= 0:
                y = y + T[L["residual"]]
            if L["relu"]:
                y = torch.relu(y)
        elif L["op"] == "maxpool":
            y = F.max_pool2d(a, L["k"], L["stride"], L["pad"])
        elif L["op"] == "gap":
            y = a.mean(dim=(2, 3), keepdim=True)
        else:
            v = a.reshape(1, -1)
            if L["flatten"] is not None:
                C, H, W = L["flatten"]
                cols = np.arange((C - 1) * H * W)
            else:
                cols = np.arange(L["in_f"] - 1)
            rows = L["out_f"] if L["final"] else L["out_f"] - 1
            W_ = p["w"][:rows][:, cols]
            y = v @ torch.from_numpy(W_.astype(np.float64)).T
            if "b" in p:
                y = y + torch.from_numpy(p["b"][:rows].astype(np.float64))
            if L["relu"]:
                y = torch.relu(y)
            y = y.reshape(1, -1, 1, 1)
        T.append(y)
    return [t[0].numpy() for t in T]


SMALL_NETS = {
    "tiny": lambda: by_name("tiny"),
    "resnet20": lambda: by_name("resnet20"),
    "resnet18": lambda: by_name("resnet18", dtype="f32", in_hw=64),
    "vgg16": lambda: by_name("vgg16", dtype="f32", in_hw=64, hidden=256,
                             classes=100),
    "mobilenetv2": lambda: by_name("mobilenetv2", dtype="f32", in_hw=64),
}


@pytest.mark.parametrize("name", list(SMALL_NETS))
def test_protected_logits_equal_pruned_network(name):
    net = SMALL_NETS[name]()
    params = gen.make_params(net)
    dp = oracle.protect_params(net, params)
    x = gen.make_inputs(net, 2)
    for xi in x:
        out = oracle.forward_image(net, dp, xi)
        ref = _pruned_forward_torch(net, params, xi)[-1].reshape(-1)
        logits = out[:-1]
        assert logits.size == net.classes and out.size == net.classes + 1
        assert np.max(np.abs(logits - ref)) <= 1e-5 * np.max(np.abs(ref))


def test_fp16_net_within_fp16_rounding_of_pruned_network():
    net = by_name("resnet18", dtype="f16", in_hw=64)
    params = gen.make_params(net)
    dp = oracle.protect_params(net, params)
    x = gen.make_inputs(net, 1)[0]
    out = oracle.forward_image(net, dp, x)
    ref = _pruned_forward_torch(net, params, x)[-1].reshape(-1)
    assert np.max(np.abs(out[:-1] - ref)) <= 2e-2 * np.max(np.abs(ref))


# -------------------------------------- BN identity, residual rule (P5, P6)

def test_bn_identity_and_residual_rule_resnet20():
    net = config("resnet20_f32_b128")
    params = gen.make_params(net)
    dp = oracle.protect_params(net, params)
    x = gen.make_inputs(net, 1)[0]
    T = oracle.forward_image(net, dp, x, keep=True)
    s = 1.0 / np.sqrt(1.0 + EPS)
    # stem: SUM role, BN identity entries of Eq. (1), ReLU
    ck1 = np.maximum(x.astype(np.float64).sum(axis=0) * s, 0)
    assert np.allclose(T[1][-1], ck1, rtol=1e-6, atol=1e-6)
    # identity block: conv1 is ZERO, conv2 sums h1, the add brings ck_in
    assert net.layers[1]["block_first"] and np.all(T[2][-1] == 0)
    ck3 = T[2][:-1].astype(np.float64).sum(axis=0) * s + T[1][-1]
    assert np.allclose(T[3][-1], ck3, rtol=1e-5)
    # projection block (stage 2): shortcut passes ck_in at stride 2
    i = next(i for i, L in enumerate(net.layers) if L["shortcut"])
    sc = T[i + 1][-1]
    xin = T[net.layers[i]["inp"]][-1]
    assert np.allclose(sc, xin[::2, ::2] * s, rtol=1e-6)
    L2 = net.layers[i + 1]
    assert L2["residual"] == i + 1
    h1 = T[L2["inp"]]
    ck = h1[:-1].astype(np.float64).sum(axis=0) * s + sc
    assert np.allclose(T[i + 2][-1], ck, rtol=1e-5)


def test_depthwise_passes_checksum_mobilenetv2():
    net = SMALL_NETS["mobilenetv2"]()
    dp = oracle.protect_params(net, gen.make_params(net))
    x = gen.make_inputs(net, 1)[0]
    T = oracle.forward_image(net, dp, x, keep=True)
    s = 1.0 / np.sqrt(1.0 + EPS)
    for i, L in enumerate(net.layers):
        if L["op"] == "conv" and L["groups"] > 1:
            st = L["stride"]
            ref = np.maximum(T[L["inp"]][-1][::st, ::st] * s, 0)
            assert np.allclose(T[i + 1][-1], ref, rtol=1e-6, atol=1e-6)


# -------------------------------------- accumulated-checksum neuron (P7)

def test_tiny_closed_form_of_S():
    """S = sum of the final features (Sec. II-B); for the tiny net the
    checksum feature unrolls to normal activations only."""
    net = config("tiny_f32_b1")
    params = gen.make_params(net)
    dp = oracle.protect_params(net, params)
    for x in gen.make_inputs(net, 3):
        S = oracle.forward_image(net, dp, x)[-1]
        P = _pruned_forward_torch(net, params, x)
        y1, y2 = P[1], P[2]                       # 15 and 31 normal channels
        ck = (y1[:, ::2, ::2].sum(axis=0)
              + np.maximum(x.astype(np.float64).sum(axis=0)[::2, ::2], 0))
        ref = y2.mean(axis=(1, 2)).sum() + ck.mean()
        assert abs(S - ref) <= 1e-5 * abs(ref)


# ------------------------------------------------------- threshold (P8)

def _tau_brute(S, alpha):
    S = np.asarray(S, np.float64)
    ref = S.sum() / S.size
    dev = np.abs(S - ref)
    ok = [d for d in dev if np.sum(dev > d) < alpha * S.size]
    return ref, min(ok)


@pytest.mark.parametrize("n,alpha", [(1, 0.01), (7, 0.3), (100, 0.01),
                                     (1000, 0.01), (1000, 0.001),
                                     (999, 0.05), (50, 0.5)])
def test_calibration_order_statistic_brute_force(n, alpha):
    S = np.random.default_rng(n).standard_normal(n) * 3 + 10
    ref, tau = oracle.calibrate(S, alpha)
    rb, tb = _tau_brute(S, alpha)
    assert abs(ref - rb) <= 1e-12 * abs(rb) and tau == tb
    assert np.sum(np.abs(S - ref) > tau) < max(alpha * n, 1)


def test_fault_free_flag_rate_is_alpha():
    """Fault-free inferences verify within tau except ~alpha of them
    (Sec. II-C); binomial 99.9% bounds on a fresh seeded set."""
    net = config("tiny_f32_b1")
    dp = oracle.protect_params(net, gen.make_params(net))
    cal = oracle.forward_batch(net, dp, gen.make_inputs(
        net, 2000, stream=gen.S_CALIB))[:, -1]
    ref, tau = oracle.calibrate(cal, 0.01)
    assert oracle.verify(cal, ref, tau).sum() <= 19
    ev = oracle.forward_batch(net, dp, gen.make_inputs(net, 2000))[:, -1]
    k = int(oracle.verify(ev, ref, tau).sum())
    assert 5 <= k <= 40


def test_verify_flags_nonfinite():
    f = oracle.verify(np.array([1.0, np.nan, np.inf, -np.inf, 1.5]), 1.0, 0.5)
    assert f.tolist() == [False, True, True, True, False]


# ---------------------------------------------- faults (P9, P10 subset)

def test_xor_involution_restores_bits():
    net = by_name("resnet18", dtype="f16", in_hw=32)
    dp = oracle.protect_params(net, gen.make_params(net))
    ref = [None if p is None else {k: v.copy() for k, v in p.items()}
           for p in dp]
    faults = gen.sample_faults(oracle.fault_sites(net, dp)[:-30], 200, 11)
    for f in faults:
        if f["site"] == gen.SITE_ACT:
            continue
        oracle.apply_param_fault(net, dp, f["site"], f["layer"], f["index"],
                                 f["bit"])
    for f in faults[::-1]:
        if f["site"] == gen.SITE_ACT:
            continue
        oracle.apply_param_fault(net, dp, f["site"], f["layer"], f["index"],
                                 f["bit"])
    for p, q in zip(dp, ref):
        if p is not None:
            for k in p:
                assert np.array_equal(p[k].view(np.uint32), q[k].view(
                    np.uint32))


def test_f16_flip_is_exact_on_every_pattern_and_bit():
    """Sec. III-A's fault is one bit of the stored representation.  For all
    65536 binary16 patterns and all 16 bits: the flipped element is the
    binary16 value whose pattern differs in exactly that bit (checked
    against numpy's binary16 decoding for non-NaN results, and NaN with the
    flipped pattern's payload otherwise), and a second flip restores the
    binary32 storage bit for bit (XOR involution, NaN payloads included)."""
    h = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    idx = np.arange(65536)
    base = h.view(np.float16).astype(np.float32)
    nan0 = np.isnan(base)
    # the stored fp32 of a NaN pattern keeps its 10-bit payload
    base.view(np.uint32)[nan0] = ((h[nan0].astype(np.uint32) & 0x8000) << 16
                                  | 0x7f800000
                                  | (h[nan0].astype(np.uint32) & 0x3ff) << 13)
    assert np.array_equal(oracle.core.f16_bits_to_f32_bits(h),
                          base.view(np.uint32))
    for bit in range(16):
        a = base.copy()
        oracle.core._flip(a, idx, bit, False)
        g = h ^ np.uint16(1 << bit)
        want = g.view(np.float16).astype(np.float32)
        fin = ~np.isnan(want)
        assert np.array_equal(a[fin].view(np.uint32),
                              want[fin].view(np.uint32)), bit
        gn = g[~fin].astype(np.uint32)
        assert np.array_equal(a[~fin].view(np.uint32),
                              (gn & 0x8000) << 16 | 0x7f800000
                              | (gn & 0x3ff) << 13), bit
        oracle.core._flip(a, idx, bit, False)
        assert np.array_equal(a.view(np.uint32), base.view(np.uint32)), bit


def test_f16_weight_fault_into_a_signalling_nan_pattern_restores():
    """Weight 1.25 (binary16 0x3d00), bit 14: the fault stores 0x7d00, a
    NaN with the quiet bit clear; applying the same fault again gives 1.25
    back (and not the quieted pattern's neighbour 1.75)."""
    net = config("tiny_f32_b1").copy(dtype="f16")
    dp = oracle.protect_params(net, gen.make_params(net))
    dp[0]["w"].reshape(-1)[5] = 1.25
    oracle.apply_param_fault(net, dp, gen.SITE_WEIGHT, 0, 5, 14)
    assert int(dp[0]["w"].reshape(-1)[5:6].view(np.uint32)[0]) == 0x7fa00000
    oracle.apply_param_fault(net, dp, gen.SITE_WEIGHT, 0, 5, 14)
    assert dp[0]["w"].reshape(-1)[5] == np.float32(1.25)
    # a fault target that holds no binary16 value is refused
    a = np.array([0.1], np.float32)
    with pytest.raises(ValueError):
        oracle.core._flip(a, 0, 3, False)


@pytest.fixture(scope="module")
def tiny_setup():
    net = config("tiny_f32_b1")
    dp = oracle.protect_params(net, gen.make_params(net))
    cal = oracle.forward_batch(net, dp, gen.make_inputs(
        net, 1000, stream=gen.S_CALIB))[:, -1]
    ref, tau = oracle.calibrate(cal, 0.01)
    x = gen.make_inputs(net, 1)[0]
    T = oracle.forward_image(net, dp, x, keep=True)
    return net, dp, x, T, ref, tau


def _run_fault(net, dp, x, T, f):
    if f["site"] == gen.SITE_ACT:
        t = int(f["layer"])
        start = max(t - 1, 0)
        acts = list(T)
        if t == 0:
            return oracle.forward_image(net, dp, x, act_faults=[
                (0, int(f["index"]), int(f["bit"]))])
        acts[t] = T[t].copy()
        oracle.core._flip(acts[t], int(f["index"]), int(f["bit"]),
                          oracle.stored_f32(net, t))
        if t == len(net.layers):
            return acts[t].reshape(-1).copy()
        return oracle.forward_image(net, dp, None, start=t, acts=acts)
    oracle.apply_param_fault(net, dp, f["site"], f["layer"], f["index"],
                             f["bit"])
    try:
        return oracle.forward_image(net, dp, x, start=int(f["layer"]),
                                    acts=T)
    finally:
        oracle.apply_param_fault(net, dp, f["site"], f["layer"],
                                 f["index"], f["bit"])


def test_tiny_structural_predictions(tiny_setup):
    """P10 on the tiny net: (i) flips of the normal logits' weights, biases
    and values never move S, so they are never detected; (ii) flips of the
    accumulated-checksum neuron's weights, bias and value never change the
    class; (iii) bit 30 of a carry-through weight (1.0 -> Inf) makes the
    next layer NaN: detected and critical; (iv) flips of the lowest
    mantissa bits stay far below tau."""
    net, dp, x, T, ref, tau = tiny_setup
    gold = T[-1].reshape(-1)
    nf = len(net.layers) - 1
    C = net.classes
    IN = dp[nf]["w"].shape[1]
    F_ = gen.FAULT_DTYPE
    # (i)
    fl = [(gen.SITE_WEIGHT, nf, o * IN + i, b) for o in range(C)
          for i in range(IN) for b in (0, 23, 30, 31)]
    fl += [(gen.SITE_BIAS, nf, o, b) for o in range(C) for b in range(32)]
    fl += [(gen.SITE_ACT, len(net.layers), o, b) for o in range(C)
           for b in range(32)]
    for s, l, i, b in fl:
        out = _run_fault(net, dp, x, T, np.array((s, l, i, b, 0), F_))
        assert out[-1] == gold[-1] and not oracle.verify(out[-1:], ref,
                                                         tau)[0]
    # (ii)
    fl = [(gen.SITE_WEIGHT, nf, C * IN + i, b) for i in range(IN)
          for b in range(32)]
    fl += [(gen.SITE_BIAS, nf, C, b) for b in range(32)]
    fl += [(gen.SITE_ACT, len(net.layers), C, b) for b in range(32)]
    for s, l, i, b in fl:
        out = _run_fault(net, dp, x, T, np.array((s, l, i, b, 0), F_))
        assert np.array_equal(out[:-1], gold[:-1])
        assert not oracle.is_critical(out[:-1], gold[:-1])
    # (iii) carry-through weights of conv1 (last filter, centre tap)
    w = dp[0]["w"]
    K, Cg, R, S = w.shape
    for c in range(Cg):
        idx = ((K - 1) * Cg + c) * R * S + (R // 2) * S + S // 2
        assert w.reshape(-1)[idx] == 1.0
        out = _run_fault(net, dp, x, T, np.array(
            (gen.SITE_WEIGHT, 0, idx, 30, 0), F_))
        assert np.isnan(out).any()
        assert oracle.verify(out[-1:], ref, tau)[0]
        assert oracle.is_critical(out[:-1], gold[:-1])
    # (iv) lowest mantissa bits of a sample of weights and activations
    sites = oracle.fault_sites(net, dp)
    fs = gen.sample_faults(sites, 300, 5)
    for f in fs:
        f["bit"] = f["bit"] % 4
        out = _run_fault(net, dp, x, T, f)
        assert abs(out[-1] - gold[-1]) < 0.01 * tau


def test_fault_sites_cover_tiny_exhaustive_count(tiny_setup):
    """The tiny net's exhaustive single-bit sweep has 1,060,544 flips per
    image: 5,451 parameters and 27,691 activation elements, 32 bits each."""
    net, dp, *_ = tiny_setup
    sites = oracle.fault_sites(net, dp)
    par = sum(s[2] for s in sites if s[0] != gen.SITE_ACT)
    act = sum(s[2] for s in sites if s[0] == gen.SITE_ACT)
    assert (par, act) == (5451, 27691)
    assert len(gen.enumerate_faults(sites)) == 1060544


# ------------------------------------------ FI-based threshold, metrics

def _tau_brute_at(S, ref, alpha):
    dev = np.abs(np.asarray(S, np.float64) - ref)
    dev = np.where(np.isnan(dev), np.inf, dev)
    ok = [d for d in dev if np.sum(dev > d) < alpha * dev.size]
    return min(ok)


@pytest.mark.parametrize("n,alpha", [(1, 0.01), (9, 0.3), (200, 0.01),
                                     (1000, 0.001), (777, 0.05)])
def test_threshold_at_ref_order_statistic_brute_force(n, alpha):
    g = np.random.default_rng(100 + n)
    S = g.standard_normal(n) * 2 + 5
    ref = 4.5
    tau = oracle.threshold_at_ref(S, ref, alpha)
    assert tau == _tau_brute_at(S, ref, alpha)
    # fewer than alpha*n of the samples deviate by more than tau
    assert np.sum(np.abs(S - ref) > tau) < max(alpha * n, 1)


def test_threshold_at_ref_at_the_mean_is_the_distribution_threshold():
    S = np.random.default_rng(5).standard_normal(3000) * 7 + 100
    ref, tau = oracle.calibrate(S, 0.01)
    assert oracle.threshold_at_ref(S, ref, 0.01) == tau


def test_threshold_at_ref_ranks_nan_last():
    S = np.array([1.0, np.nan, 2.0, np.nan, 3.0, 1.5, 0.5, 2.5, 1.2, 1.1])
    # k = 10 - 1 + 1 = 10 at alpha 0.1: the largest deviation, a NaN -> inf
    assert oracle.threshold_at_ref(S, 1.0, 0.1) == np.inf
    # alpha 0.3: k = 8 -> 8th smallest of {0, inf, 1, inf, 2, .5, .5, 1.5,
    # .2, .1} = 2.0
    assert oracle.threshold_at_ref(S, 1.0, 0.3) == 2.0


def test_detection_rates_by_hand():
    flags = [1, 0, 1, 1, 0, 0, 1, 0]
    crit = [1, 1, 1, 0, 0, 0, 0, 0]
    tpr, fpr, j = oracle.detection_rates(flags, crit)
    assert tpr == 2 / 3 and fpr == 2 / 5 and j == tpr - fpr


def test_leveugle_sample_size():
    # large population -> 9604 (95% confidence, 1% margin, p = 0.5)
    assert gen.leveugle_sample_size(10 ** 12) == 9604
    # N = 10000: 10000 / (1 + 9999/9604) = 4899.2 -> 4900
    assert gen.leveugle_sample_size(10000) == 4900
    assert gen.leveugle_sample_size(1) == 1


# ------------------------------- L1-norm channel selection (Sec. II-A)

def test_l1_selection_preserves_the_unprotected_function():
    """Swapping a channel everywhere in its group is a relabelling: the
    unprotected network computes the same logits (up to fp32 summation
    order)."""
    for label in ("tiny_f32_b1", "resnet20_f32_b128"):
        net = config(label)
        p = gen.make_params(net)
        q, chosen = oracle.select_channels_l1(net, p)
        assert any(c >= 0 and c != L.get("c_out", -1) - 1
                   for c, L in zip(chosen, net.layers))
        x = gen.make_inputs(net, 2)
        for xi in x:
            a = oracle.forward_image(net, oracle.protect_params(
                net, p, protect=False), xi, protect=False)
            b = oracle.forward_image(net, oracle.protect_params(
                net, q, protect=False), xi, protect=False)
            assert np.allclose(a, b, rtol=1e-5, atol=1e-5 * np.abs(a).max())


def test_l1_selection_picks_the_brute_force_argmin():
    net = config("tiny_f32_b1")          # conv 3->16, conv 16->32 s2, gap, fc
    p = gen.make_params(net)
    _, chosen = oracle.select_channels_l1(net, p)
    w1, w2, wf = p[0]["w"], p[1]["w"], p[3]["w"]
    imp1 = [sum(abs(float(v)) for v in w1[c].ravel()) +
            sum(abs(float(v)) for v in w2[:, c].ravel()) for c in range(16)]
    assert chosen[0] == int(np.argmin(imp1))
    # conv2's channels are tied to the GAP output: the FC columns count too
    imp2 = [sum(abs(float(v)) for v in w2[c].ravel()) +
            sum(abs(float(v)) for v in wf[:, c]) for c in range(32)]
    assert chosen[1] == chosen[2] == int(np.argmin(imp2))
    assert chosen[3] == -1               # the classifier is not pruned


def test_l1_selection_one_channel_per_residual_stream():
    net = config("resnet20_f32_b128")
    _, chosen = oracle.select_channels_l1(net, gen.make_params(net))
    grp = oracle.channel_groups(net)
    by_group = {}
    for i, c in enumerate(chosen):
        by_group.setdefault(grp[i + 1], set()).add(c)
    assert all(len(v) == 1 for v in by_group.values())
    # the three residual streams: stem output + 3 block outputs; the stage-2
    # projection output + 3 block outputs; the stage-3 projection output +
    # 3 block outputs + the GAP output tied to them
    sizes = sorted(sum(1 for g in grp if g == r) for r in set(grp))
    assert sizes[-3:] == [4, 4, 5] and sizes[:-3] == [1] * (len(sizes) - 3)


def test_l1_selection_prunes_exactly_the_chosen_filter():
    """After the swap and the construction, the normal filters of a layer
    are the original ones minus the chosen channel (Sec. II-A: prune the
    least important filter, append the carry-through filter)."""
    net = config("tiny_f32_b1")
    p = gen.make_params(net)
    q, chosen = oracle.select_channels_l1(net, p)
    dp = oracle.protect_params(net, q)
    w_orig = p[0]["w"]
    kept = dp[0]["w"][:-1]
    want = np.delete(w_orig, chosen[0], axis=0)
    got = sorted(map(bytes, kept.reshape(15, -1)))
    assert got == sorted(map(bytes, want.reshape(15, -1)))


# ------------------------------------------- append mode (extra channels)

def test_append_mode_keeps_the_unprotected_logits_exactly():
    """Append mode prunes nothing: the protected network's logits are the
    unmodified network's, bit for bit in the oracle's fixed-order fp32
    arithmetic (the added channels only add exact zeros)."""
    for label in ("tiny_f32_b1", "resnet20_f32_b128"):
        net = config(label)
        p = gen.make_params(net)
        wn, wp = oracle.append_network(net, p)
        dp = oracle.protect_params(wn, wp)
        for xi in gen.make_inputs(net, 2):
            a = oracle.forward_image(net, oracle.protect_params(
                net, p, protect=False), xi, protect=False)
            b = oracle.forward_image(wn, dp, xi)
            assert np.array_equal(a.view(np.uint32), b[:-1].view(np.uint32))


def test_append_mode_carries_the_channel_sum():
    """P1 in append mode on the tiny net: the carry-through channel of the
    second conv is relu(s_id * (sum of every input channel at the centre
    tap)), s_id = 1/sqrt(1 + eps) (identity BN), and S is the sum of all
    GAP features (normal ones and the carried checksum)."""
    net = config("tiny_f32_b1")
    p = gen.make_params(net)
    wn, wp = oracle.append_network(net, p)
    dp = oracle.protect_params(wn, wp)
    x = gen.make_inputs(net, 1)[0]
    T = oracle.forward_image(wn, dp, x, keep=True)
    y1, y2 = T[1].astype(np.float64), T[2].astype(np.float64)
    s_id = 1.0 / np.sqrt(1.0 + 1e-5)
    ck = np.maximum(0.0, s_id * y1[:, ::2, ::2].sum(axis=0))
    assert np.allclose(y2[-1], ck, rtol=1e-5, atol=1e-4)
    gap = T[3].astype(np.float64).reshape(-1)
    S = T[-1].reshape(-1)[-1]
    assert abs(S - gap.sum()) <= 1e-5 * abs(gap).sum()
    # the padding channels between the normal ones and the checksum are 0
    assert wn.layers[0]["c_out"] == 20 and not T[1][16:19].any()
