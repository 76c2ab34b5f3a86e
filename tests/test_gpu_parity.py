"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Kernel level: every conv shape class (ragged pixel / channel / reduction
tails, strides, 1x1, 7x7 stem, depthwise, residual epilogue) in fp32 and
fp16, bit-exact on integer data (every partial sum exact, so summation
order cannot matter) and within tolerance on random data.  Network level:
logits and the accumulated checksum S of every workload at its full batch
size (sampled rows for the 224x224 nets), detection flags, re-execution,
and flags / critical labels under seeded single-bit faults.

Tolerances: 1e-4 (fp32) and 2e-2 (fp16) relative to the largest logit of
an image, and relative to |S| for S.
"""

import os

import numpy as np
import pytest

import oracle
from workloads import by_name, config, gen

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

RTOL = {"f32": 1e-4, "f16": 2e-2}
THREADS = min(16, os.cpu_count() or 1)


@pytest.fixture(scope="module")
def P():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_16742_amd as pkg
    return pkg


def _say(*a):
    print(*a, flush=True)


# --------------------------------------------------------------- kernels

def _pack_krsc(w, cs):
    K, C, R, S = w.shape
    out = np.zeros((K, R, S, cs), np.float32)
    out[..., :C] = w.transpose(0, 2, 3, 1)
    return out


def _oracle_conv(x, w, stride, pad, groups):
    """Raw convolution sums, one image at a time (NCHW)."""
    n, C, H, W = x.shape
    K, Cg, R, S = w.shape
    P_ = (H + 2 * pad - R) // stride + 1
    Q_ = (W + 2 * pad - S) // stride + 1
    y = np.empty((n, K, P_, Q_), np.float32)
    for i in range(n):
        xi = np.ascontiguousarray(x[i])
        oracle.lib().or_conv(xi.ctypes.data, C, H, W, w.ctypes.data, K, R, S,
                             stride, pad, groups, None, None, None, None,
                             None, 1e-5, None, 0, 0, y[i].ctypes.data)
    return y


CONV_CASES = [
    # n, C, H, W, K, k, stride, pad, groups, residual
    (2, 16, 9, 9, 16, 3, 1, 1, 1, False),
    (3, 32, 11, 13, 48, 3, 2, 1, 1, False),
    (2, 4, 15, 15, 64, 7, 2, 3, 1, False),
    # fp16 stem kernel (4 stored input channels): 3x3 stride 1 and 2 with
    # ragged 16x16 output tiles, 64, 32 and 8 channels, 7x7 stride 2 above
    # (a partly filled tile) and on a 40x40 input (several tiles)
    (2, 4, 20, 35, 64, 3, 1, 1, 1, False),
    (3, 4, 17, 33, 32, 3, 1, 1, 1, False),
    (1, 4, 9, 9, 8, 3, 1, 1, 1, False),
    (3, 4, 37, 29, 32, 3, 2, 1, 1, False),
    (2, 4, 40, 40, 64, 7, 2, 3, 1, False),
    (3, 4, 29, 37, 32, 7, 2, 3, 1, False),
    (2, 64, 7, 7, 128, 1, 1, 0, 1, True),
    (2, 96, 8, 8, 96, 1, 2, 0, 1, False),
    (1, 8, 10, 10, 24, 3, 1, 1, 1, True),
    (2, 200, 5, 6, 136, 3, 1, 1, 1, False),
    (2, 32, 9, 9, 32, 3, 1, 1, 32, False),
    (2, 48, 9, 8, 48, 3, 2, 1, 48, False),
    # fp16 whole-image kernel on 7x7 and 14x14 maps (one and several
    # 64-channel planes, residual), fp32 the implicit GEMM
    (3, 64, 7, 7, 64, 3, 1, 1, 1, True),
    (2, 192, 7, 7, 128, 3, 1, 1, 1, False),
    (2, 128, 14, 14, 128, 3, 1, 1, 1, True),
    (3, 64, 14, 14, 192, 3, 1, 1, 1, False),
    # ... and with stride 2 from 14x14 to 7x7
    (3, 64, 14, 14, 64, 3, 2, 1, 1, False),
    (2, 192, 14, 14, 128, 3, 2, 1, 1, True),
    # fp16 64-half K steps: several M and N tiles with tails, K tails
    (2, 64, 14, 14, 256, 3, 1, 1, 1, True),
    (3, 128, 9, 7, 200, 3, 2, 1, 1, False),
    (4, 16, 112, 112, 128, 1, 1, 0, 1, True),
    # fp16 256x256 tiles (8 waves, epilogue in two row passes)
    (32, 72, 32, 32, 256, 1, 1, 0, 1, True),
    (33, 8, 32, 31, 256, 3, 1, 1, 1, False),
    # fp16 pointwise kernel (1x1, <= 64 input channels): pixel tails past
    # the last wave's tiles, channel tiles with 4 of 16 channels, two
    # 32-channel k steps with a half-empty second one, 8 input channels
    (32, 32, 32, 32, 256, 1, 1, 0, 1, True),
    (3, 24, 13, 11, 36, 1, 1, 0, 1, False),
    (2, 40, 9, 10, 4, 1, 1, 0, 1, True),
    (5, 8, 7, 9, 20, 1, 1, 0, 1, False),
    # ... with 96 to 160 input channels (three to five k steps) and output
    # channel groups (128 channels per workgroup past 192; group tails of
    # 64, 72 and, for 8-byte row pieces, 36 channels)
    (2, 96, 14, 14, 576, 1, 1, 0, 1, False),
    (3, 160, 7, 7, 200, 1, 1, 0, 1, True),
    (2, 144, 9, 9, 24, 1, 1, 0, 1, False),
    (2, 120, 5, 5, 36, 1, 1, 0, 1, True),
    # spatial-tile kernel (fp32, 16..64 input channels): ResNet-20 shapes,
    # ragged tiles, stride 2, 1x1 stride 2, channel tails
    (3, 16, 32, 32, 16, 3, 1, 1, 1, True),
    (2, 16, 32, 32, 32, 3, 2, 1, 1, False),
    (2, 32, 16, 16, 64, 1, 2, 0, 1, False),
    (4, 64, 8, 8, 64, 3, 1, 1, 1, True),
    (2, 48, 13, 11, 20, 3, 1, 1, 1, False),
    (1, 64, 5, 37, 8, 3, 2, 1, 1, True),
]


@pytest.mark.parametrize("dtype", ["f32", "f16"])
@pytest.mark.parametrize("case", CONV_CASES)
@pytest.mark.parametrize("integer", [True, False])
def test_conv2d_forward_parity(P, dtype, case, integer):
    ctc = P.ctc
    n, C, H, W, K, k, st, pad, g, res = case
    _say("conv case", dtype, case, "integer" if integer else "random")
    rng = np.random.default_rng(CONV_CASES.index(case) * 4 + 2 * (
        dtype == "f16") + int(integer))
    Cg = C // g
    if integer:
        x = rng.integers(-3, 4, (n, C, H, W)).astype(np.float32)
        w = rng.integers(-2, 3, (K, Cg, k, k)).astype(np.float32)
        scale = np.ones(K, np.float32)
        shift = rng.integers(-4, 5, K).astype(np.float32)
    else:
        x = rng.standard_normal((n, C, H, W)).astype(np.float32)
        w = (rng.standard_normal((K, Cg, k, k)) /
             np.sqrt(Cg * k * k)).astype(np.float32)
        scale = rng.uniform(0.5, 1.5, K).astype(np.float32)
        shift = rng.standard_normal(K).astype(np.float32)
    if dtype == "f16":
        x, w = oracle.round_f16(x), oracle.round_f16(w)
    Pq = (H + 2 * pad - k) // st + 1
    Qq = (W + 2 * pad - k) // st + 1
    r = None
    if res:
        r = rng.integers(-3, 4, (n, K, Pq, Qq)).astype(np.float32)
        if dtype == "f16":
            r = oracle.round_f16(r)
    acc = _oracle_conv(x, w, st, pad, g).astype(np.float64)
    ref = acc * scale[None, :, None, None] + shift[None, :, None, None]
    if res:
        ref = ref + r
    ref = np.maximum(ref, 0)
    tdt = torch.float16 if dtype == "f16" else torch.float32
    dev = "cuda"
    xd = torch.from_numpy(x.transpose(0, 2, 3, 1).copy()).to(dev, tdt)
    if g == 1:
        wp = _pack_krsc(w, C)
    else:
        wp = w[:, 0].transpose(1, 2, 0).copy()        # [R][S][C]
    wd = torch.from_numpy(wp).to(dev, tdt).contiguous()
    sd = torch.from_numpy(scale).to(dev)
    hd = torch.from_numpy(shift).to(dev)
    rd = None if r is None else torch.from_numpy(
        r.transpose(0, 2, 3, 1).copy()).to(dev, tdt)
    yd = torch.full((n, Pq, Qq, K), float("nan"), dtype=tdt, device=dev)
    d = ctc.layer_desc(C, K, k, k, st, pad, g, 0, ctc.CTC_ROLE_NONE)
    ctc.ctc_conv2d_forward(d, ctc.DTYPES[dtype], n, H, W, xd, wd, sd, hd, rd,
                           1, yd)
    torch.cuda.synchronize()
    y = yd.float().cpu().numpy().transpose(0, 3, 1, 2)
    if integer:
        want = ref.astype(np.float32)
        if dtype == "f16":
            want = oracle.round_f16(want)
        assert np.array_equal(y, want)
    else:
        tol = 1e-5 if dtype == "f32" else 4e-3
        assert np.max(np.abs(y - ref)) <= tol * np.max(np.abs(ref))


def _host_maxpool2(y):
    """2x2 stride-2 max pool of NCHW values (floor of odd sizes), NaN if any
    window value is NaN: the definition the fused pools must reproduce on
    the stored values."""
    n, c, h, w = y.shape
    v = y[:, :, :h // 2 * 2, :w // 2 * 2].reshape(n, c, h // 2, 2, w // 2, 2)
    v = v.transpose(0, 1, 2, 4, 3, 5).reshape(n, c, h // 2, w // 2, 4)
    out = v.max(axis=-1)
    out[np.isnan(v).any(axis=-1)] = np.nan
    return out


# n, C, H, W, K, pool, images the oracle recomputes, kernel expected
PP_CASES = [
    # 224-pixel tiles, 256-channel tiles: raster tiles with a ragged tail
    (15, 64, 55, 53, 256, 0, [0, 7, 14], "conv_pp<256, 224, 0, false>"),
    # the pool in conv_pp's epilogue (28 x 8 tiles, 2 of 56 columns empty)
    (15, 64, 56, 54, 256, 2, [0, 14], "conv_pp<256, 224, 8, true>"),
    # ... on 28 x 28 maps: 28 x 8 and 14 x 16 tiles tie, the 8-wide one
    (64, 64, 28, 28, 512, 2, [0, 63], "conv_pp<256, 224, 8, true>"),
    # ... 14 x 16 tiles where they are fewer (42 x 16 maps: 3 against 4)
    (32, 64, 42, 16, 512, 2, [0, 31], "conv_pp<256, 224, 16, true>"),
    # the pool in conv_dma's epilogue (8 x 16 tiles), 64 and 128 channels
    (4, 32, 96, 112, 64, 2, [1, 3],
     "conv_dma<_Float16, 128, 64, 2, 2, 2, true, 16, true, 0>"),
    (8, 64, 64, 96, 128, 2, [5],
     "conv_dma<_Float16, 128, 128, 2, 2, 2, true, 16, true, 0>"),
    # conv_dma with the halo tile (64 input channels): ragged 8 x 16 tiles
    # (60 x 60 maps), with and without the pool, 64, 40 and 128 channels
    (9, 64, 60, 60, 64, 2, [0, 8],
     "conv_dma<_Float16, 128, 64, 2, 2, 2, true, 16, true, 1>"),
    (8, 64, 60, 60, 40, 0, [0, 7],
     "conv_dma<_Float16, 128, 64, 2, 2, 2, true, 16, false, 1>"),
    (8, 64, 60, 60, 128, 0, [3],
     "conv_dma<_Float16, 128, 128, 2, 2, 2, true, 16, false, 1>"),
    # whole-image kernel at ResNet-18's 14x14 stage size
    (64, 256, 14, 14, 256, 0, [0, 37, 63], "conv_img<14, false, 1>"),
]


@pytest.mark.parametrize("case", PP_CASES)
def test_conv2d_forward_large_tiles_and_fused_pool(P, case):
    """Shapes that take the 224-pixel ping-pong kernel or a pooled epilogue
    (integer data: every sum exact, so any summation order gives the same
    bits).  Unpooled output: equal to the oracle's convolution on the
    sampled images.  Pooled output: bit-identical to the library's own
    unpooled output max-pooled on the host, on every image."""
    ctc = P.ctc
    n, C, H, W, K, pool, sample, kname = case
    _say("conv large tiles / pool", case)
    rng = np.random.default_rng(sum(case[:6]))
    x = rng.integers(-3, 4, (n, C, H, W)).astype(np.float32)
    w = rng.integers(-2, 3, (K, C, 3, 3)).astype(np.float32)
    shift = rng.integers(-4, 5, K).astype(np.float32)
    scale = np.ones(K, np.float32)
    d = ctc.layer_desc(C, K, 3, 3, 1, 1, 1, 0, ctc.CTC_ROLE_NONE)
    assert ctc.ctc_conv2d_workspace_bytes(d, ctc.CTC_F16, n, H, W, pool) == 0
    assert ctc.ctc_conv2d_kernel_name(d, ctc.CTC_F16, n, H, W, pool) == kname
    dev = "cuda"
    xd = torch.from_numpy(x.transpose(0, 2, 3, 1).copy()).to(dev, torch.float16)
    wd = torch.from_numpy(_pack_krsc(w, C)).to(dev, torch.float16).contiguous()
    sd = torch.from_numpy(scale).to(dev)
    hd = torch.from_numpy(shift).to(dev)
    y = torch.full((n, H, W, K), float("nan"), dtype=torch.float16, device=dev)
    ctc.ctc_conv2d_forward(d, ctc.CTC_F16, n, H, W, xd, wd, sd, hd, None, 1, y)
    if pool:
        yp = torch.full((n, H // 2, W // 2, K), float("nan"), dtype=torch.float16,
                        device=dev)
        ctc.ctc_conv2d_forward(d, ctc.CTC_F16, n, H, W, xd, wd, sd, hd, None, 1,
                               yp, pool=2)
    torch.cuda.synchronize()
    full = y.float().cpu().numpy().transpose(0, 3, 1, 2)
    acc = _oracle_conv(x[sample], w, 1, 1, 1).astype(np.float64)
    want = oracle.round_f16(np.maximum(acc + shift[None, :, None, None], 0)
                            .astype(np.float32))
    assert np.array_equal(full[sample], want)
    if pool:
        got = yp.cpu().numpy().view(np.uint16).transpose(0, 3, 1, 2)
        ref = _host_maxpool2(full).astype(np.float16).view(np.uint16)
        assert np.array_equal(got, ref)


def test_conv2d_forward_pool_rejected_without_kernel(P):
    """A pool request for a conv whose kernel has no pooled epilogue (fp32)
    is refused before anything runs."""
    ctc = P.ctc
    d = ctc.layer_desc(16, 16, 3, 3, 1, 1, 1, 0, ctc.CTC_ROLE_NONE)
    x = torch.zeros(1, 8, 8, 16, device="cuda")
    with pytest.raises(ctc.CtcError) as e:
        ctc.ctc_conv2d_forward(d, ctc.CTC_F32, 1, 8, 8, x, x, x[0, 0, 0],
                               x[0, 0, 0], None, 1, x, pool=2)
    assert e.value.status == ctc.CTC_ERR_UNSUPPORTED


def test_conv2d_forward_split_k_workspace(P):
    """A deep layer on an 8x8 map (K = 4608, 64 pixels per image): with the
    workspace ctc_conv2d_workspace_bytes asks for, K is split over four
    workgroup ranges; the result equals the oracle's (integer data) and the
    unsplit call's."""
    ctc = P.ctc
    n, C, H, K = 3, 512, 8, 64
    rng = np.random.default_rng(11)
    x = rng.integers(-2, 3, (n, C, H, H)).astype(np.float32)
    w = rng.integers(-1, 2, (K, C, 3, 3)).astype(np.float32)
    shift = rng.integers(-4, 5, K).astype(np.float32)
    d = ctc.layer_desc(C, K, 3, 3, 1, 1, 1, 0, ctc.CTC_ROLE_NONE)
    for dt, tdt in (("f16", torch.float16), ("f32", torch.float32)):
        nb = ctc.ctc_conv2d_workspace_bytes(d, ctc.DTYPES[dt], n, H, H)
        assert nb == 4 * n * H * H * K * 4, nb
        xd = torch.from_numpy(x.transpose(0, 2, 3, 1).copy()).to("cuda", tdt)
        wd = torch.from_numpy(_pack_krsc(w, C)).to("cuda", tdt).contiguous()
        sd = torch.ones(K, device="cuda")
        hd = torch.from_numpy(shift).cuda()
        ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
        ys = torch.full((n, H, H, K), float("nan"), dtype=tdt, device="cuda")
        yu = torch.full_like(ys, float("nan"))
        ctc.ctc_conv2d_forward(d, ctc.DTYPES[dt], n, H, H, xd, wd, sd, hd, None,
                               1, ys, workspace=ws, ws_bytes=nb)
        ctc.ctc_conv2d_forward(d, ctc.DTYPES[dt], n, H, H, xd, wd, sd, hd, None,
                               1, yu)
        torch.cuda.synchronize()
        acc = _oracle_conv(x, w, 1, 1, 1).astype(np.float64)
        want = np.maximum(acc + shift[None, :, None, None], 0).astype(np.float32)
        if dt == "f16":
            want = oracle.round_f16(want)
        got = ys.float().cpu().numpy().transpose(0, 3, 1, 2)
        assert np.array_equal(got, want)
        assert np.array_equal(yu.float().cpu().numpy().transpose(0, 3, 1, 2), want)


def test_conv2d_forward_rejects_bad_args(P):
    ctc = P.ctc
    d = ctc.layer_desc(6, 8, 3, 3, 1, 1, 1, 0, ctc.CTC_ROLE_NONE)
    x = torch.zeros(1, 4, 4, 6, device="cuda")
    with pytest.raises(ctc.CtcError) as e:
        ctc.ctc_conv2d_forward(d, ctc.CTC_F32, 1, 4, 4, x, x, x, x, None, 1, x)
    assert e.value.status == ctc.CTC_ERR_UNSUPPORTED


# -------------------------------------------------------------- detector

def test_verify_kernel_flags_and_indices(P):
    ctc = P.ctc
    rng = np.random.default_rng(3)
    for B in (1, 7, 64, 1000, 3000):
        _say("verify batch", B)
        S = rng.standard_normal(B).astype(np.float32) * 3
        S[rng.integers(0, B, max(1, B // 50))] = np.nan
        if B > 2:
            S[1], S[2] = np.inf, -np.inf
        Sd = torch.from_numpy(S).cuda()
        fl = torch.zeros(B, dtype=torch.uint8, device="cuda")
        cnt = torch.zeros(1, dtype=torch.int32, device="cuda")
        idx = torch.full((B,), -1, dtype=torch.int32, device="cuda")
        ctc.ctc_verify(Sd, B, 1, 0.25, 2.5, fl, cnt, idx)
        torch.cuda.synchronize()
        want = oracle.verify(S, 0.25, 2.5)
        assert np.array_equal(fl.cpu().numpy().astype(bool), want)
        n = int(cnt.item())
        assert n == want.sum()
        assert np.array_equal(idx.cpu().numpy()[:n], np.nonzero(want)[0])


# --------------------------------------------------------------- networks

def _net(P, net, params, protect=True, max_batch=None):
    return P.CtcNet(net.layers, net.in_shape, net.classes, net.dtype, params,
                    protect=protect, max_batch=max_batch or net.batch)


def _oracle_rows(net, dp, x, rows):
    return oracle.forward_batch(net, dp, x[rows], threads=THREADS)


def _check_outputs(gpu, ref, dtype):
    rt = RTOL[dtype]
    el = es = 0.0
    for g, r in zip(gpu, ref):
        lg, lr = g[:-1], r[:-1]
        assert np.max(np.abs(lg - lr)) <= rt * np.max(np.abs(lr)), \
            (np.max(np.abs(lg - lr)), np.max(np.abs(lr)))
        assert abs(g[-1] - r[-1]) <= rt * abs(r[-1]), (g[-1], r[-1])
        el = max(el, np.max(np.abs(lg - lr)) / np.max(np.abs(lr)))
        es = max(es, abs(g[-1] - r[-1]) / abs(r[-1]))
    _say("  rows", len(gpu), "max rel err: logits %.3g, S %.3g" % (el, es))


# sampled rows of the 224x224 nets: the batch's first and last image always
NET_CASES = [
    ("tiny_f32_b1", None),
    ("resnet20_f32_b128", None),
    ("resnet18_f16_b64", [0, 17, 40, 63]),
    ("resnet18_f32_b64", [0, 33, 63]),
    ("mobilenetv2_f16_b128", [0, 5, 64, 100, 127]),
    ("vgg16_f16_b32", [0, 13, 31]),
]


def test_mobilenetv2_expand_convs_take_the_pointwise_kernel(P):
    """The 1x1 convs of MobileNetV2 with at most 64 input channels, or up
    to 160 and at most 192 output channels, run on conv_pw; the others on
    the implicit GEMM."""
    net = config("mobilenetv2_f16_b128")
    cn = _net(P, net, gen.make_params(net))
    cn.set_fusion(P.ctc.CTC_FUSE_BLOCK | P.ctc.CTC_FUSE_STEM | P.ctc.CTC_FUSE_POOL)
    names = [P.ctc.ctc_net_op_kernel(cn.h, i, net.batch)
             for i in range(len(net.layers))]
    def pointwise(L):
        return L["op"] == "conv" and L["k"] == 1 and L["stride"] == 1 and \
            L["groups"] == 1
    def narrow(L):
        return L["c_in"] <= 64 or (L["c_in"] <= 160 and L["c_out"] <= 192)
    pw = [i for i, L in enumerate(net.layers) if pointwise(L) and narrow(L)]
    assert len(pw) >= 14, pw
    for i in pw:
        assert names[i].startswith("conv_pw<"), (i, names[i])
    wide = [i for i, L in enumerate(net.layers) if pointwise(L) and not narrow(L)]
    assert wide and all(names[i].startswith("conv_dma<") for i in wide)


@pytest.mark.parametrize("label,rows", NET_CASES)
def test_network_parity_full_batch(P, label, rows):
    net = config(label)
    _say("network", label, "batch", net.batch, "rows", rows)
    params = gen.make_params(net)
    dp = oracle.protect_params(net, params)
    x = gen.make_inputs(net, net.batch)
    cn = _net(P, net, params)
    xd = torch.from_numpy(x).cuda()
    out = cn.forward(xd)
    torch.cuda.synchronize()
    gpu = out.cpu().numpy()
    assert gpu.shape == (net.batch, net.classes + 1)
    rows = list(range(net.batch)) if rows is None else rows
    ref = _oracle_rows(net, dp, x, rows)
    _check_outputs(gpu[rows], ref, net.dtype)
    # repeat run is bit-identical (no races, deterministic order)
    out2 = cn.forward(xd)
    torch.cuda.synchronize()
    assert np.array_equal(out2.cpu().numpy().view(np.uint32),
                          gpu.view(np.uint32))


@pytest.mark.parametrize("label,rows", [("resnet20_f32_b128", list(range(0, 128, 9))),
                                        ("mobilenetv2_f16_b128", [3, 77]),
                                        ("vgg16_f16_b32", [5])])
def test_network_parity_l1_selected_channels(P, label, rows):
    """Networks whose pruned channels were chosen by L1 norm (Sec. II-A)
    through the library, against the oracle's own choice and construction;
    the unprotected output of the swapped parameters equals that of the
    original ones (the swap is a relabelling)."""
    net = config(label)
    _say("network L1 selection", label, rows)
    params = gen.make_params(net)
    q_lib, ch_lib = P.ctc.ctc_select_channels_l1(net.layers, params)
    q_or, ch_or = oracle.select_channels_l1(net, params)
    assert ch_lib == ch_or
    dp = oracle.protect_params(net, q_or)
    x = gen.make_inputs(net, net.batch)
    cn = _net(P, net, q_lib)
    gpu = cn.forward(torch.from_numpy(x).cuda()).cpu().numpy()
    _check_outputs(gpu[rows], _oracle_rows(net, dp, x, rows), net.dtype)
    un_a = P.CtcNet(net.layers, net.in_shape, net.classes, net.dtype, params,
                    protect=False, max_batch=net.batch)
    un_b = P.CtcNet(net.layers, net.in_shape, net.classes, net.dtype, q_lib,
                    protect=False, max_batch=net.batch)
    xd = torch.from_numpy(x).cuda()
    a = un_a.forward(xd).cpu().numpy()
    b = un_b.forward(xd).cpu().numpy()
    rt = 1e-4 if net.dtype == "f32" else 2e-2
    assert np.max(np.abs(a - b)) <= rt * np.max(np.abs(a))


@pytest.mark.parametrize("label,rows", [("tiny_f32_b1", None),
                                        ("resnet20_f32_b128", list(range(3, 128, 11))),
                                        ("resnet18_f16_b64", [2, 50]),
                                        ("mobilenetv2_f16_b128", [9, 120]),
                                        ("vgg16_f16_b32", [17])])
def test_network_parity_append_mode(P, label, rows):
    """Append mode (one extra carry-through channel per layer, widths
    rounded up; nothing pruned) against the oracle's own widening and
    construction; its logits equal the unprotected network's."""
    net = config(label)
    _say("network append mode", label, rows)
    params = gen.make_params(net)
    wn, wp = oracle.append_network(net, params)
    dp = oracle.protect_params(wn, wp)
    x = gen.make_inputs(net, net.batch)
    xd = torch.from_numpy(x).cuda()
    cn = P.CtcNet(net.layers, net.in_shape, net.classes, net.dtype, params,
                  protect="append", max_batch=net.batch)
    gpu = cn.forward(xd).cpu().numpy()
    rows = list(range(net.batch)) if rows is None else rows
    _check_outputs(gpu[rows], _oracle_rows(wn, dp, x, rows), net.dtype)
    got = [tuple(int(v) for v in si) for si in cn.fault_sites(with_acts=True)]
    assert got == [tuple(int(v) for v in si) for si in oracle.fault_sites(wn, dp)]
    un = _net(P, net, params, protect=False)
    u = un.forward(xd).cpu().numpy()
    rt = 1e-4 if net.dtype == "f32" else 2e-2
    assert np.max(np.abs(u - gpu[:, :-1])) <= rt * np.max(np.abs(u))


def test_fused_inverted_residual_blocks(P):
    """With fusion on, MobileNetV2's expand -> depthwise -> project blocks
    (and the first block's depthwise -> project pair) run as one kernel;
    the outputs equal those of the separate kernels (same roundings of the
    internal tensors), and a pass with an activation fault armed on an
    internal tensor runs the separate kernels (the fault lands exactly as
    without fusion)."""
    net = config("mobilenetv2_f16_b128")
    _say("fused inverted residual blocks")
    params = gen.make_params(net)
    B = 16
    cn = _net(P, net, params, max_batch=B)
    names = [P.ctc.ctc_net_op_kernel(cn.h, i, B) for i in range(len(net.layers))]
    nf = sum(n.startswith("conv_ir") for n in names)
    # on by default: 12 of the 16 blocks with an expand conv (not the ones
    # on 7x7 maps)
    assert nf == 3 * 12, names
    assert names[6].startswith("conv_ir<1") and not names[42].startswith("conv_ir")
    assert names[3].startswith("conv_ir<2") and names[21].startswith("conv_ir<1")
    # and the first block (no expand conv): depthwise + pointwise in one
    assert names[1] == names[2] == "conv_dwpw", names[:3]
    x = torch.from_numpy(gen.make_inputs(net, B)).cuda()
    fused = cn.forward(x).cpu().numpy()
    cn.set_fusion(False)
    sep = cn.forward(x).cpu().numpy()
    # same roundings of the internal tensors, same k order: the same bits
    assert np.array_equal(fused.view(np.uint32), sep.view(np.uint32))
    # and the fused path against the oracle directly
    xh = gen.make_inputs(net, B)
    assert np.array_equal(xh, x.cpu().numpy())
    rows = [0, 7, B - 1]
    _check_outputs(fused[rows], _oracle_rows(
        net, oracle.protect_params(net, params), xh, rows), net.dtype)
    # an armed fault on the expand output of block 2 (tensor 7): the fused
    # path falls back to the separate kernels for that pass
    f = [(gen.SITE_ACT, 7, 12345, 14, 3)]
    cn.set_fusion(False)
    cn.inject(f)
    a = cn.forward(x).cpu().numpy()
    cn.clear_faults()
    cn.set_fusion(True)
    cn.inject(f)
    b = cn.forward(x).cpu().numpy()
    cn.clear_faults()
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert not np.array_equal(a[3], sep[3])
    # the same for the depthwise output of the first block (tensor 2)
    f = [(gen.SITE_ACT, 2, 4321, 14, 5)]
    cn.set_fusion(False)
    cn.inject(f)
    a = cn.forward(x).cpu().numpy()
    cn.clear_faults()
    cn.set_fusion(True)
    cn.inject(f)
    b = cn.forward(x).cpu().numpy()
    cn.clear_faults()
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert not np.array_equal(a[5], sep[5])


def _ir_chunk_net():
    """Small fp16 inverted-residual net whose expanded widths end in short
    chunks of the fused kernel's 64-channel walk: E = 88 (64 + 24), 40
    (one chunk of 40), 72 (64 + 8) and 144 (64 + 64 + 16), at stride 1
    and 2, with and without the residual."""
    from workloads.nets import Net, _B
    b = _B()
    t = b.conv(0, 3, 32, 3, 2, 1)                           # 48 -> 24
    for c, e, w, s in ((32, 88, 32, 1), (32, 40, 24, 2), (24, 72, 24, 1),
                       (24, 144, 32, 1)):
        res = s == 1 and c == w
        x = t
        t = b.conv(t, c, e, 1, 1, 0, block_first=res)
        t = b.conv(t, e, e, 3, s, 1, groups=e)
        t = b.conv(t, e, w, 1, 1, 0, relu=False, residual=x if res else -1,
                   gamma_small=res)
    t = b.conv(t, 32, 64, 1, 1, 0)
    t = b.gap(t)
    b.fc(t, 64, 10, final=True)
    return Net("ir_chunks", (3, 48, 48), b.layers, 10, "f16", 8)


def test_fused_inverted_residual_short_chunks(P):
    """Blocks whose expanded width leaves a short last chunk (the waves then
    split the halo tiles) or a single chunk of fewer than 64 channels: the
    fused kernel gives the separate kernels' bits and the oracle's values."""
    net = _ir_chunk_net()
    _say("fused inverted residual, short chunks")
    params = gen.make_params(net, seed=4242)
    B = net.batch
    cn = _net(P, net, params, max_batch=B)
    names = [P.ctc.ctc_net_op_kernel(cn.h, i, B) for i in range(len(net.layers))]
    assert [names[1 + 3 * k].startswith("conv_ir") for k in range(4)] == [True] * 4, names
    xh = gen.make_inputs(net, B, seed=4242)
    x = torch.from_numpy(xh).cuda()
    fused = cn.forward(x).cpu().numpy()
    cn.set_fusion(False)
    sep = cn.forward(x).cpu().numpy()
    assert np.array_equal(fused.view(np.uint32), sep.view(np.uint32))
    rows = [0, 3, B - 1]
    _check_outputs(fused[rows], _oracle_rows(
        net, oracle.protect_params(net, params), xh, rows), net.dtype)


def _dwpw_net():
    """Small fp16 net with two blocks without an expand conv on a 20x20 map
    (16x16 tiles with a ragged edge): depthwise 24 -> pointwise 24 with the
    block input added, then depthwise 24 -> pointwise 40 (three 16-channel
    output tiles, the last one partial)."""
    from workloads.nets import Net, _B
    b = _B()
    t = b.conv(0, 3, 24, 3, 2, 1)                           # 40 -> 20
    x = t
    t = b.conv(t, 24, 24, 3, 1, 1, groups=24)
    t = b.conv(t, 24, 24, 1, 1, 0, relu=False, residual=x, gamma_small=True)
    t = b.conv(t, 24, 24, 3, 1, 1, groups=24)
    t = b.conv(t, 24, 40, 1, 1, 0, relu=False)
    t = b.conv(t, 40, 64, 1, 1, 0)
    t = b.gap(t)
    b.fc(t, 64, 10, final=True)
    return Net("dwpw_pairs", (3, 40, 40), b.layers, 10, "f16", 6)


def test_fused_depthwise_pointwise_pairs(P):
    """Depthwise -> pointwise pairs (no expand conv) on ragged 16x16 tiles,
    with a residual and with several output-channel tiles: the fused
    kernel gives the separate kernels' bits and the oracle's values."""
    net = _dwpw_net()
    _say("fused depthwise + pointwise pairs")
    params = gen.make_params(net, seed=777)
    B = net.batch
    cn = _net(P, net, params, max_batch=B)
    names = [P.ctc.ctc_net_op_kernel(cn.h, i, B) for i in range(len(net.layers))]
    assert names[1:5] == ["conv_dwpw"] * 4, names
    xh = gen.make_inputs(net, B, seed=777)
    x = torch.from_numpy(xh).cuda()
    fused = cn.forward(x).cpu().numpy()
    cn.set_fusion(False)
    sep = cn.forward(x).cpu().numpy()
    assert np.array_equal(fused.view(np.uint32), sep.view(np.uint32))
    rows = [0, 2, B - 1]
    _check_outputs(fused[rows], _oracle_rows(
        net, oracle.protect_params(net, params), xh, rows), net.dtype)


def test_fused_basic_blocks(P):
    """ResNet-20's identity basic blocks (16, 32 and 64 channels) run as one
    kernel per block at full batch (the stem in the first one's kernel, the
    GAP and the classifier in the last one's); the outputs match the
    separate kernels and the oracle, small passes keep the separate
    kernels, and a pass with an activation fault armed on a block's
    internal tensor runs the separate kernels (the fault lands exactly as
    without fusion)."""
    net = config("resnet20_f32_b128")
    params = gen.make_params(net)
    dp = oracle.protect_params(net, params)
    B = 128
    cn = _net(P, net, params, max_batch=B)
    names = [P.ctc.ctc_net_op_kernel(cn.h, i, B) for i in range(len(net.layers))]
    nb = sum(n.startswith("conv_block") for n in names)
    nd = sum(n.startswith("conv_down") for n in names)
    _say("fused basic blocks", names)
    assert nb == 2 * 7 + 1 + 2, names   # 3 blocks at 16, 2 at 32, 2 at 64 channels
    assert names[0] == names[1]         # + the stem, fused into the first block
    # + the GAP and the FC, fused into the last block
    assert names[19] == names[21] == names[22] == "conv_block_gw<4, 8, 1, true>", names
    assert nd == 3 * 2, names           # the 16 -> 32 and 32 -> 64 blocks
    small = [P.ctc.ctc_net_op_kernel(cn.h, i, 8) for i in range(len(net.layers))]
    assert not any(n.startswith("conv_block") for n in small), small
    assert sum(n.startswith("conv_down") for n in small) == 6, small
    assert small[21] == small[22] == "gap_fc_k<1>", small
    x = gen.make_inputs(net, B)
    xd = torch.from_numpy(x).cuda()
    fused = cn.forward(xd).cpu().numpy()
    cn.set_fusion(0)
    sep = cn.forward(xd).cpu().numpy()
    d = np.abs(fused - sep)
    _say("fused vs separate: max abs diff", float(d.max()))
    assert np.max(d) <= 1e-5 * np.max(np.abs(sep))
    rows = [0, 63, 127]
    _check_outputs(fused[rows], _oracle_rows(net, dp, x, rows), "f32")
    # fault on the internal tensor of the first block (tensor 2: output of
    # op 1, read only by op 2): with fusion on, that pass runs the block's
    # two convs separately, so tensor 2 is stored and the fault flips the
    # same bit of it as without fusion
    t2 = cn.tensor(2, B).cpu().numpy().copy()        # fusion off, no fault
    f = [(gen.SITE_ACT, 2, 4321, 30, 5)]
    cn.inject(f)
    a = cn.forward(xd).cpu().numpy()                 # fusion off, fault
    cn.clear_faults()
    cn.set_fusion(P.ctc.CTC_FUSE_BLOCK)
    cn.inject(f)
    b = cn.forward(xd).cpu().numpy()                 # fusion on, fault
    t2f = cn.tensor(2, B).cpu().numpy()
    cn.clear_faults()
    diff = np.nonzero(t2f.view(np.uint32) != t2.view(np.uint32))
    assert len(diff[0]) == 1 and diff[0][0] == 5, diff
    xor = t2f.view(np.uint32)[diff] ^ t2.view(np.uint32)[diff]
    assert int(xor[0]) == 1 << 30
    assert np.max(np.abs(a - b)) <= 1e-5 * np.max(np.abs(a))
    assert not np.array_equal(a[5], sep[5])
    # the same for the stem output (tensor 1, internal to the stem + first
    # block kernel) and the two internal tensors of the 16 -> 32
    # downsampling block (ops 7, 8, 9: tensors 8 = conv1 output, 9 =
    # shortcut output)
    # and the last block's output and the pooled features (tensors 21, 22:
    # internal to the last block's kernel, which then leaves them to the
    # GAP + FC kernel or the separate GAP and FC kernels)
    for t, el in ((1, 777), (8, 777), (9, 777), (21, 777), (22, 7)):
        cn.set_fusion(0)
        cn.forward(xd)
        ref_t = cn.tensor(t, B).cpu().numpy().copy()
        f = [(gen.SITE_ACT, t, el, 29, 9)]
        cn.inject(f)
        a = cn.forward(xd).cpu().numpy()
        cn.clear_faults()
        cn.set_fusion(P.ctc.CTC_FUSE_BLOCK)
        cn.inject(f)
        b = cn.forward(xd).cpu().numpy()
        got_t = cn.tensor(t, B).cpu().numpy()
        cn.clear_faults()
        diff = np.nonzero(got_t.view(np.uint32) != ref_t.view(np.uint32))
        assert len(diff[0]) == 1 and diff[0][0] == 9, (t, diff)
        assert int((got_t.view(np.uint32)[diff] ^ ref_t.view(np.uint32)[diff])[0]) == 1 << 29
        assert np.max(np.abs(a - b)) <= 1e-5 * np.max(np.abs(a))


def test_fused_stem_pool_resnet18_f16(P):
    """ResNet-18 fp16: the 7x7 stride-2 stem and the max pool after it run
    as one kernel, bit-identical to the two separate kernels; a pass with a
    fault armed on the stem output runs them separately, so the fault lands
    in the stored stem output exactly as without the fusion."""
    ctc = P.ctc
    net = config("resnet18_f16_b64")
    params = gen.make_params(net)
    B = 16
    cn = _net(P, net, params, max_batch=B)
    assert [ctc.ctc_net_op_kernel(cn.h, i, B) for i in (0, 1)] == \
        ["conv_stem_pool<7, 2, 2>"] * 2
    x = torch.from_numpy(gen.make_inputs(net, B)).cuda()
    fused = cn.forward(x).cpu().numpy()
    pooled_f = cn.tensor(2, B).cpu().numpy().copy()
    cn.set_fusion(ctc.CTC_FUSE_BLOCK)              # the stem fusion off
    sep = cn.forward(x).cpu().numpy()
    pooled_s = cn.tensor(2, B).cpu().numpy()
    assert np.array_equal(fused.view(np.uint32), sep.view(np.uint32))
    assert np.array_equal(pooled_f.view(np.uint16), pooled_s.view(np.uint16))
    stem = cn.tensor(1, B).cpu().numpy().copy()    # stored while unfused
    f = [(gen.SITE_ACT, 1, 777, 14, 3)]
    cn.inject(f)
    a = cn.forward(x).cpu().numpy()
    cn.clear_faults()
    cn.set_fusion(ctc.CTC_FUSE_BLOCK | ctc.CTC_FUSE_STEM)
    cn.inject(f)
    b = cn.forward(x).cpu().numpy()
    stem_f = cn.tensor(1, B).cpu().numpy()
    cn.clear_faults()
    diff = np.nonzero(stem_f.view(np.uint16) != stem.view(np.uint16))
    assert len(diff[0]) == 1 and diff[0][0] == 3, diff
    assert int((stem_f.view(np.uint16)[diff] ^ stem.view(np.uint16)[diff])[0]) == 1 << 14
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_fused_conv_pool_vgg16(P):
    """VGG-16 fp16: the 2x2 max pools run in the epilogue of the conv before
    them (every one whose kernel has the pool: all but the 14x14 one), with
    results bit-identical to the separate kernels; a pass with a fault armed
    on a pooled conv's output runs the conv and the pool separately, so the
    fault lands in the stored conv output exactly as without the fusion."""
    ctc = P.ctc
    net = config("vgg16_f16_b32")
    params = gen.make_params(net)
    B = net.batch
    cn = _net(P, net, params, max_batch=B)
    names = [ctc.ctc_net_op_kernel(cn.h, i, B) for i in range(len(net.layers))]
    pools = [i for i, L in enumerate(net.layers) if L["op"] == "maxpool"]
    _say("vgg16 kernels", names)
    fused = [i for i in pools if names[i] == names[i - 1]]
    assert len(pools) == 5 and len(fused) == 4, names
    assert names.count("maxpool_fixed<_Float16, 2, 2>") == 1
    assert any(n.startswith("conv_pp<256, 224, 8, true>") for n in names)
    # conv1_2 pools in the halo-tile epilogue, conv2_2 in conv_dma's
    assert "conv_dma<_Float16, 128, 64, 2, 2, 2, true, 16, true, 1>" in names
    assert "conv_dma<_Float16, 128, 128, 2, 2, 2, true, 16, true, 0>" in names
    x = torch.from_numpy(gen.make_inputs(net, B)).cuda()
    on = cn.forward(x).cpu().numpy()
    pooled_on = [cn.tensor(i + 1, B).cpu().numpy().copy() for i in fused]
    cn.set_fusion(ctc.CTC_FUSE_BLOCK | ctc.CTC_FUSE_STEM)
    off = cn.forward(x).cpu().numpy()
    pooled_off = [cn.tensor(i + 1, B).cpu().numpy().copy() for i in fused]
    assert np.array_equal(on.view(np.uint32), off.view(np.uint32))
    for a, b in zip(pooled_on, pooled_off):
        assert np.array_equal(a.view(np.uint16), b.view(np.uint16))
    # fault on the output of the conv before the third pool (internal to
    # the fused kernel): fusion on and off give the same stored tensor
    t = fused[2]                          # conv output tensor id = pool op
    conv_out = cn.tensor(t, B).cpu().numpy().copy()     # unfused, no fault
    f = [(gen.SITE_ACT, t, 4321, 14, 7)]
    cn.inject(f)
    a = cn.forward(x).cpu().numpy()
    cn.clear_faults()
    cn.set_fusion(ctc.CTC_FUSE_BLOCK | ctc.CTC_FUSE_STEM | ctc.CTC_FUSE_POOL)
    cn.inject(f)
    b = cn.forward(x).cpu().numpy()
    got = cn.tensor(t, B).cpu().numpy()
    cn.clear_faults()
    diff = np.nonzero(got.view(np.uint16) != conv_out.view(np.uint16))
    assert len(diff[0]) == 1 and diff[0][0] == 7, diff
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


# VGG-16 convs on a 32x32 input (one 512-channel pixel into the FCs) with
# hidden / classifier widths that give ragged row blocks, k tails, one or
# several k ranges and 1-3 image tiles of fc_sk (and fc_k for small layers)
FC_CASES = [
    # dtype, batch, hidden, classes, classifier_f32, rows
    ("f16", 1, 200, 37, True, [0]),
    ("f16", 33, 1000, 300, True, [0, 16, 32]),
    ("f16", 70, 520, 1001, True, [0, 47, 69]),
    ("f16", 20, 264, 63, False, [0, 19]),
    ("f32", 40, 300, 100, True, [0, 21, 39]),
]


@pytest.mark.parametrize("dtype,B,hidden,classes,f32c,rows", FC_CASES)
def test_fc_layers_split_k(P, dtype, B, hidden, classes, f32c, rows):
    """The FC kernels (fc_sk over k ranges + fc_sk_reduce, fc_k for small
    layers) in every input / weight / output type combination the runner
    uses, against the oracle, at the full batch and for one image; the
    repeat run is bit-identical."""
    net = by_name("vgg16", batch=B, dtype=dtype, classes=classes,
                  classifier_f32=f32c, in_hw=32, hidden=hidden)
    params = gen.make_params(net)
    dp = oracle.protect_params(net, params)
    x = gen.make_inputs(net, B)
    cn = _net(P, net, params)
    names = [P.ctc.ctc_net_op_kernel(cn.h, i, B)
             for i in range(len(net.layers)) if net.layers[i]["op"] == "fc"]
    _say("fc case", dtype, B, hidden, classes, f32c, names)
    assert any(n.startswith("fc_sk<") for n in names), names
    xd = torch.from_numpy(x).cuda()
    out = cn.forward(xd)
    torch.cuda.synchronize()
    gpu = out.cpu().numpy()
    _check_outputs(gpu[rows], _oracle_rows(net, dp, x, rows), dtype)
    out2 = cn.forward(xd)
    torch.cuda.synchronize()
    assert np.array_equal(out2.cpu().numpy().view(np.uint32), gpu.view(np.uint32))
    # the last image alone (one image tile, the same k ranges)
    one = cn.forward(xd[B - 1:B].contiguous())
    torch.cuda.synchronize()
    _check_outputs(one.cpu().numpy(), _oracle_rows(net, dp, x, [B - 1]), dtype)


def test_fused_head_reads_the_current_pass(P):
    """The last block's kernel pools tiles that other workgroups of the same
    launch stored: three different batches back to back, each bit-identical
    to the separate kernels."""
    net = config("resnet20_f32_b128")
    params = gen.make_params(net)
    B = 128
    cn = _net(P, net, params, max_batch=B)
    assert P.ctc.ctc_net_op_kernel(cn.h, 21, B).endswith("true>")
    xs = [torch.from_numpy(gen.make_inputs(net, B, offset=k * B)).cuda()
          for k in range(3)]
    fused = [cn.forward(x).cpu().numpy() for x in xs]
    cn.set_fusion(0)
    sep = [cn.forward(x).cpu().numpy() for x in xs]
    for f, s in zip(fused, sep):
        assert np.array_equal(f.view(np.uint32), s.view(np.uint32))
    assert not np.array_equal(fused[0], fused[1])


@pytest.mark.parametrize("shape,B,kernel,nfused", [
    ((3, 20, 28), 128, "conv_block<16, 8, 16, 32", 17),
    ((3, 32, 32), 64, "conv_block<16, 4, 8, 32", 7),
    ((3, 31, 17), 16, "conv_tile", 0)])
def test_fused_basic_blocks_ragged_and_small_tiles(P, shape, B, kernel, nfused):
    """Fused blocks on images that do not divide into tiles (20 x 28: tiles
    run past the bottom and right edges at every width; 31 x 17: odd sizes
    into the stride-2 blocks, a batch too small for the identity blocks to
    fuse) and with the 8 x 32 tile of half batches (whose 32- and 64-channel
    identity blocks are too few tiles to fuse), against the oracle."""
    net = config("resnet20_f32_b128").copy(in_shape=shape, batch=B)
    _say("fused blocks", shape, B)
    params = gen.make_params(net)
    dp = oracle.protect_params(net, params)
    cn = _net(P, net, params, max_batch=B)
    names = [P.ctc.ctc_net_op_kernel(cn.h, i, B) for i in range(len(net.layers))]
    assert names[1].startswith(kernel) and names[2].startswith(kernel), names
    assert sum(n.startswith("conv_block") for n in names) == nfused, names
    assert sum(n.startswith("conv_down") for n in names) == 6, names
    x = gen.make_inputs(net, B)
    out = cn.forward(torch.from_numpy(x).cuda()).cpu().numpy()
    rows = [0, B // 2 + 1, B - 1]
    _check_outputs(out[rows], _oracle_rows(net, dp, x, rows), "f32")


@pytest.mark.parametrize("B,maxb", [(128, 128), (96, 96), (100, 128)])
def test_fused_stem_stages_the_pass_input(P, B, maxb):
    """When a pass converts exactly the caller's images, the fused stem +
    block kernel reads them itself (no assembly launch) and stores the
    converted input that later re-executions read: tensor 0 holds the
    images in NHWC with a zero fourth channel, bit for bit; the outputs
    equal the unfused path's; with every image flagged, the deferred re-runs
    (read back from those stored copies) give the same rows.  Batch 128
    takes the 16 x 32 tile, batch 96 the 8 x 32 one; 100 images on a net
    bound for 128 run a pass below the bound."""
    ctc = P.ctc
    net = config("resnet20_f32_b128").copy(batch=B)
    _say("fused stem staging", B, maxb)
    params = gen.make_params(net)
    cn = _net(P, net, params, max_batch=maxb)
    kern = "conv_block<16, 8, 16, 32" if B == 128 else "conv_block<16, 4, 8, 32"
    assert ctc.ctc_net_op_kernel(cn.h, 0, B).startswith(kern)
    x = gen.make_inputs(net, B, offset=7)
    xd = torch.from_numpy(x).cuda()
    cn.set_threshold(0.0, float("inf"))
    out = cn.forward(xd).clone()
    torch.cuda.synchronize()
    t0 = cn.tensor(0, B).cpu().numpy()
    exp = np.zeros((B, 32, 32, 4), np.float32)
    exp[..., :3] = x.transpose(0, 2, 3, 1)
    assert np.array_equal(t0.view(np.uint32), exp.view(np.uint32))
    cn.set_fusion(0)
    unfused = cn.forward(xd).clone()
    cn.set_fusion(ctc.CTC_FUSE_BLOCK | ctc.CTC_FUSE_STEM)
    assert np.array_equal(out.cpu().numpy(), unfused.cpu().numpy())
    cn.set_threshold(0.0, -1.0)
    o = torch.full_like(out, float("nan"))
    fl = torch.zeros(B, dtype=torch.uint8, device="cuda")
    cn.forward(xd, out=o, flags=fl, reexec=ctc.CTC_REEXEC_DEFERRED)
    cn.flush()
    torch.cuda.synchronize()
    assert fl.cpu().numpy().all()
    assert np.array_equal(o.cpu().numpy(), out.cpu().numpy())


def test_fused_stem_stages_reruns_and_overflow(P):
    """Deferred passes of the usual mixed shape, staged inside the fused
    stem + block kernel: two images of call 1 flagged (a fault on their S)
    come back in a later call's pass as its last two rows, read from their
    ring slots, and push that call's last two images into ring slots
    (converted by the kernel's extra workgroups), which the next pass reads.
    Ten calls, so the re-runs land in a pass of a call, not in the flush.
    Every row ends up equal to the fault-free result of the unfused
    path."""
    ctc = P.ctc
    B = 128
    net = config("resnet20_f32_b128")
    _say("fused stem staging, re-runs + overflow")
    params = gen.make_params(net)
    cn = _net(P, net, params, max_batch=B)
    assert ctc.ctc_net_op_kernel(cn.h, 0, B).startswith("conv_block<16, 8, 16, 32")
    xs = [torch.from_numpy(gen.make_inputs(net, B, offset=B * i)).cuda()
          for i in range(10)]
    cn.set_fusion(0)
    clean = [cn.forward(x).clone() for x in xs]
    cn.set_fusion(ctc.CTC_FUSE_BLOCK | ctc.CTC_FUSE_STEM)
    S = torch.cat(clean)[:, -1].cpu().numpy().astype(np.float64)
    cn.set_threshold(float(S.mean()), float(np.abs(S - S.mean()).max() * 1.01))
    cn.inject([(ctc.CTC_SITE_ACT, len(net.layers), net.classes, 30, 5),
               (ctc.CTC_SITE_ACT, len(net.layers), net.classes, 30, 70)])
    outs = [torch.full_like(clean[0], float("nan")) for _ in range(10)]
    fl = torch.zeros(B, dtype=torch.uint8, device="cuda")
    cn.forward(xs[0], out=outs[0], flags=fl, reexec=ctc.CTC_REEXEC_DEFERRED)
    cn.clear_faults()
    for x, o in zip(xs[1:], outs[1:]):
        cn.forward(x, out=o, reexec=ctc.CTC_REEXEC_DEFERRED)
    cn.flush()
    torch.cuda.synchronize()
    f = fl.cpu().numpy()
    assert f[5] == 1 and f[70] == 1 and f.sum() == 2
    for o, c in zip(outs, clean):
        assert np.array_equal(o.cpu().numpy(), c.cpu().numpy())


def test_deferred_and_single_pass_calls_interleaved(P):
    """Deferred calls interleaved with single-pass (NONE) calls on one net,
    twelve calls: the flag rows of deferred passes reach the host through
    later passes of either kind (four at a time) or the flush, and waits
    use the events of later passes.  A fault on S of image 9 in the first
    deferred call is re-executed; every deferred row ends equal to the
    fault-free result, and the single-pass calls give their own rows and
    flags (all clear) at once."""
    ctc = P.ctc
    B = 64
    net = config("resnet20_f32_b128")
    _say("interleaved deferred / single-pass calls")
    params = gen.make_params(net)
    cn = _net(P, net, params, max_batch=B)
    xs = [torch.from_numpy(gen.make_inputs(net, B, offset=B * i)).cuda()
          for i in range(12)]
    clean = [cn.forward(x).clone() for x in xs]
    S = torch.cat(clean)[:, -1].cpu().numpy().astype(np.float64)
    cn.set_threshold(float(S.mean()), float(np.abs(S - S.mean()).max() * 1.01))
    outs = [torch.full_like(clean[0], float("nan")) for _ in range(12)]
    fls = [torch.full((B,), 7, dtype=torch.uint8, device="cuda") for _ in range(12)]
    for i, (x, o, f) in enumerate(zip(xs, outs, fls)):
        if i == 0:
            cn.inject([(ctc.CTC_SITE_ACT, len(net.layers), net.classes, 30, 9)])
        m = ctc.CTC_REEXEC_DEFERRED if i % 3 != 2 else ctc.CTC_REEXEC_NONE
        cn.forward(x, out=o, flags=f, reexec=m)
        if i == 0:
            cn.clear_faults()
        if m == ctc.CTC_REEXEC_NONE:
            torch.cuda.synchronize()
            assert np.array_equal(o.cpu().numpy(), clean[i].cpu().numpy()), i
            assert not f.cpu().numpy().any(), i
    cn.flush()
    torch.cuda.synchronize()
    f0 = fls[0].cpu().numpy()
    assert f0[9] == 1 and f0.sum() == 1
    for i in range(1, 12):
        assert not fls[i].cpu().numpy().any(), i
    for i, (o, c) in enumerate(zip(outs, clean)):
        assert np.array_equal(o.cpu().numpy(), c.cpu().numpy()), i


def test_intermediate_tensors_resnet20(P):
    """Every stored tensor of the protected ResNet-20 against the oracle's
    (debug-mode parity), including the checksum channels.  Fusion off: a
    fused block does not store its internal tensors."""
    net = config("resnet20_f32_b128")
    params = gen.make_params(net)
    dp = oracle.protect_params(net, params)
    x = gen.make_inputs(net, 4)
    cn = _net(P, net, params, max_batch=4)
    cn.set_fusion(0)
    cn.forward(torch.from_numpy(x).cuda())
    torch.cuda.synchronize()
    T = oracle.forward_image(net, dp, x[2], keep=True)
    for t in range(1, len(net.layers)):
        g = cn.tensor(t, 4)[2].float().cpu().numpy()
        r = T[t].transpose(1, 2, 0)
        g = g[..., :r.shape[2]]
        assert np.max(np.abs(g - r)) <= 1e-4 * max(np.max(np.abs(r)), 1e-3), t


def test_unprotected_network_matches_oracle(P):
    net = config("resnet20_f32_b128")
    params = gen.make_params(net)
    dpu = oracle.protect_params(net, params, protect=False)
    x = gen.make_inputs(net, 16)
    cn = _net(P, net, params, protect=False, max_batch=16)
    out = cn.forward(torch.from_numpy(x).cuda())
    torch.cuda.synchronize()
    gpu = out.cpu().numpy()
    assert gpu.shape == (16, net.classes)
    ref = np.stack([oracle.forward_image(net, dpu, xi, protect=False)
                    for xi in x[:4]])
    for g, r in zip(gpu[:4], ref):
        assert np.max(np.abs(g - r)) <= 1e-4 * np.max(np.abs(r))


def _band(S, ref, tau, rt):
    """Rows whose deviation sits within the rounding band of tau."""
    dev = np.abs(np.asarray(S, np.float64) - ref)
    return np.abs(dev - tau) <= 4 * rt * np.maximum(np.abs(S), abs(ref))


def test_flags_match_oracle_tiny(P):
    """Distribution-based tau from the oracle's calibration set; the GPU's
    flags on 512 fresh images equal the oracle's outside the band."""
    net = config("tiny_f32_b1")
    params = gen.make_params(net)
    dp = oracle.protect_params(net, params)
    cal = oracle.forward_batch(net, dp, gen.make_inputs(
        net, 1000, stream=gen.S_CALIB), threads=THREADS)[:, -1]
    ref, tau = oracle.calibrate(cal, 0.05)
    x = gen.make_inputs(net, 512)
    So = oracle.forward_batch(net, dp, x, threads=THREADS)[:, -1]
    cn = _net(P, net, params, max_batch=512)
    cn.set_threshold(ref, tau)
    fl = torch.zeros(512, dtype=torch.uint8, device="cuda")
    out = cn.forward(torch.from_numpy(x).cuda(), flags=fl)
    torch.cuda.synchronize()
    f_gpu = fl.cpu().numpy().astype(bool)
    f_or = oracle.verify(So, ref, tau)
    keep = ~_band(So, ref, tau, 1e-4)
    assert f_or.sum() > 5
    assert np.array_equal(f_gpu[keep], f_or[keep])
    assert np.array_equal(f_gpu, oracle.verify(out.cpu().numpy()[:, -1], ref,
                                               tau))


@pytest.mark.parametrize("mode", ["sync", "deferred"])
def test_reexecution_rewrites_flagged_rows(P, mode):
    """tau = -1 flags every image; each is re-executed once and its row
    rewritten with an identical result (faults absent), the re-run's own
    flag being ignored."""
    ctc = P.ctc
    net = config("resnet20_f32_b128")
    params = gen.make_params(net)
    cn = _net(P, net, params, max_batch=32)
    xs = [torch.from_numpy(gen.make_inputs(net, 32, offset=32 * i)).cuda()
          for i in range(4)]
    cn.set_threshold(0.0, float("inf"))
    base = [cn.forward(x).clone() for x in xs]
    cn.set_threshold(0.0, -1.0)
    m = ctc.CTC_REEXEC_SYNC if mode == "sync" else ctc.CTC_REEXEC_DEFERRED
    outs = []
    for x in xs:
        o = torch.full_like(base[0], float("nan"))
        fl = torch.zeros(32, dtype=torch.uint8, device="cuda")
        cn.forward(x, out=o, flags=fl, reexec=m)
        outs.append((o, fl))
    cn.flush()
    torch.cuda.synchronize()
    for (o, fl), b in zip(outs, base):
        assert fl.cpu().numpy().all()
        assert np.array_equal(o.cpu().numpy(), b.cpu().numpy())


def test_deferred_reexec_replaces_faulty_rows(P):
    """An activation fault that corrupts S of one image: the flagged image
    is re-run (fault gone, transient) two calls later and its row ends up
    equal to the fault-free result."""
    ctc = P.ctc
    net = config("resnet20_f32_b128")
    params = gen.make_params(net)
    cn = _net(P, net, params, max_batch=16)
    x = torch.from_numpy(gen.make_inputs(net, 16)).cuda()
    clean = cn.forward(x).clone()
    S = clean[:, -1].cpu().numpy().astype(np.float64)
    ref, tau = float(S.mean()), float(np.abs(S - S.mean()).max() * 1.01)
    cn.set_threshold(ref, tau)
    # top exponent bit of S of image 5 (S ~ 4e2: the flip makes it ~0)
    cn.inject([(ctc.CTC_SITE_ACT, len(net.layers), net.classes, 30, 5)])
    o1 = torch.empty_like(clean)
    f1 = torch.zeros(16, dtype=torch.uint8, device="cuda")
    cn.forward(x, out=o1, flags=f1, reexec=ctc.CTC_REEXEC_DEFERRED)
    torch.cuda.synchronize()
    assert f1.cpu().numpy().tolist() == [0] * 5 + [1] + [0] * 10
    assert o1[5, -1].item() != clean[5, -1].item()
    cn.clear_faults()
    o2 = torch.empty_like(clean)
    o3 = torch.empty_like(clean)
    cn.forward(x, out=o2, reexec=ctc.CTC_REEXEC_DEFERRED)
    cn.forward(x, out=o3, reexec=ctc.CTC_REEXEC_DEFERRED)   # re-runs image 5
    cn.flush()
    torch.cuda.synchronize()
    assert np.array_equal(o1.cpu().numpy(), clean.cpu().numpy())
    assert np.array_equal(o3.cpu().numpy(), clean.cpu().numpy())


def test_deferred_reexec_input_fault_is_transient(P):
    """A fault armed on the network input (tensor 0) of one image: the pass
    it hits flags the image, and the re-execution reads the input as it was
    staged before the fault, so the row ends up equal to the fault-free
    result.  The later calls (no fault armed) convert their images straight
    into ring slots and copy the re-run in after them."""
    ctc = P.ctc
    net = config("resnet20_f32_b128")
    params = gen.make_params(net)
    cn = _net(P, net, params, max_batch=16)
    x = torch.from_numpy(gen.make_inputs(net, 16)).cuda()
    clean = cn.forward(x).clone()
    S = clean[:, -1].cpu().numpy().astype(np.float64)
    ref, tau = float(S.mean()), float(np.abs(S - S.mean()).max() * 1.01)
    cn.set_threshold(ref, tau)
    # top exponent bit of input channel 0, pixel 100 of image 3
    cn.inject([(ctc.CTC_SITE_ACT, 0, 100, 30, 3)])
    o1 = torch.empty_like(clean)
    f1 = torch.zeros(16, dtype=torch.uint8, device="cuda")
    cn.forward(x, out=o1, flags=f1, reexec=ctc.CTC_REEXEC_DEFERRED)
    torch.cuda.synchronize()
    assert f1.cpu().numpy().tolist() == [0] * 3 + [1] + [0] * 12
    assert o1[3, -1].item() != clean[3, -1].item()
    cn.clear_faults()
    outs = [torch.empty_like(clean) for _ in range(3)]
    for o in outs:
        cn.forward(x, out=o, reexec=ctc.CTC_REEXEC_DEFERRED)
    cn.flush()
    torch.cuda.synchronize()
    assert np.array_equal(o1.cpu().numpy(), clean.cpu().numpy())
    for o in outs:
        assert np.array_equal(o.cpu().numpy(), clean.cpu().numpy())


# ----------------------------------------------------------------- faults

def _oracle_fault_run(net, dp, x, T, f):
    if f["site"] == gen.SITE_ACT:
        t = int(f["layer"])
        if t == 0:
            return oracle.forward_image(net, dp, x, act_faults=[
                (0, int(f["index"]), int(f["bit"]))])
        acts = list(T)
        acts[t] = T[t].copy()
        oracle.core._flip(acts[t], int(f["index"]), int(f["bit"]),
                          oracle.stored_f32(net, t))
        if t == len(net.layers):
            return acts[t].reshape(-1).copy()
        return oracle.forward_image(net, dp, None, start=t, acts=acts)
    oracle.apply_param_fault(net, dp, f["site"], f["layer"], f["index"],
                             f["bit"])
    try:
        return oracle.forward_image(net, dp, x, start=int(f["layer"]), acts=T)
    finally:
        oracle.apply_param_fault(net, dp, f["site"], f["layer"], f["index"],
                                 f["bit"])


def test_fault_campaign_flags_match_oracle_tiny(P):
    """Seeded single-bit faults (parameters one at a time, activations one
    per batch row) on the tiny net: identical detection flags and critical
    labels, outside the rounding band of tau and of near-ties."""
    ctc = P.ctc
    net = config("tiny_f32_b1")
    params = gen.make_params(net)
    dp = oracle.protect_params(net, params)
    cal = oracle.forward_batch(net, dp, gen.make_inputs(
        net, 1000, stream=gen.S_CALIB), threads=THREADS)[:, -1]
    ref, tau = oracle.calibrate(cal, 0.01)
    x = gen.make_inputs(net, 1)
    T = oracle.forward_image(net, dp, x[0], keep=True)
    gold = T[-1].reshape(-1)
    sites = oracle.fault_sites(net, dp)
    psites = [s for s in sites if s[0] != gen.SITE_ACT]
    asites = [s for s in sites if s[0] == gen.SITE_ACT]
    pf = gen.sample_faults(psites, 600, 21)
    af = gen.sample_faults(asites, 1024, 22)
    B = 256
    cn = _net(P, net, params, max_batch=B)
    cn.set_threshold(ref, tau)
    x1 = torch.from_numpy(x).cuda()
    xb = x1.expand(B, -1, -1, -1).contiguous()
    gpu_out, gpu_flag = [], []
    fl = torch.zeros(B, dtype=torch.uint8, device="cuda")
    for f in pf:
        cn.inject([tuple(f)])
        gpu_out.append(cn.forward(x1, flags=fl[:1]).cpu().numpy()[0])
        gpu_flag.append(bool(fl[0].item()))
        cn.clear_faults()
    for s in range(0, len(af), B):
        chunk = af[s:s + B].copy()
        chunk["image"] = np.arange(len(chunk))
        cn.inject([tuple(f) for f in chunk])
        n = len(chunk)
        gpu_out.extend(cn.forward(xb[:n], flags=fl[:n]).cpu().numpy())
        gpu_flag.extend(fl[:n].cpu().numpy().astype(bool).tolist())
        cn.clear_faults()
    allf = np.concatenate([pf, af])
    _say("faults", len(allf))
    from concurrent.futures import ThreadPoolExecutor

    def orun(f):
        ldp = [None if p is None else {k: v.copy() for k, v in p.items()}
               for p in dp]
        return _oracle_fault_run(net, ldp, x[0], T, f)
    with ThreadPoolExecutor(THREADS) as ex:
        or_out = list(ex.map(orun, allf))
    n_band = n_cmp = n_flag = n_crit = 0
    for f, g, r, fg in zip(allf, gpu_out, or_out, gpu_flag):
        Sg, So = g[-1], r[-1]
        # the flag byte the fused detector wrote, decided on the GPU's S
        assert fg == bool(oracle.verify([Sg], ref, tau)[0])
        fo = bool(oracle.verify([So], ref, tau)[0])
        cg = oracle.is_critical(g[:-1], gold[:-1])
        co = oracle.is_critical(r[:-1], gold[:-1])
        near = np.isfinite(So) and _band([So], ref, tau, 1e-4)[0]
        lr = r[:-1]
        if np.all(np.isfinite(lr)):
            top2 = np.sort(lr)[-2:]
            near = near or (top2[1] - top2[0]) <= 4e-4 * np.max(np.abs(lr))
        if near:
            n_band += 1
            continue
        n_cmp += 1
        n_flag += fo
        n_crit += co
        assert fg == fo, (tuple(f), Sg, So)
        assert cg == co, (tuple(f), g, r)
    _say("compared", n_cmp, "band", n_band, "flagged", n_flag, "critical",
         n_crit)
    assert n_band <= 0.01 * len(allf) and n_flag > 10 and n_crit > 10
