"""Host-side checks of libctc.so that need no GPU: every symbol declared in
include/ctc.h is exported, the carry-through construction is bit-identical
to the oracle's, the threshold helper matches the oracle, and plan
validation rejects unsupported networks before any device work."""

import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from workloads import CONFIGS, by_name, config, gen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

ctc = pytest.importorskip("paper_2609_16742_amd.ctc")


def _declared_symbols():
    src = open(os.path.join(ROOT, "include", "ctc.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ctc_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    syms = _declared_symbols()
    assert len(syms) >= 18
    lib = ctypes.CDLL(ctc.LIB_PATH)
    for s in syms:
        assert hasattr(lib, s), s
    assert sorted(ctc.EXPORTS) == syms
    assert ctc.ctc_abi_version() == 3


ALL_NETS = {lab: config(lab) for lab in CONFIGS if lab != "resnet18_f32_b64"}


@pytest.fixture(scope="module")
def nets_and_params():
    out = {}
    for lab, net in ALL_NETS.items():
        if net.name == "vgg16":   # same layer structure, smaller classifier
            net = by_name("vgg16", in_hw=64, hidden=256, classes=100)
        out[lab] = (net, gen.make_params(net))
    return out


def test_builder_matches_oracle_construction(nets_and_params):
    """Each side builds the protected parameters on its own; the results
    must agree bit for bit on every layer of every workload."""
    for lab, (net, params) in nets_and_params.items():
        dp = oracle.protect_params(net.copy(dtype="f32"), params)
        for i, (L, p, q) in enumerate(zip(net.layers, params, dp)):
            if L["op"] == "conv":
                role = {oracle.ROLE_SUM: ctc.CTC_ROLE_SUM,
                        oracle.ROLE_ZERO: ctc.CTC_ROLE_ZERO,
                        oracle.ROLE_PASS: ctc.CTC_ROLE_PASS}[
                            oracle.conv_role(L)]
                d = ctc.layer_desc(L["c_in"], L["c_out"], L["k"], L["k"],
                                   L["stride"], L["pad"], L["groups"],
                                   int(L["inp"] != 0), role)
                arrs = {k: v.copy() for k, v in p.items()}
                ctc.ctc_build_filters(d, arrs["w"], arrs.get("b"),
                                      arrs.get("mean"), arrs.get("var"),
                                      arrs.get("gamma"), arrs.get("beta"))
                for k in arrs:
                    assert np.array_equal(arrs[k].view(np.uint32),
                                          q[k].view(np.uint32)), (lab, i, k)
            elif L["op"] == "fc":
                ck = oracle.checksum_features(net, L)
                rows = L["out_f"] + (1 if L["final"] else 0)
                w = np.zeros((rows, L["in_f"]), np.float32)
                b = np.zeros(rows, np.float32)
                ctc.ctc_build_fc(L["in_f"], L["out_f"], int(ck[0]), len(ck),
                                 int(L["final"]), p["w"], p["b"], w, b)
                assert np.array_equal(w, q["w"]) and np.array_equal(b, q["b"])


def test_builder_rejects_bad_layers():
    w = np.zeros((4, 4, 2, 2), np.float32)
    with pytest.raises(ctc.CtcError) as e:
        ctc.ctc_build_filters(ctc.layer_desc(4, 4, 2, 2, 1, 0, 1, 1,
                                             ctc.CTC_ROLE_SUM), w)
    assert e.value.status == ctc.CTC_ERR_UNSUPPORTED
    with pytest.raises(ctc.CtcError) as e:
        ctc.ctc_build_filters(ctc.layer_desc(4, 8, 3, 3, 1, 1, 2, 1,
                                             ctc.CTC_ROLE_SUM),
                              np.zeros((8, 2, 3, 3), np.float32))
    assert e.value.status == ctc.CTC_ERR_UNSUPPORTED
    with pytest.raises(ctc.CtcError):
        ctc.ctc_build_filters(ctc.layer_desc(4, 4, 3, 3, 1, 1, 1, 1, 9),
                              np.zeros((4, 4, 3, 3), np.float32))


@pytest.mark.parametrize("n,alpha", [(1, 0.01), (10, 0.1), (1000, 0.01),
                                     (997, 0.05), (5000, 0.001)])
def test_threshold_matches_oracle(n, alpha):
    S = np.random.default_rng(n).standard_normal(n) * 5 + 100
    r1, t1 = ctc.ctc_threshold_from_samples(S, alpha)
    r2, t2 = oracle.calibrate(S, alpha)
    # the means differ only by summation order; tau moves with them
    assert abs(r1 - r2) <= 1e-12 * abs(r2)
    assert abs(t1 - t2) <= abs(r1 - r2) + 1e-12 * abs(t2)


@pytest.mark.parametrize("n,alpha", [(1, 0.01), (10, 0.1), (1000, 0.01),
                                     (997, 0.05), (5000, 0.001)])
def test_threshold_at_ref_matches_oracle(n, alpha):
    g = np.random.default_rng(7 + n)
    S = g.standard_normal(n) * 5 + 100
    S[g.random(n) < 0.02] = np.nan          # non-finite faulty S values
    S[g.random(n) < 0.01] = np.inf
    assert ctc.ctc_threshold_at_ref(S, 99.0, alpha) == \
        oracle.threshold_at_ref(S, 99.0, alpha)


def test_threshold_rejects_bad_args():
    with pytest.raises(ctc.CtcError):
        ctc.ctc_threshold_from_samples(np.zeros(0), 0.01)
    with pytest.raises(ctc.CtcError):
        ctc.ctc_threshold_from_samples(np.zeros(4), 1.5)
    with pytest.raises(ctc.CtcError):
        ctc.ctc_threshold_at_ref(np.zeros(0), 0.0, 0.01)
    with pytest.raises(ctc.CtcError):
        ctc.ctc_threshold_at_ref(np.zeros(4), float("nan"), 0.01)


def test_roles_derived_like_oracle():
    for lab in ("resnet20_f32_b128", "mobilenetv2_f16_b128",
                "resnet18_f16_b64", "tiny_f32_b1"):
        net = config(lab)
        h = ctc.ctc_net_create(ctc.ops_from_layers(net.layers),
                               *net.in_shape, net.classes,
                               ctc.DTYPES[net.dtype], 1)
        try:
            for i, L in enumerate(net.layers):
                r = ctc.ctc_net_role(h, i)
                if L["op"] != "conv":
                    assert r == ctc.CTC_ROLE_NONE
                    continue
                want = {oracle.ROLE_SUM: ctc.CTC_ROLE_SUM,
                        oracle.ROLE_ZERO: ctc.CTC_ROLE_ZERO,
                        oracle.ROLE_PASS: ctc.CTC_ROLE_PASS}[
                            oracle.conv_role(L)]
                assert r == want, (lab, i)
            assert ctc.ctc_net_workspace_bytes(h, net.batch) > 0
        finally:
            ctc.ctc_net_destroy(h)


def test_net_create_rejects_unsupported():
    net = by_name("tiny")
    layers = [dict(L) for L in net.layers]
    layers[0]["c_out"] = 18          # not a multiple of 4
    layers[1]["c_in"] = 18
    with pytest.raises(ctc.CtcError) as e:
        ctc.ctc_net_create(ctc.ops_from_layers(layers), 3, 32, 32, 10,
                           ctc.CTC_F32, 1)
    assert e.value.status == ctc.CTC_ERR_UNSUPPORTED
    layers = [dict(L) for L in net.layers]
    layers[1]["c_in"] = 8            # shape mismatch
    with pytest.raises(ctc.CtcError) as e:
        ctc.ctc_net_create(ctc.ops_from_layers(layers), 3, 32, 32, 10,
                           ctc.CTC_F32, 1)
    assert e.value.status == ctc.CTC_ERR_ARG
    with pytest.raises(ctc.CtcError):
        ctc.ctc_net_create(ctc.ops_from_layers(net.layers), 5, 32, 32, 10,
                           ctc.CTC_F32, 1)


@pytest.mark.parametrize("label", ["tiny_f32_b1", "resnet20_f32_b128",
                                   "resnet18_f16_b64", "vgg16_f16_b32",
                                   "mobilenetv2_f16_b128"])
def test_l1_selection_matches_oracle(label):
    """The library's L1-norm channel choice and swap (Sec. II-A) equal the
    oracle's, array for array, bit for bit."""
    from workloads import config, gen
    net = config(label)
    params = gen.make_params(net)
    got, ch_got = ctc.ctc_select_channels_l1(net.layers, params)
    want, ch_want = oracle.select_channels_l1(net, params)
    assert ch_got == ch_want
    for g, w in zip(got, want):
        if w is None:
            assert g is None
            continue
        assert sorted(g) == sorted(w)
        for k in w:
            assert np.array_equal(g[k].view(np.uint32), w[k].view(np.uint32)), k


def test_l1_selection_rejects_bad_ops():
    from workloads import config, gen
    net = config("tiny_f32_b1")
    params = gen.make_params(net)
    layers = [dict(L) for L in net.layers]
    layers[1]["inp"] = 5                    # reads a tensor not yet written
    with pytest.raises(ctc.CtcError):
        ctc.ctc_select_channels_l1(layers, params)
