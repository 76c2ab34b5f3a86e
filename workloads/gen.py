"""Seeded synthetic inputs, canonical parameters and fault lists.

Everything is drawn from numpy ``Generator(PCG64)`` with one base seed per
workload and separate streams per purpose, so that the CPU oracle and the
GPU library consume identical data.  Canonical parameters are fp32 in
PyTorch layout (conv weight [K][C/g][kh][kw], FC weight [out][in]).

Distributions (synthetic stand-ins for trained CIFAR / ImageNet models):
  input            x ~ N(0, 1), NCHW fp32
  conv / FC weight He-normal N(0, 2/fan_in), fan_in = (C/g)*kh*kw
                   (the classifier uses N(0, 1/fan_in))
  bias             U(-1/sqrt(fan_in), 1/sqrt(fan_in)) where no BN follows
  BN               gamma U(0.5, 1.5) (U(0.2, 0.5) on a conv that closes a
                   residual branch), beta N(0, 0.1^2); running mean and
                   variance are the per-channel statistics of the pre-BN
                   activation over 4 seeded synthetic images (the plain
                   network run in float64 with torch on the CPU), as a
                   trained network's running statistics would be.  Random
                   statistics that do not match the activations let the
                   activations of deep nets grow without bound.

Nothing here implements any part of the detection method.
"""

from __future__ import annotations

import math

import numpy as np

# Purpose streams
S_WEIGHTS, S_EVAL, S_CALIB, S_FAULTS, S_BNSTAT = 0, 1, 2, 3, 4
BN_STAT_IMAGES = 4

BASE_SEEDS = {"tiny": 1000, "resnet20": 1001, "resnet18": 1002,
              "vgg16": 1003, "mobilenetv2": 1004}


def rng(base_seed, stream):
    return np.random.Generator(np.random.PCG64([int(base_seed), int(stream)]))


def make_params(net, seed=None):
    """Canonical fp32 parameters, one dict per layer (None for pool/GAP).

    conv: {'w', 'b'?, 'mean'?, 'var'?, 'gamma'?, 'beta'?}; fc: {'w', 'b'?}.
    """
    seed = BASE_SEEDS[net.name] if seed is None else seed
    g = rng(seed, S_WEIGHTS)
    out = []
    for L in net.layers:
        if L["op"] == "conv":
            k, cg = L["c_out"], L["c_in"] // L["groups"]
            fan_in = cg * L["k"] * L["k"]
            p = {"w": (g.standard_normal((k, cg, L["k"], L["k"]),
                                         dtype=np.float32)
                       * np.float32(np.sqrt(2.0 / fan_in)))}
            if L["bias"]:
                bnd = 1.0 / np.sqrt(fan_in)
                p["b"] = g.uniform(-bnd, bnd, k).astype(np.float32)
            if L["bn"]:
                p["mean"] = np.zeros(k, np.float32)   # set by _bn_statistics
                p["var"] = np.ones(k, np.float32)
                lo, hi = (0.2, 0.5) if L["gamma_small"] else (0.5, 1.5)
                p["gamma"] = g.uniform(lo, hi, k).astype(np.float32)
                p["beta"] = (0.1 * g.standard_normal(k)).astype(np.float32)
            out.append(p)
        elif L["op"] == "fc":
            fan_in = L["in_f"]
            gain = 1.0 if L["final"] else 2.0
            p = {"w": (g.standard_normal((L["out_f"], L["in_f"]),
                                         dtype=np.float32)
                       * np.float32(np.sqrt(gain / fan_in)))}
            if L["bias"]:
                bnd = 1.0 / np.sqrt(fan_in)
                p["b"] = g.uniform(-bnd, bnd, L["out_f"]).astype(np.float32)
            out.append(p)
        else:
            out.append(None)
    if any(L["op"] == "conv" and L["bn"] for L in net.layers):
        _bn_statistics(net, out, seed)
    return out


def _bn_statistics(net, params, seed):
    """Set every BN's running mean/var to the statistics of its input over
    a few seeded images, running the plain (unprotected) network layer by
    layer in float64."""
    import torch
    import torch.nn.functional as F
    x = make_inputs(net, BN_STAT_IMAGES, stream=S_BNSTAT, seed=seed)
    T = [torch.from_numpy(x.astype(np.float64))]
    for L, p in zip(net.layers, params):
        a = T[L["inp"]]
        if L["op"] == "conv":
            y = F.conv2d(a, torch.from_numpy(p["w"].astype(np.float64)),
                         None if "b" not in p else
                         torch.from_numpy(p["b"].astype(np.float64)),
                         stride=L["stride"], padding=L["pad"],
                         groups=L["groups"])
            if L["bn"]:
                m = y.mean(dim=(0, 2, 3))
                v = y.var(dim=(0, 2, 3), unbiased=False)
                p["mean"] = m.numpy().astype(np.float32)
                p["var"] = v.numpy().astype(np.float32)
                mm = torch.from_numpy(p["mean"].astype(np.float64))
                vv = torch.from_numpy(p["var"].astype(np.float64))
                gg = torch.from_numpy(p["gamma"].astype(np.float64))
                bb = torch.from_numpy(p["beta"].astype(np.float64))
                y = ((y - mm[None, :, None, None])
                     / torch.sqrt(vv[None, :, None, None] + 1e-5)
                     * gg[None, :, None, None] + bb[None, :, None, None])
            if L["residual"] >= 0:
                y = y + T[L["residual"]]
            if L["relu"]:
                y = torch.relu(y)
        elif L["op"] == "maxpool":
            y = F.max_pool2d(a, L["k"], L["stride"], L["pad"])
        elif L["op"] == "gap":
            y = a.mean(dim=(2, 3), keepdim=True)
        else:
            break                       # nothing after the first FC has BN
        T.append(y)


def make_inputs(net, n, stream=S_EVAL, seed=None, offset=0):
    """n images ~ N(0, 1), NCHW fp32.  ``offset`` skips images so that a
    large set can be produced in pieces with identical values."""
    return next(input_chunks(net, n, max(n, 1), stream, seed, offset))


def input_chunks(net, n, chunk, stream=S_EVAL, seed=None, offset=0):
    """The images of make_inputs(net, n, stream, seed, offset) in pieces of
    ``chunk`` images, drawn from one generator (linear cost for a large
    set; the skipped prefix is drawn in bounded pieces)."""
    seed = BASE_SEEDS[net.name] if seed is None else seed
    g = rng(seed, stream)
    per = int(np.prod(net.in_shape))
    left = offset * per
    while left:
        k = min(left, 1 << 24)
        g.standard_normal(k, dtype=np.float32)
        left -= k
    if n == 0:
        yield np.empty((0,) + net.in_shape, np.float32)
        return
    for s in range(0, n, chunk):
        yield g.standard_normal((min(chunk, n - s),) + net.in_shape,
                                dtype=np.float32)


def leveugle_sample_size(population, e=0.01, t=1.96, p=0.5):
    """Statistical fault-injection sample size (Leveugle et al., DATE 2009):
    n = N / (1 + e^2 (N - 1) / (t^2 p (1 - p))), rounded up; 9604 for a
    large population at 95% confidence (t = 1.96) and a 1% margin."""
    N = float(population)
    return int(math.ceil(N / (1.0 + e * e * (N - 1.0) / (t * t * p * (1.0 - p)))))


def sample_faults(sites, n, seed, stream=S_FAULTS, n_images=1):
    """Uniform single-bit faults over a list of sites.

    ``sites`` is a list of (site_kind, layer, n_elements, n_bits); a fault
    is drawn with probability proportional to n_elements*n_bits.  Returns a
    structured array with fields site, layer, index, bit, image.
    """
    g = rng(seed, stream)
    w = np.array([s[2] * s[3] for s in sites], dtype=np.float64)
    cum = np.cumsum(w)
    u = g.uniform(0, cum[-1], n)
    which = np.searchsorted(cum, u, side="right")
    out = np.zeros(n, dtype=FAULT_DTYPE)
    for i, si in enumerate(which):
        kind, layer, ne, nb = sites[si]
        out[i] = (kind, layer, g.integers(0, ne), g.integers(0, nb),
                  g.integers(0, n_images))
    return out


def enumerate_faults(sites, image=0):
    """Every (element, bit) of every site: the exhaustive single-bit sweep."""
    total = sum(s[2] * s[3] for s in sites)
    out = np.zeros(total, dtype=FAULT_DTYPE)
    o = 0
    for kind, layer, ne, nb in sites:
        cnt = ne * nb
        idx = np.arange(cnt, dtype=np.int64)
        out["site"][o:o + cnt] = kind
        out["layer"][o:o + cnt] = layer
        out["index"][o:o + cnt] = idx // nb
        out["bit"][o:o + cnt] = idx % nb
        out["image"][o:o + cnt] = image
        o += cnt
    return out


# Fault site kinds (shared numbering with the C interface)
SITE_WEIGHT, SITE_BIAS, SITE_BN_MEAN, SITE_BN_VAR, SITE_BN_GAMMA, \
    SITE_BN_BETA, SITE_ACT = range(7)

FAULT_DTYPE = np.dtype([("site", np.int32), ("layer", np.int32),
                        ("index", np.int64), ("bit", np.int32),
                        ("image", np.int32)])
