"""Host logic of bench.py (no GPU): the algorithmic work and bytes it
divides by measured time, the crediting of ops that run inside another
op's kernel, and the single-GPU refusal; the seeded input sets that bench
and the campaigns draw in pieces."""

import math
import os
import subprocess
import sys

import numpy as np
import pytest

import bench
from workloads import config, gen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_layer_flops_and_bytes_closed_forms():
    net = config("vgg16_f16_b32")
    shp = net.shapes()
    lf, lb = bench.layer_flops(net), bench.layer_bytes(net)
    # conv3_2: 256 -> 256 channels, 3x3, on 56x56
    i = next(k for k, L in enumerate(net.layers)
             if L["op"] == "conv" and L["c_in"] == 256 and shp[k + 1][1] == 56)
    assert lf[i] == 2.0 * 56 * 56 * 256 * 256 * 9
    io = 2 * 56 * 56 * 256 * 2                     # fp16 in + out per image
    assert lb[i] == io + 256 * 256 * 9 * 2 / net.batch
    # the final FC carries the accumulated-checksum neuron
    fc = len(net.layers) - 1
    L = net.layers[fc]
    assert lf[fc] == 2.0 * (L["out_f"] + 1) * L["in_f"]
    # pools and GAP do no FLOPs but move bytes
    pools = [k for k, L in enumerate(net.layers) if L["op"] == "maxpool"]
    assert pools and all(lf[k] == 0.0 and lb[k] > 0 for k in pools)


def test_fused_ops_are_credited_to_the_launching_kernel():
    """A pool run in the conv's epilogue: its FLOPs and bytes go to the
    conv, less the write and the read of the tensor between them."""
    net = config("vgg16_f16_b32")
    shp = net.shapes()
    lf, lb = bench.layer_flops(net), bench.layer_bytes(net)
    i = next(k for k, L in enumerate(net.layers) if L["op"] == "maxpool")
    names = ["k%d" % k for k in range(len(net.layers))]
    names[i] = names[i - 1]                        # the pool inside the conv
    launches = [0 if k == i else 1 for k in range(len(net.layers))]
    f0, b0 = lf[i - 1] + lf[i], lb[i - 1] + lb[i]
    merged = bench.merge_fused(net, names, launches, lf, lb)
    assert merged == {i}
    assert lf[i] == lb[i] == 0.0 and lf[i - 1] == f0
    assert lb[i - 1] == b0 - 2.0 * math.prod(shp[i]) * 2


def test_traffic_accounting_of_fused_inverted_residual_blocks():
    """A fused expand -> depthwise -> project block is one launch whose
    algorithmic bytes are its input, output and weights: the 6x-wide
    expanded and depthwise tensors are not counted."""
    net = config("mobilenetv2_f16_b128")
    shp = net.shapes()
    B = net.batch
    n = len(net.layers)
    names = ["k%d" % k for k in range(n)]
    # ops 9-11: 24 -> 144 -> 32, stride 2 (56x56 -> 28x28), as one kernel
    for k in (9, 10, 11):
        names[k] = "conv_ir<2, 32, 1, 32>"
    alg = bench.alg_bytes_by_kernel(net, names)
    b, launches = alg["conv_ir<2, 32, 1, 32>"]
    assert launches == 1
    lb = bench.layer_bytes(net)
    inner = 2 * 2 * (math.prod(shp[10]) + math.prod(shp[11]))   # fp16 w + r
    assert b == pytest.approx((lb[9] + lb[10] + lb[11] - inner) * B)
    x_in, y_out = math.prod(shp[9]) * 2, math.prod(shp[12]) * 2
    weights = sum(lb[k] - 2 * (math.prod(shp[net.layers[k]["inp"]]) +
                               math.prod(shp[k + 1]))
                  for k in (9, 10, 11))
    assert b == pytest.approx((x_in + y_out + weights) * B)


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"),
                        "--gpus", "2"], capture_output=True, text=True,
                       cwd=ROOT, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_input_pieces_equal_the_whole_set():
    """Images drawn piecewise (with and without a skipped prefix) are the
    same images as one make_inputs call over the whole range."""
    net = config("tiny_f32_b1")
    whole = gen.make_inputs(net, 45)
    assert np.array_equal(gen.make_inputs(net, 38, offset=7), whole[7:])
    for chunk in (1, 8, 38, 100):
        parts = list(gen.input_chunks(net, 38, chunk, offset=7))
        assert [len(p) for p in parts][:-1] == [chunk] * (len(parts) - 1)
        assert np.array_equal(np.concatenate(parts), whole[7:])
    assert gen.make_inputs(net, 0).shape == (0,) + net.in_shape
