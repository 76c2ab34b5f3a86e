"""Architecture descriptors of the five synthetic CNN workloads.

Pure data: each network is a list of layer dicts in execution order, with
the structural facts (groups, the first conv of a residual block, a 1x1
projection shortcut, which tensor a residual add reads) that both the CPU
oracle and the GPU library need.  No carry-through arithmetic lives here:
each side derives the carry-through roles from these facts on its own.

Tensor naming: tensor 0 is the network input; layer i writes tensor i+1.
``inp`` and ``residual`` are tensor ids.

Layer keys
  op        'conv' | 'maxpool' | 'gap' | 'fc'
  conv      c_in, c_out, k, stride, pad, groups, bias, bn, relu,
            residual (tensor id added before the activation, or -1),
            block_first (first conv of a residual block), shortcut
            (1x1 projection shortcut), gamma_small (BN gamma drawn from
            the small range: the conv closes a residual branch)
  maxpool   k, stride, pad
  gap       -
  fc        in_f, out_f, bias, relu, final (the classifier), flatten
            ((C, H, W) of the feature map flattened in NCHW order, or
            None), out_f32 (store the output in fp32 even in fp16 nets)
"""

from __future__ import annotations

import copy


class Net:
    """A network: input shape, layer list, number of classes, dtype."""

    def __init__(self, name, in_shape, layers, classes, dtype, batch):
        self.name = name
        self.in_shape = tuple(in_shape)  # (C, H, W)
        self.layers = layers
        self.classes = classes
        self.dtype = dtype  # 'f32' | 'f16'
        self.batch = batch

    def copy(self, **kw):
        n = copy.deepcopy(self)
        for k, v in kw.items():
            setattr(n, k, v)
        return n

    def shapes(self):
        """(C, H, W) of every tensor, tensor 0 = input."""
        shp = [self.in_shape]
        for L in self.layers:
            c, h, w = shp[L["inp"]]
            if L["op"] == "conv":
                p = (h + 2 * L["pad"] - L["k"]) // L["stride"] + 1
                q = (w + 2 * L["pad"] - L["k"]) // L["stride"] + 1
                shp.append((L["c_out"], p, q))
            elif L["op"] == "maxpool":
                p = (h + 2 * L["pad"] - L["k"]) // L["stride"] + 1
                q = (w + 2 * L["pad"] - L["k"]) // L["stride"] + 1
                shp.append((c, p, q))
            elif L["op"] == "gap":
                shp.append((c, 1, 1))
            elif L["op"] == "fc":
                shp.append((L["out_f"], 1, 1))
            else:
                raise ValueError(L["op"])
        return shp


class _B:
    """Small builder that appends layers and tracks tensor ids."""

    def __init__(self):
        self.layers = []

    def conv(self, inp, c_in, c_out, k, stride, pad, groups=1, bias=False,
             bn=True, relu=True, residual=-1, block_first=False,
             shortcut=False, gamma_small=False):
        self.layers.append(dict(
            op="conv", inp=inp, c_in=c_in, c_out=c_out, k=k, stride=stride,
            pad=pad, groups=groups, bias=bias, bn=bn, relu=relu,
            residual=residual, block_first=block_first, shortcut=shortcut,
            gamma_small=gamma_small))
        return len(self.layers)

    def maxpool(self, inp, k, stride, pad):
        self.layers.append(dict(op="maxpool", inp=inp, k=k, stride=stride,
                                pad=pad))
        return len(self.layers)

    def gap(self, inp):
        self.layers.append(dict(op="gap", inp=inp))
        return len(self.layers)

    def fc(self, inp, in_f, out_f, relu=False, final=False, flatten=None,
           bias=True, out_f32=False):
        self.layers.append(dict(op="fc", inp=inp, in_f=in_f, out_f=out_f,
                                bias=bias, relu=relu, final=final,
                                flatten=flatten, out_f32=out_f32))
        return len(self.layers)


def tiny(batch=1, dtype="f32"):
    """3x32x32 -> conv3x3 3->16 -> conv3x3 16->32 s2 -> GAP -> FC 32->10."""
    b = _B()
    t = b.conv(0, 3, 16, 3, 1, 1, bias=True, bn=False)
    t = b.conv(t, 16, 32, 3, 2, 1, bias=True, bn=False)
    t = b.gap(t)
    b.fc(t, 32, 10, final=True)
    return Net("tiny", (3, 32, 32), b.layers, 10, dtype, batch)


def _basic_block(b, x, c_in, c_out, stride):
    h1 = b.conv(x, c_in, c_out, 3, stride, 1, block_first=True)
    if stride != 1 or c_in != c_out:
        sc = b.conv(x, c_in, c_out, 1, stride, 0, relu=False, shortcut=True)
    else:
        sc = x
    return b.conv(h1, c_out, c_out, 3, 1, 1, residual=sc, gamma_small=True)


def resnet20(batch=128, dtype="f32", classes=10):
    """CIFAR ResNet-20: 3 stages x 3 basic blocks (16/32/64), 1x1
    projection shortcuts where the shape changes."""
    b = _B()
    t = b.conv(0, 3, 16, 3, 1, 1)
    c = 16
    for stage, w in enumerate((16, 32, 64)):
        for i in range(3):
            s = 2 if (stage > 0 and i == 0) else 1
            t = _basic_block(b, t, c, w, s)
            c = w
    t = b.gap(t)
    b.fc(t, 64, classes, final=True)
    return Net("resnet20", (3, 32, 32), b.layers, classes, dtype, batch)


def resnet18(batch=64, dtype="f16", classes=1000, in_hw=224):
    """ImageNet-shaped ResNet-18: conv7x7/2, maxpool 3x3/2, 4 stages x 2
    basic blocks (64/128/256/512)."""
    b = _B()
    t = b.conv(0, 3, 64, 7, 2, 3)
    t = b.maxpool(t, 3, 2, 1)
    c = 64
    for stage, w in enumerate((64, 128, 256, 512)):
        for i in range(2):
            s = 2 if (stage > 0 and i == 0) else 1
            t = _basic_block(b, t, c, w, s)
            c = w
    t = b.gap(t)
    b.fc(t, 512, classes, final=True)
    return Net("resnet18", (3, in_hw, in_hw), b.layers, classes, dtype, batch)


def vgg16(batch=32, dtype="f16", classes=1000, classifier_f32=True,
          in_hw=224, hidden=4096):
    """VGG-16: 13 conv3x3 (+bias, ReLU) with 5 maxpools, then
    FC 25088->4096->4096->classes.  ``classifier_f32`` keeps the two hidden
    FC outputs in fp32 storage (their weights stay in the net dtype)."""
    b = _B()
    t = 0
    c = 3
    for v in (64, 64, "M", 128, 128, "M", 256, 256, 256, "M",
              512, 512, 512, "M", 512, 512, 512, "M"):
        if v == "M":
            t = b.maxpool(t, 2, 2, 0)
        else:
            t = b.conv(t, c, v, 3, 1, 1, bias=True, bn=False)
            c = v
    f32 = classifier_f32 and dtype == "f16"
    s = in_hw // 32
    t = b.fc(t, 512 * s * s, hidden, relu=True, flatten=(512, s, s),
             out_f32=f32)
    t = b.fc(t, hidden, hidden, relu=True, out_f32=f32)
    b.fc(t, hidden, classes, final=True)
    return Net("vgg16", (3, in_hw, in_hw), b.layers, classes, dtype, batch)


MBV2_SETTINGS = ((1, 16, 1, 1), (6, 24, 2, 2), (6, 32, 3, 2), (6, 64, 4, 2),
                 (6, 96, 3, 1), (6, 160, 3, 2), (6, 320, 1, 1))


def mobilenetv2(batch=128, dtype="f16", classes=1000, in_hw=224):
    """MobileNetV2 (width 1.0) with plain ReLU: stem conv3x3/2 32ch, 17
    inverted-residual blocks (expand x t, depthwise 3x3, linear 1x1
    project, residual add when stride 1 and widths match), conv1x1 1280,
    GAP, FC."""
    b = _B()
    t = b.conv(0, 3, 32, 3, 2, 1)
    c = 32
    for (e, w, n, s) in MBV2_SETTINGS:
        for i in range(n):
            stride = s if i == 0 else 1
            res = stride == 1 and c == w
            x = t
            hid = c * e
            if e != 1:
                t = b.conv(t, c, hid, 1, 1, 0, block_first=res)
            t = b.conv(t, hid, hid, 3, stride, 1, groups=hid)
            t = b.conv(t, hid, w, 1, 1, 0, relu=False,
                       residual=x if res else -1, gamma_small=res)
            c = w
    t = b.conv(t, c, 1280, 1, 1, 0)
    t = b.gap(t)
    b.fc(t, 1280, classes, final=True)
    return Net("mobilenetv2", (3, in_hw, in_hw), b.layers, classes, dtype,
               batch)


def by_name(name, **kw):
    return {"tiny": tiny, "resnet20": resnet20, "resnet18": resnet18,
            "vgg16": vgg16, "mobilenetv2": mobilenetv2}[name](**kw)


# The five workload configurations: (label, builder kwargs).
CONFIGS = {
    "tiny_f32_b1": ("tiny", dict(batch=1, dtype="f32")),
    "resnet20_f32_b128": ("resnet20", dict(batch=128, dtype="f32")),
    "resnet18_f16_b64": ("resnet18", dict(batch=64, dtype="f16")),
    "resnet18_f32_b64": ("resnet18", dict(batch=64, dtype="f32")),
    "vgg16_f16_b32": ("vgg16", dict(batch=32, dtype="f16")),
    "mobilenetv2_f16_b128": ("mobilenetv2", dict(batch=128, dtype="f16")),
}


def config(label):
    name, kw = CONFIGS[label]
    return by_name(name, **kw)
