"""CPU oracle for carry-through checksum CNN inference: TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module.  It shares no code with the GPU
library; the two meet only in the seeded generators of ``workloads``.

What it computes, in the order of Sec. II of the paper:

* carry-through construction (Sec. II-A, Eq. 1, Sec. II-B) on canonical
  fp32 parameters, written with numpy: :func:`protect_params`;
* the forward pass, layer by layer through the nested-loop C kernels of
  ``ctc_oracle.c``: :func:`forward_image`, :func:`forward_batch`;
* distribution-based threshold (Sec. II-C): :func:`calibrate`;
* detection and the critical-fault label (Sec. II-B, Sec. III-A):
  :func:`verify`, :func:`is_critical`;
* single-bit faults on stored parameters and activations (Sec. III-A):
  :func:`fault_sites`, :func:`apply_param_fault`.

Readings where the paper is silent are fixed here and listed in the design
notes: the reference value is the calibration mean, the deviation is
two-sided, BN epsilon is 1e-5 and is applied literally (so the "identity"
BN scales the checksum by 1/sqrt(1+eps)), the carry-through filter's bias is
0, a depthwise conv and a 1x1 projection shortcut pass the incoming
checksum through, NaN/Inf propagate and are flagged.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from workloads import gen

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ctc_oracle.c")
_SO = os.path.join(_HERE, "libctc_oracle.so")
BN_EPS = 1e-5

ROLE_SUM, ROLE_ZERO, ROLE_PASS = "SUM", "ZERO", "PASS"


def build():
    """Compile the C oracle (plain gcc, IEEE single precision, no FMA)."""
    tmp = "%s.tmp%d.%d" % (_SO, os.getpid(), threading.get_ident())
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared",
                           "-ffp-contract=off", "-fno-fast-math",
                           "-fexcess-precision=standard", "-o", tmp, _SRC,
                           "-lm"])
    os.replace(tmp, _SO)


_lib_handle = None
_lib_lock = threading.Lock()


def lib():
    global _lib_handle
    if _lib_handle is not None:
        return _lib_handle
    with _lib_lock:
        return _load()


def _load():
    global _lib_handle
    if _lib_handle is None:
        if not os.path.exists(_SO) or (os.path.getmtime(_SO)
                                       < os.path.getmtime(_SRC)):
            build()
        L = ctypes.CDLL(_SO)
        P = ctypes.c_void_p
        i, f = ctypes.c_int, ctypes.c_float
        L.or_conv.argtypes = [P, i, i, i, P, i, i, i, i, i, i, P, P, P, P, P,
                              f, P, i, i, P]
        L.or_conv.restype = None
        L.or_maxpool.argtypes = [P, i, i, i, i, i, i, i, P]
        L.or_gap.argtypes = [P, i, i, i, i, P]
        L.or_fc.argtypes = [P, i, P, i, P, i, i, P]
        L.or_f32_to_f16_array.argtypes = [P, P, ctypes.c_int64]
        L.or_f16_to_f32_array.argtypes = [P, P, ctypes.c_int64]
        L.or_round_f16_array.argtypes = [P, ctypes.c_int64]
        L.or_f16_flip_stored.argtypes = [P, P, P, ctypes.c_int64]
        L.or_f16_flip_stored.restype = ctypes.c_int64
        L.or_f16_widen_bits_array.argtypes = [P, P, ctypes.c_int64]
        L.or_f16_narrow_exact_array.argtypes = [P, P, ctypes.c_int64]
        _lib_handle = L
    return _lib_handle


def _p(a):
    return None if a is None else a.ctypes.data


# ---------------------------------------------------------------- binary16

def f32_to_f16_bits(x):
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.empty(x.shape, dtype=np.uint16)
    lib().or_f32_to_f16_array(_p(x), _p(y), x.size)
    return y


def f16_bits_to_f32(h):
    h = np.ascontiguousarray(h, dtype=np.uint16)
    y = np.empty(h.shape, dtype=np.float32)
    lib().or_f16_to_f32_array(_p(h), _p(y), h.size)
    return y


def f16_bits_to_f32_bits(h):
    """binary32 patterns of binary16 patterns, exact (NaN payloads kept)."""
    h = np.ascontiguousarray(h, dtype=np.uint16)
    y = np.empty(h.shape, dtype=np.uint32)
    lib().or_f16_widen_bits_array(_p(h), _p(y), h.size)
    return y


def f16_pattern_of_stored(a):
    """The binary16 patterns that fp16-stored elements (held as fp32) stand
    for, recovered exactly (NaN payloads included); -1 where an element is
    not a binary16 value."""
    u = np.ascontiguousarray(np.asarray(a, np.float32)).view(np.uint32)
    y = np.empty(u.shape, dtype=np.int32)
    lib().or_f16_narrow_exact_array(_p(u), _p(y), u.size)
    return y


def round_f16(x):
    """fp32 values rounded (RNE) to the nearest binary16 value, as fp32."""
    y = np.array(x, dtype=np.float32, copy=True, order="C")
    lib().or_round_f16_array(_p(y), y.size)
    return y


# ------------------------------------------------- carry-through structure

def has_checksum(net, tensor, protect=True):
    """Does ``tensor`` carry a checksum in its last channel / feature?
    Only the network input does not (Sec. II-A: every conv and every hidden
    FC of a protected net produces one)."""
    return bool(protect) and tensor != 0


def conv_role(L):
    """Role of a conv's last output channel (Sec. II-A and its extension to
    residual and depthwise layers):

    SUM  carry-through filter, 1 at the kernel centre on every input channel;
    ZERO first conv of a residual block: last filter all zero, so the
         checksum entering the block is not counted twice;
    PASS depthwise conv or 1x1 projection shortcut: the last filter copies
         the incoming checksum channel (a depthwise filter cannot sum across
         channels, and the shortcut must deliver the checksum to the add).
    """
    if L["groups"] > 1:
        if L["groups"] != L["c_in"] or L["c_in"] != L["c_out"]:
            raise ValueError("only depthwise grouped convs are supported")
        return ROLE_PASS
    if L["shortcut"]:
        return ROLE_PASS
    if L["block_first"]:
        return ROLE_ZERO
    return ROLE_SUM


def protect_params(net, params, protect=True):
    """Deployed parameters: canonical fp32 params with the carry-through
    construction applied (``protect``), then weights rounded to the net's
    storage type.  Returns a new list; the input is not modified."""
    out = []
    for li, (L, p) in enumerate(zip(net.layers, params)):
        if p is None:
            out.append(None)
            continue
        q = {k: v.astype(np.float32).copy() for k, v in p.items()}
        if protect and L["op"] == "conv":
            _protect_conv(net, L, q)
        elif protect and L["op"] == "fc":
            _protect_fc(net, L, q)
        if net.dtype == "f16":
            q["w"] = round_f16(q["w"])
        out.append(q)
    return out


def _protect_conv(net, L, q):
    w = q["w"]                                # [K][C/g][R][S]
    K, Cg, R, S = w.shape
    r0, s0 = R // 2, S // 2                   # kernel centre
    role = conv_role(L)
    in_ck = has_checksum(net, L["inp"])
    if in_ck and L["groups"] == 1:
        # input-channel level: normal filters ignore the incoming checksum
        w[:K - 1, Cg - 1, :, :] = 0.0
    # output-channel level: the last filter is replaced
    w[K - 1] = 0.0
    if role == ROLE_SUM:
        w[K - 1, :, r0, s0] = 1.0
    elif role == ROLE_PASS:
        if L["groups"] > 1:
            w[K - 1, 0, r0, s0] = 1.0         # depthwise: own channel
        elif in_ck:
            w[K - 1, Cg - 1, r0, s0] = 1.0    # shortcut: checksum channel
    if "b" in q:
        q["b"][K - 1] = 0.0
    if "mean" in q:                           # BN identity entries, Eq. (1)
        q["mean"][K - 1] = 0.0
        q["var"][K - 1] = 1.0
        q["gamma"][K - 1] = 1.0
        q["beta"][K - 1] = 0.0


def channel_groups(net):
    """Tensors whose channel indices are tied: a depthwise conv, a pooling
    layer and a residual add keep channel c of one tensor in channel c of
    another, so pruning a channel of one prunes it in all of them.  Returns
    the group representative of every tensor id (0 = input, i+1 = output
    of layer i)."""
    nt = len(net.layers) + 1
    parent = list(range(nt))

    def find(a):
        while parent[a] != a:
            a = parent[a]
        return a

    def union(a, b):
        a, b = find(a), find(b)
        if a != b:
            parent[max(a, b)] = min(a, b)

    for i, L in enumerate(net.layers):
        if L["op"] == "conv":
            if L["groups"] > 1:
                union(L["inp"], i + 1)
            if L["residual"] >= 0:
                union(i + 1, L["residual"])
        elif L["op"] in ("maxpool", "gap"):
            union(L["inp"], i + 1)
    return [find(t) for t in range(nt)]


def _abs_sums(rows):
    """Sum of |x| along each row, left to right in fp64."""
    a = np.abs(np.asarray(rows, np.float64))
    return np.cumsum(a, axis=1)[:, -1] if a.shape[1] else np.zeros(len(a))


def select_channels_l1(net, params):
    """Output-channel level of Sec. II-A with the paper's choice of channel:
    in every channel group that a conv or hidden FC produces, the channel
    whose combined L1 norm is smallest is the one pruned -- the norm of its
    filters where the group is produced plus the norm of the 2-D slices (or
    FC columns) that read it where the group is consumed; for a group tied
    by residual adds, depthwise convs or pooling, all producers and
    consumers of the group count (the rule for shared residual-stream
    channels).  The chosen channel is swapped with the last one everywhere
    in the group, which leaves the unprotected network's function
    unchanged; the carry-through construction then replaces the last
    channel.  Norms are fp64 sums, each layer's slice in memory order,
    layers added in order; ties go to the lowest channel.  Returns (new
    canonical params, chosen channel of every layer's output group or -1).
    """
    grp = channel_groups(net)
    nl = len(net.layers)
    imp = {}

    def add(g, v):
        imp[g] = imp[g] + v if g in imp else v

    produced = set()
    for i, L in enumerate(net.layers):
        p = params[i]
        if L["op"] == "conv":
            w = p["w"]
            K = w.shape[0]
            add(grp[i + 1], _abs_sums(w.reshape(K, -1)))
            produced.add(grp[i + 1])
            if L["groups"] == 1:
                add(grp[L["inp"]], _abs_sums(
                    w.transpose(1, 0, 2, 3).reshape(w.shape[1], -1)))
        elif L["op"] == "fc":
            w = p["w"]
            if not L["final"]:
                add(grp[i + 1], _abs_sums(w))
                produced.add(grp[i + 1])
            if L["flatten"] is not None:
                C, H, W = L["flatten"]
                blk = w.reshape(w.shape[0], C, H * W).transpose(1, 0, 2)
                add(grp[L["inp"]], _abs_sums(blk.reshape(C, -1)))
            else:
                add(grp[L["inp"]], _abs_sums(w.T))
    chosen_g = {}
    for g in produced:
        if g == grp[0] or g == grp[nl]:
            continue
        chosen_g[g] = int(np.argmin(imp[g]))
    out = [None if p is None else {k: v.copy() for k, v in p.items()}
           for p in params]

    def swap(a, axis, c, last):
        idx = [slice(None)] * a.ndim
        idx[axis] = [c, last]
        jdx = list(idx)
        jdx[axis] = [last, c]
        a[tuple(idx)] = a[tuple(jdx)]

    for i, L in enumerate(net.layers):
        q = out[i]
        if L["op"] == "conv":
            g = grp[i + 1]
            if g in chosen_g and chosen_g[g] != L["c_out"] - 1:
                for k in q:
                    swap(q[k], 0, chosen_g[g], L["c_out"] - 1)
            gi = grp[L["inp"]]
            if L["groups"] == 1 and gi in chosen_g and \
                    chosen_g[gi] != L["c_in"] - 1:
                swap(q["w"], 1, chosen_g[gi], L["c_in"] - 1)
        elif L["op"] == "fc":
            g = grp[i + 1]
            if not L["final"] and g in chosen_g and \
                    chosen_g[g] != L["out_f"] - 1:
                for k in q:
                    swap(q[k], 0, chosen_g[g], L["out_f"] - 1)
            gi = grp[L["inp"]]
            if gi in chosen_g:
                c = chosen_g[gi]
                if L["flatten"] is not None:
                    C, H, W = L["flatten"]
                    if c != C - 1:
                        v = q["w"].reshape(q["w"].shape[0], C, H * W)
                        swap(v, 1, c, C - 1)
                elif c != L["in_f"] - 1:
                    swap(q["w"], 1, c, L["in_f"] - 1)
    chosen = [chosen_g.get(grp[i + 1], -1) for i in range(nl)]
    return out, chosen


def append_network(net, params):
    """The "extra checksum output channels" reading of
    Sec. II-A (append mode): every conv and hidden FC gets one more output
    channel, its width rounded up to whole 16-byte channel vectors (4 in
    fp32, 8 in fp16); the original filters stay at their indices, the added
    channels start as zero filters with identity BN (mean 0, var 1, gamma 1,
    beta 0) and zero bias, and the readers of a widened tensor get zero
    weights for the added channels.  protect_params() on the result then
    makes the last channel the carry-through channel; no channel is pruned.
    Returns (widened net, widened canonical params)."""
    A = 8 if net.dtype == "f16" else 4
    shp = net.shapes()
    width = [shp[0][0]]
    layers = []
    for i, L in enumerate(net.layers):
        M = dict(L)
        ci = width[L["inp"]]
        if L["op"] == "conv":
            M["c_in"] = ci
            if L["groups"] > 1:
                M["groups"] = M["c_out"] = ci
            else:
                M["c_out"] = -(-(L["c_out"] + 1) // A) * A
            width.append(M["c_out"])
        elif L["op"] == "fc":
            if L["flatten"] is not None:
                _, H, W = L["flatten"]
                M["flatten"] = (ci, H, W)
                M["in_f"] = ci * H * W
            else:
                M["in_f"] = ci
            if not L["final"]:
                M["out_f"] = -(-(L["out_f"] + 1) // A) * A
            width.append(M["out_f"])
        else:
            width.append(ci)
        layers.append(M)
    wnet = net.copy(layers=layers)
    out = []
    ident = {"b": 0.0, "mean": 0.0, "var": 1.0, "gamma": 1.0, "beta": 0.0}
    for L, M, p in zip(net.layers, layers, params):
        if p is None:
            out.append(None)
            continue
        q = {}
        w = p["w"]
        if L["op"] == "conv":
            K, Cg = w.shape[0], w.shape[1]
            w2 = np.zeros((M["c_out"], M["c_in"] // M["groups"]) + w.shape[2:],
                          np.float32)
            w2[:K, :Cg] = w
        else:
            # NCHW flatten: the added channels' features come after the
            # original ones, so every original feature keeps its index
            w2 = np.zeros((M["out_f"], M["in_f"]), np.float32)
            w2[:w.shape[0], :w.shape[1]] = w
        q["w"] = w2
        n_out = w2.shape[0]
        for k, v in p.items():
            if k == "w":
                continue
            a = np.full(n_out, ident[k], np.float32)
            a[:v.size] = v
            q[k] = a
        out.append(q)
    return wnet, out


def checksum_features(net, L):
    """Indices of the input features of an FC layer that hold checksum
    values: after GAP or another FC the last feature; after a flatten of a
    (C, H, W) map in NCHW order, the H*W features of channel C-1."""
    if L["flatten"] is not None:
        C, H, W = L["flatten"]
        return np.arange((C - 1) * H * W, C * H * W)
    return np.array([L["in_f"] - 1])


def _protect_fc(net, L, q):
    w = q["w"]
    ck = checksum_features(net, L) if has_checksum(net, L["inp"]) else []
    if L["final"]:
        # accumulated-checksum neuron (Sec. II-B): one more output with
        # weight 1 on every input and bias 0; the logits ignore the
        # incoming checksum feature(s)
        w[:, ck] = 0.0
        q["w"] = np.concatenate([w, np.ones((1, w.shape[1]), np.float32)])
        if "b" in q:
            q["b"] = np.concatenate([q["b"], np.zeros(1, np.float32)])
    else:
        # hidden FC: same scheme as a conv, last neuron sums every input
        w[:-1, ck] = 0.0
        w[-1, :] = 1.0
        if "b" in q:
            q["b"][-1] = 0.0


# ----------------------------------------------------------------- forward

def stored_f32(net, tensor):
    """Is a tensor stored in fp32 (True) or in the net dtype?"""
    if net.dtype == "f32":
        return True
    if tensor == 0:
        return False
    L = net.layers[tensor - 1]
    return L["op"] == "fc" and (L["final"] or L["out_f32"])


def _store(net, tensor, a):
    if not stored_f32(net, tensor):
        lib().or_round_f16_array(_p(a), a.size)
    return a


def _flip(a, flat_index, bit, f32):
    """XOR one bit of the stored representation of a[flat_index] in place
    (Sec. III-A's single-bit fault).  ``flat_index`` and ``bit`` may be
    arrays (one flip per entry).  fp32 elements: bit of the binary32
    pattern.  fp16-stored elements (held here as the fp32 value of their
    binary16 pattern): the pattern is recovered exactly, bit ``bit`` of it
    is XOR-ed and the result widened exactly, all on integer patterns, so
    NaN payloads survive and flipping twice restores every bit."""
    if a.dtype != np.float32 or not a.flags.c_contiguous:
        raise ValueError("faults apply to contiguous fp32 storage")
    u = a.reshape(-1).view(np.uint32)
    idx = np.ascontiguousarray(np.atleast_1d(flat_index), dtype=np.int64)
    bits = np.ascontiguousarray(np.broadcast_to(np.asarray(bit, np.int32),
                                                idx.shape))
    if f32:
        if np.any((bits < 0) | (bits > 31)):
            raise ValueError("fp32 fault bit out of range")
        np.bitwise_xor.at(u, idx, np.left_shift(np.uint32(1),
                                                bits.astype(np.uint32)))
        return
    bad = lib().or_f16_flip_stored(_p(u), _p(idx), _p(bits), idx.size)
    if bad:
        raise ValueError("%d fault target(s) hold no binary16 value or the "
                         "bit is out of range" % bad)


def forward_image(net, dp, x, protect=True, start=0, acts=None,
                  act_faults=(), keep=False):
    """Forward one image (x: (C, H, W) fp32).

    ``acts``: tensors of a previous run to start from (with ``start`` the
    first layer to recompute).  ``act_faults``: iterable of (tensor, flat
    index, bit) flipped right after the tensor is produced (the stored
    value).  Returns the final FC output (fp32, classes + protect values),
    or the list of all tensors when ``keep``.
    """
    L_ = lib()
    shp = net.shapes()
    T = [None] * (len(net.layers) + 1) if acts is None else list(acts)
    faults = {}
    for (t, idx, bit) in act_faults:
        faults.setdefault(t, []).append((idx, bit))

    def post(t, a):
        for idx, bit in faults.get(t, ()):
            _flip(a, idx, bit, stored_f32(net, t))
        return a

    if start == 0:
        T[0] = post(0, _store(net, 0, np.array(x, np.float32, copy=True)))
    else:
        for t in faults:
            if t < start + 1:
                raise ValueError("activation fault before the restart point")
    r16 = 1 if net.dtype == "f16" else 0
    for i in range(start, len(net.layers)):
        L = net.layers[i]
        p = dp[i]
        xin = T[L["inp"]]
        C, H, W = shp[L["inp"]]
        oc, oh, ow = shp[i + 1]
        y = np.empty((oc, oh, ow), np.float32)
        if L["op"] == "conv":
            res = T[L["residual"]] if L["residual"] >= 0 else None
            bn = "mean" in p
            L_.or_conv(_p(xin), C, H, W, _p(p["w"]), oc, L["k"], L["k"],
                       L["stride"], L["pad"], L["groups"], _p(p.get("b")),
                       _p(p["mean"]) if bn else None,
                       _p(p["var"]) if bn else None,
                       _p(p["gamma"]) if bn else None,
                       _p(p["beta"]) if bn else None, BN_EPS, _p(res),
                       int(L["relu"]), r16, _p(y))
        elif L["op"] == "maxpool":
            L_.or_maxpool(_p(xin), C, H, W, L["k"], L["stride"], L["pad"],
                          r16, _p(y))
        elif L["op"] == "gap":
            L_.or_gap(_p(xin), C, H, W, r16, _p(y))
        elif L["op"] == "fc":
            xin = np.ascontiguousarray(xin.reshape(-1))
            n_out = p["w"].shape[0]
            y = np.empty((n_out, 1, 1), np.float32)
            L_.or_fc(_p(xin), xin.size, _p(p["w"]), n_out, _p(p.get("b")),
                     int(L["relu"]), 0 if stored_f32(net, i + 1) else r16,
                     _p(y))
        T[i + 1] = post(i + 1, y)
    if keep:
        return T
    return T[-1].reshape(-1).copy()


def forward_batch(net, dp, X, protect=True, threads=None):
    """Forward a batch (N, C, H, W) with one thread per image in flight.
    Returns (N, classes + protect) fp32."""
    threads = threads or os.cpu_count() or 1
    with ThreadPoolExecutor(max_workers=threads) as ex:
        outs = list(ex.map(lambda xi: forward_image(net, dp, xi, protect), X))
    return np.stack(outs)


# ------------------------------------------------- detection and threshold

def calibrate(S, alpha):
    """Distribution-based threshold (Sec. II-C): ref = mean of fault-free S
    (fp64), dev_i = |S_i - ref|, tau = the k-th smallest deviation with
    k = N - ceil(alpha N) + 1, so that fewer than alpha*N fault-free
    inferences exceed tau."""
    S = np.asarray(S, np.float64)
    n = S.size
    if n == 0:
        raise ValueError("empty calibration set")
    ref = float(np.sum(S) / n)
    dev = np.sort(np.abs(S - ref))
    k = n - int(np.ceil(alpha * n - 1e-12)) + 1
    k = min(max(k, 1), n)
    return ref, float(dev[k - 1])


def threshold_at_ref(S, ref, alpha):
    """FI-based threshold (Sec. II-C): the same order statistic as the
    distribution-based one, taken over the accumulated-checksum values of
    the non-critical faulty inferences of a campaign on training inputs,
    with the fault-free reference ``ref``: tau = k-th smallest |S_i - ref|,
    k = N - ceil(alpha N) + 1, so that fewer than alpha*N of those
    non-critical faults would be flagged.  A NaN deviation ranks above
    every number."""
    S = np.asarray(S, np.float64)
    n = S.size
    if n == 0:
        raise ValueError("empty sample")
    dev = np.abs(S - float(ref))
    dev[np.isnan(dev)] = np.inf
    dev = np.sort(dev)
    k = n - int(np.ceil(alpha * n - 1e-12)) + 1
    k = min(max(k, 1), n)
    return float(dev[k - 1])


def detection_rates(flags, critical):
    """Sec. III-A metrics: TPR = flagged critical / critical, FPR = flagged
    non-critical / non-critical, Youden's J = TPR - FPR (Sec. III-A)."""
    flags = np.asarray(flags, bool)
    critical = np.asarray(critical, bool)
    nc, nn = int(critical.sum()), int((~critical).sum())
    tpr = float((flags & critical).sum() / nc) if nc else float("nan")
    fpr = float((flags & ~critical).sum() / nn) if nn else float("nan")
    return tpr, fpr, tpr - fpr


def verify(S, ref, tau):
    """Detection flag (Sec. II-B): deviation from the reference beyond tau.
    Taken in fp32 (ref and tau rounded to fp32), so NaN and Inf are
    flagged: flag = not(|S - ref| <= tau)."""
    S = np.asarray(S, np.float32)
    dev = np.abs(S - np.float32(ref))
    return ~(dev <= np.float32(tau))


def top1(logits):
    """Index of the largest logit, lowest index on ties; -1 if any NaN."""
    logits = np.asarray(logits)
    if np.isnan(logits).any():
        return -1
    return int(np.argmax(logits))


def is_critical(logits, golden_logits):
    """A fault is critical when it changes the golden top-1 class
    (Sec. II-B, Sec. III-A); a NaN logit counts as a change."""
    t = top1(logits)
    return t < 0 or t != top1(golden_logits)


# ------------------------------------------------------------------ faults

def fault_sites(net, dp, protect=True):
    """All single-bit fault sites: (kind, layer-or-tensor, elements, bits).

    Parameters as deployed: weights in the net dtype (16 bits in fp16
    nets), biases and BN parameters 32 bits.  Activations: every stored
    tensor (the layer boundaries), keyed by tensor id."""
    sites = []
    wbits = 16 if net.dtype == "f16" else 32
    for i, (L, p) in enumerate(zip(net.layers, dp)):
        if p is None:
            continue
        sites.append((gen.SITE_WEIGHT, i, p["w"].size, wbits))
        for key, kind in (("b", gen.SITE_BIAS), ("mean", gen.SITE_BN_MEAN),
                          ("var", gen.SITE_BN_VAR),
                          ("gamma", gen.SITE_BN_GAMMA),
                          ("beta", gen.SITE_BN_BETA)):
            if key in p:
                sites.append((kind, i, p[key].size, 32))
    shp = net.shapes()
    for t, s in enumerate(shp):
        n = int(np.prod(s))
        if t == len(shp) - 1:
            n = dp[-1]["w"].shape[0]
        sites.append((gen.SITE_ACT, t, n, 32 if stored_f32(net, t) else 16))
    return sites


_PKEY = {gen.SITE_WEIGHT: "w", gen.SITE_BIAS: "b", gen.SITE_BN_MEAN: "mean",
         gen.SITE_BN_VAR: "var", gen.SITE_BN_GAMMA: "gamma",
         gen.SITE_BN_BETA: "beta"}


def apply_param_fault(net, dp, site, layer, index, bit):
    """Flip one bit of a deployed parameter in place (call again to undo:
    XOR is an involution)."""
    key = _PKEY[int(site)]
    f32 = key != "w" or net.dtype == "f32"
    _flip(dp[int(layer)][key], int(index), int(bit), f32)
