"""ctypes binding of libctc.so: the C ABI declared in include/ctc.h.

Argument marshalling only: every step of the inference path runs in the
library's HIP kernels and C++ host runtime.  Device buffers are passed as
torch tensors (``data_ptr()``), host arrays as numpy arrays, streams as
``torch.cuda.Stream`` / raw handles.  Functions keep the C names; a failed
call raises :class:`CtcError` with the library's message.  If the library
is missing the import fails: there is no fallback path.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np
# torch ships its own HIP runtime (SONAME libamdhip64.so.7).  Loading it
# first makes libctc.so bind to that same runtime instead of pulling in a
# second copy from /opt/rocm: device pointers and streams come from torch,
# so both sides must share one runtime.
import torch  # noqa: F401  (import order matters, see above)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libctc.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        "libctc.so is not built (%s); run __graft_entry__.build() or "
        "python paper_2609_16742_amd/build.py" % LIB_PATH)

_lib = ctypes.CDLL(LIB_PATH)

CTC_OK, CTC_ERR_ARG, CTC_ERR_UNSUPPORTED, CTC_ERR_DEVICE, \
    CTC_ERR_WORKSPACE, CTC_ERR_STATE = 0, -1, -2, -3, -4, -5
CTC_F32, CTC_F16 = 0, 1
CTC_ROLE_NONE, CTC_ROLE_SUM, CTC_ROLE_ZERO, CTC_ROLE_PASS = 0, 1, 2, 3
CTC_OP_CONV, CTC_OP_MAXPOOL, CTC_OP_GAP, CTC_OP_FC = 1, 2, 3, 4
CTC_REEXEC_NONE, CTC_REEXEC_SYNC, CTC_REEXEC_DEFERRED = 0, 1, 2
CTC_SITE_WEIGHT, CTC_SITE_BIAS, CTC_SITE_BN_MEAN, CTC_SITE_BN_VAR, \
    CTC_SITE_BN_GAMMA, CTC_SITE_BN_BETA, CTC_SITE_ACT = range(7)
DTYPES = {"f32": CTC_F32, "f16": CTC_F16}

CTC_PROTECT_NONE, CTC_PROTECT_REPLACE, CTC_PROTECT_APPEND = 0, 1, 2
CTC_FUSE_IR, CTC_FUSE_BLOCK, CTC_FUSE_STEM, CTC_FUSE_POOL = 1, 2, 4, 8

EXPORTS = ["ctc_build_filters", "ctc_build_fc", "ctc_threshold_from_samples",
           "ctc_threshold_at_ref", "ctc_net_fault_sites",
           "ctc_select_channels_l1", "ctc_net_set_fusion",
           "ctc_conv2d_forward", "ctc_conv2d_workspace_bytes",
           "ctc_conv2d_kernel_name", "ctc_conv2d_forward_noalloc",
           "ctc_verify", "ctc_net_create",
           "ctc_net_workspace_bytes", "ctc_net_bind", "ctc_net_set_threshold",
           "ctc_network_forward", "ctc_network_flush", "ctc_inject_bitflip",
           "ctc_clear_faults", "ctc_net_tensor", "ctc_net_weight_address",
           "ctc_net_role",
           "ctc_net_profile", "ctc_net_profile_read", "ctc_net_op_kernel",
           "ctc_graph_create", "ctc_graph_launch", "ctc_graph_destroy",
           "ctc_net_destroy", "ctc_last_error", "ctc_abi_version"]


class ctc_layer_desc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("c_in", "c_out", "kh", "kw", "stride", "pad", "groups",
                 "in_has_ck", "role")]


class ctc_op(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("kind", "input", "residual", "c_in", "c_out", "k", "stride",
                 "pad", "groups", "has_bias", "has_bn", "relu", "block_first",
                 "shortcut", "final_fc", "flatten_c", "flatten_h",
                 "flatten_w", "out_f32")]


class ctc_fault(ctypes.Structure):
    _fields_ = [("site", ctypes.c_int32), ("layer", ctypes.c_int32),
                ("index", ctypes.c_int64), ("bit", ctypes.c_int32),
                ("image", ctypes.c_int32)]


assert ctypes.sizeof(ctc_fault) == 24


class ctc_site_info(ctypes.Structure):
    _fields_ = [("site", ctypes.c_int32), ("layer", ctypes.c_int32),
                ("elements", ctypes.c_int64), ("bits", ctypes.c_int32),
                ("pad", ctypes.c_int32)]


assert ctypes.sizeof(ctc_site_info) == 24


class CtcError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("ctc status %d: %s" % (status, msg))
        self.status = status


_P, _I32, _I64, _F32, _F64 = (ctypes.c_void_p, ctypes.c_int32,
                              ctypes.c_int64, ctypes.c_float, ctypes.c_double)
_SZ = ctypes.c_size_t


def _sig(name, args, res=ctypes.c_int):
    f = getattr(_lib, name)
    f.argtypes = args
    f.restype = res
    return f


_sig("ctc_build_filters", [ctypes.POINTER(ctc_layer_desc)] + [_P] * 6)
_sig("ctc_build_fc", [_I32, _I32, _I32, _I32, _I32, _P, _P, _P, _P])
_sig("ctc_threshold_from_samples", [_P, _I64, _F64, _P, _P])
_sig("ctc_threshold_at_ref", [_P, _I64, _F64, _F64, _P])
_sig("ctc_select_channels_l1", [ctypes.POINTER(ctc_op), _I32, _P, _P])
_sig("ctc_conv2d_forward", [ctypes.POINTER(ctc_layer_desc), _I32, _I32, _I32,
                            _I32, _P, _P, _P, _P, _P, _I32, _I32, _P, _P, _SZ,
                            _P])
_sig("ctc_conv2d_workspace_bytes", [ctypes.POINTER(ctc_layer_desc), _I32, _I32,
                                    _I32, _I32, _I32, ctypes.POINTER(_SZ)])
_sig("ctc_conv2d_forward_noalloc", [ctypes.POINTER(ctc_layer_desc), _I32, _I32,
                                    _I32, _I32, _P, _P, _P, _P, _P, _I32, _I32,
                                    _P, _P])
_sig("ctc_conv2d_kernel_name", [ctypes.POINTER(ctc_layer_desc), _I32, _I32, _I32,
                                _I32, _I32, ctypes.c_char_p, _I32])
_sig("ctc_verify", [_P, _I32, _I32, _F32, _F32, _P, _P, _P, _P])
_sig("ctc_net_create", [ctypes.POINTER(ctc_op), _I32, _I32, _I32, _I32, _I32,
                        _I32, _I32, ctypes.POINTER(_P)])
_sig("ctc_net_workspace_bytes", [_P, _I32, ctypes.POINTER(_SZ)])
_sig("ctc_net_bind", [_P, ctypes.POINTER(_P), _P, _SZ, _I32, _P])
_sig("ctc_net_set_threshold", [_P, _F32, _F32])
_sig("ctc_net_set_fusion", [_P, _I32])
_sig("ctc_network_forward", [_P, _I32, _P, _P, _P, _I32, _P])
_sig("ctc_network_flush", [_P, _P])
_sig("ctc_inject_bitflip", [_P, ctypes.POINTER(ctc_fault), _I32, _P])
_sig("ctc_clear_faults", [_P, _P])
_sig("ctc_net_tensor", [_P, _I32, ctypes.POINTER(_P)] +
     [ctypes.POINTER(_I32)] * 4)
_sig("ctc_net_weight_address", [_P, _I32, _I64, ctypes.POINTER(_P),
                                ctypes.POINTER(_I32)])
_sig("ctc_net_role", [_P, _I32], _I32)
_sig("ctc_net_fault_sites", [_P, _I32, _P, _I32, ctypes.POINTER(_I32)])
_sig("ctc_net_profile", [_P, _I32])
_sig("ctc_net_profile_read", [_P, _P, _P])
_sig("ctc_net_op_kernel", [_P, _I32, _I32, ctypes.c_char_p, _I32])
_sig("ctc_graph_create", [_P, _I32, _I32, _P, _P, _P, ctypes.POINTER(_P)])
_sig("ctc_graph_launch", [_P, _I32, ctypes.POINTER(_I32), _P])
_sig("ctc_graph_destroy", [_P], None)
_sig("ctc_net_destroy", [_P], None)
_sig("ctc_last_error", [], ctypes.c_char_p)
_sig("ctc_abi_version", [], _I32)


def ctc_last_error():
    return _lib.ctc_last_error().decode()


def ctc_abi_version():
    return _lib.ctc_abi_version()


def _check(st):
    if st != CTC_OK:
        raise CtcError(st, ctc_last_error())


def _ptr(a):
    """Address of a torch tensor, numpy array, raw int or None."""
    if a is None:
        return None
    if isinstance(a, int):
        return a
    if isinstance(a, np.ndarray):
        if not a.flags.c_contiguous:
            raise ValueError("array must be C-contiguous")
        return a.ctypes.data
    if hasattr(a, "data_ptr"):
        if not a.is_contiguous():
            raise ValueError("tensor must be contiguous")
        return a.data_ptr()
    raise TypeError("cannot take the address of %r" % type(a))


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _f32(a, name):
    if a is None:
        return None
    if not (isinstance(a, np.ndarray) and a.dtype == np.float32
            and a.flags.c_contiguous):
        raise TypeError("%s must be a C-contiguous float32 numpy array" % name)
    return a


def layer_desc(c_in, c_out, kh, kw, stride, pad, groups, in_has_ck, role):
    return ctc_layer_desc(c_in, c_out, kh, kw, stride, pad, groups,
                          in_has_ck, role)


# ----------------------------------------------------------- host builders

def ctc_build_filters(desc, w, bias=None, bn_mean=None, bn_var=None,
                      bn_gamma=None, bn_beta=None):
    """In place on float32 numpy arrays (canonical layout)."""
    arrs = [_f32(w, "w"), _f32(bias, "bias"), _f32(bn_mean, "bn_mean"),
            _f32(bn_var, "bn_var"), _f32(bn_gamma, "bn_gamma"),
            _f32(bn_beta, "bn_beta")]
    _check(_lib.ctc_build_filters(ctypes.byref(desc), *[_ptr(a)
                                                         for a in arrs]))


def ctc_build_fc(in_f, out_f, ck_first, ck_count, is_final, w_in, b_in,
                 w_out, b_out):
    _check(_lib.ctc_build_fc(in_f, out_f, ck_first, ck_count, is_final,
                             _ptr(_f32(w_in, "w_in")),
                             _ptr(_f32(b_in, "b_in")),
                             _ptr(_f32(w_out, "w_out")),
                             _ptr(_f32(b_out, "b_out"))))


def ctc_threshold_from_samples(S, alpha):
    S = np.ascontiguousarray(S, dtype=np.float64)
    ref, tau = ctypes.c_double(), ctypes.c_double()
    _check(_lib.ctc_threshold_from_samples(_ptr(S), S.size, float(alpha),
                                           ctypes.byref(ref),
                                           ctypes.byref(tau)))
    return ref.value, tau.value


def ctc_threshold_at_ref(S, ref, alpha):
    S = np.ascontiguousarray(S, dtype=np.float64)
    tau = ctypes.c_double()
    _check(_lib.ctc_threshold_at_ref(_ptr(S), S.size, float(ref),
                                     float(alpha), ctypes.byref(tau)))
    return tau.value


def ctc_net_fault_sites(h, with_acts):
    """List of (site, layer, elements, bits) of a bound network."""
    n = ctypes.c_int32()
    _check(_lib.ctc_net_fault_sites(h, int(with_acts), None, 0,
                                    ctypes.byref(n)))
    arr = (ctc_site_info * max(n.value, 1))()
    _check(_lib.ctc_net_fault_sites(h, int(with_acts), arr, n.value,
                                    ctypes.byref(n)))
    return [(a.site, a.layer, a.elements, a.bits) for a in arr[:n.value]]


# ------------------------------------------------------ device entry points

def ctc_conv2d_forward(desc, dtype, n, h, w, x, w_packed, scale, shift,
                       residual, relu, y, stream=None, pool=0, workspace=None,
                       ws_bytes=0):
    _check(_lib.ctc_conv2d_forward(ctypes.byref(desc), dtype, n, h, w,
                                   _ptr(x), _ptr(w_packed), _ptr(scale),
                                   _ptr(shift), _ptr(residual), int(relu),
                                   int(pool), _ptr(y), _ptr(workspace),
                                   int(ws_bytes), _stream(stream)))


def ctc_conv2d_forward_noalloc(desc, dtype, n, h, w, x, w_packed, scale,
                               shift, residual, relu, y, stream=None, pool=0):
    _check(_lib.ctc_conv2d_forward_noalloc(ctypes.byref(desc), dtype, n, h, w,
                                           _ptr(x), _ptr(w_packed),
                                           _ptr(scale), _ptr(shift),
                                           _ptr(residual), int(relu),
                                           int(pool), _ptr(y),
                                           _stream(stream)))


def ctc_conv2d_kernel_name(desc, dtype, n, h, w, pool=0):
    buf = ctypes.create_string_buffer(128)
    _check(_lib.ctc_conv2d_kernel_name(ctypes.byref(desc), dtype, n, h, w,
                                       int(pool), buf, 128))
    return buf.value.decode()


def ctc_conv2d_workspace_bytes(desc, dtype, n, h, w, pool=0):
    b = _SZ()
    _check(_lib.ctc_conv2d_workspace_bytes(ctypes.byref(desc), dtype, n, h, w,
                                           int(pool), ctypes.byref(b)))
    return b.value


def ctc_verify(S, batch, stride, ref, tau, flags, n_flagged, idx,
               stream=None):
    _check(_lib.ctc_verify(_ptr(S), batch, stride, float(ref), float(tau),
                           _ptr(flags), _ptr(n_flagged), _ptr(idx),
                           _stream(stream)))


def ctc_net_create(ops, in_c, in_h, in_w, classes, dtype, protect):
    arr = (ctc_op * len(ops))(*ops)
    h = _P()
    _check(_lib.ctc_net_create(arr, len(ops), in_c, in_h, in_w, classes,
                               dtype, int(protect), ctypes.byref(h)))
    return h.value


def ctc_net_workspace_bytes(net, max_batch):
    b = _SZ()
    _check(_lib.ctc_net_workspace_bytes(net, max_batch, ctypes.byref(b)))
    return b.value


def ctc_net_bind(net, host_params, workspace, ws_bytes, max_batch,
                 stream=None):
    arr = (_P * len(host_params))(*[_ptr(p) for p in host_params])
    _check(_lib.ctc_net_bind(net, arr, _ptr(workspace), ws_bytes, max_batch,
                             _stream(stream)))


def ctc_net_set_fusion(net, kinds):
    """kinds: bit mask of CTC_FUSE_IR / CTC_FUSE_BLOCK / CTC_FUSE_STEM (0:
    none)."""
    _check(_lib.ctc_net_set_fusion(net, int(kinds)))


def ctc_net_set_threshold(net, ref, tau):
    _check(_lib.ctc_net_set_threshold(net, float(ref), float(tau)))


def ctc_network_forward(net, batch, x, out, flags=None,
                        reexec=CTC_REEXEC_NONE, stream=None):
    _check(_lib.ctc_network_forward(net, batch, _ptr(x), _ptr(out),
                                    _ptr(flags), reexec, _stream(stream)))


def ctc_network_flush(net, stream=None):
    _check(_lib.ctc_network_flush(net, _stream(stream)))


def ctc_graph_create(net, batch, passes, x, out, flags=None):
    """Captures `passes` one-pass inferences of `batch` images as a HIP
    graph; returns its handle."""
    g = _P()
    _check(_lib.ctc_graph_create(net, batch, passes, _ptr(x), _ptr(out),
                                 _ptr(flags), ctypes.byref(g)))
    return g


def ctc_graph_launch(graph, reexec=CTC_REEXEC_NONE, stream=None):
    """Replays the graph; returns the number of flagged images (SYNC)."""
    n = _I32(0)
    _check(_lib.ctc_graph_launch(graph, reexec, ctypes.byref(n),
                                 _stream(stream)))
    return n.value


def ctc_graph_destroy(graph):
    _lib.ctc_graph_destroy(graph)


def ctc_inject_bitflip(net, faults, stream=None):
    """faults: iterable of (site, layer, index, bit, image) or a numpy
    structured array with those fields."""
    fl = [ctc_fault(int(f[0]), int(f[1]), int(f[2]), int(f[3]), int(f[4]))
          for f in faults]
    arr = (ctc_fault * max(len(fl), 1))(*fl)
    _check(_lib.ctc_inject_bitflip(net, arr, len(fl), _stream(stream)))


def ctc_clear_faults(net, stream=None):
    _check(_lib.ctc_clear_faults(net, _stream(stream)))


def ctc_net_tensor(net, t):
    dev = _P()
    c, h, w, dt = _I32(), _I32(), _I32(), _I32()
    _check(_lib.ctc_net_tensor(net, t, ctypes.byref(dev), ctypes.byref(c),
                               ctypes.byref(h), ctypes.byref(w),
                               ctypes.byref(dt)))
    return dev.value, c.value, h.value, w.value, dt.value


def ctc_net_weight_address(net, layer, index):
    """(device address, stored bits) of deployed weight `index` of op
    `layer`."""
    dev, bits = _P(), _I32()
    _check(_lib.ctc_net_weight_address(net, layer, index, ctypes.byref(dev),
                                       ctypes.byref(bits)))
    return dev.value, bits.value


def ctc_net_role(net, i):
    return _lib.ctc_net_role(net, i)


def ctc_net_profile(net, enable):
    _check(_lib.ctc_net_profile(net, int(enable)))


def ctc_net_profile_read(net, n_ops):
    """(launches, total_ms) per slot: [stage, op 0 .. op n-1, detector]."""
    launches = np.zeros(n_ops + 2, np.int32)
    ms = np.zeros(n_ops + 2, np.float64)
    _check(_lib.ctc_net_profile_read(net, launches.ctypes.data,
                                     ms.ctypes.data))
    return launches, ms


def ctc_net_op_kernel(net, i, nimg):
    buf = ctypes.create_string_buffer(128)
    _check(_lib.ctc_net_op_kernel(net, i, nimg, buf, 128))
    return buf.value.decode()


def ctc_net_destroy(net):
    _lib.ctc_net_destroy(net)


# -------------------------------------------------- network description

def ops_from_layers(layers):
    """ctc_op structs from layer dicts (keys as in the workload
    descriptors: op, inp, c_in, c_out, k, stride, pad, groups, bias, bn,
    relu, residual, block_first, shortcut; fc: in_f, out_f, final, flatten,
    out_f32)."""
    ops = []
    for L in layers:
        o = ctc_op()
        o.input = L["inp"]
        o.residual = -1
        if L["op"] == "conv":
            o.kind = CTC_OP_CONV
            o.c_in, o.c_out, o.k = L["c_in"], L["c_out"], L["k"]
            o.stride, o.pad, o.groups = L["stride"], L["pad"], L["groups"]
            o.has_bias, o.has_bn = int(L["bias"]), int(L["bn"])
            o.relu, o.residual = int(L["relu"]), L["residual"]
            o.block_first, o.shortcut = int(L["block_first"]), \
                int(L["shortcut"])
        elif L["op"] == "maxpool":
            o.kind = CTC_OP_MAXPOOL
            o.k, o.stride, o.pad = L["k"], L["stride"], L["pad"]
        elif L["op"] == "gap":
            o.kind = CTC_OP_GAP
        elif L["op"] == "fc":
            o.kind = CTC_OP_FC
            o.c_in, o.c_out = L["in_f"], L["out_f"]
            o.has_bias, o.relu = int(L["bias"]), int(L["relu"])
            o.final_fc = int(L["final"])
            if L["flatten"] is not None:
                o.flatten_c, o.flatten_h, o.flatten_w = L["flatten"]
            o.out_f32 = int(L.get("out_f32", False))
        else:
            raise ValueError(L["op"])
        ops.append(o)
    return ops


def ctc_select_channels_l1(layers, params):
    """L1-norm choice of the pruned channel (Sec. II-A) on canonical params
    (list of dicts as from the workload generator).  Returns (new params,
    chosen channel per op); the input is not modified."""
    ops = ops_from_layers(layers)
    oa = (ctc_op * len(ops))(*ops)
    host = host_param_list(layers, params)
    host = [None if h is None else h.copy() for h in host]
    arr = (_P * len(host))(*[_ptr(h) for h in host])
    chosen = np.zeros(len(ops), np.int32)
    _check(_lib.ctc_select_channels_l1(oa, len(ops), arr, _ptr(chosen)))
    out = []
    keys = ("w", "b", "mean", "var", "gamma", "beta")
    for i, p in enumerate(params):
        if p is None:
            out.append(None)
            continue
        out.append({k: host[6 * i + j].reshape(p[k].shape)
                    for j, k in enumerate(keys) if k in p})
    return out, chosen.tolist()


def host_param_list(layers, params):
    """6 pointers' worth of arrays per op (w, bias, mean, var, gamma,
    beta), None where absent; float32 C-contiguous copies."""
    out = []
    for L, p in zip(layers, params):
        if p is None:
            out += [None] * 6
            continue
        for k in ("w", "b", "mean", "var", "gamma", "beta"):
            v = p.get(k)
            out.append(None if v is None else
                       np.ascontiguousarray(v, dtype=np.float32))
    return out
