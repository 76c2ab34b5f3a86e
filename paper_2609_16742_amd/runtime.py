"""Convenience owner of a bound network: workspace (a torch uint8 tensor on
the device), the ctc_net handle and thin wrappers of the forward, detector
and fault entry points.  Marshalling only; the work runs in libctc.so."""

from __future__ import annotations

import torch

from . import ctc


class CtcNet:
    def __init__(self, layers, in_shape, classes, dtype, params, protect=True,
                 max_batch=128, device="cuda", stream=None):
        self.layers = layers
        self.in_shape = tuple(in_shape)
        self.classes = classes
        self.dtype = dtype
        # protect: False / True (replace mode) / "append"
        mode = {False: 0, True: 1, "replace": 1, "append": 2}[protect]
        self.protect = mode > 0
        self.mode = mode
        self.max_batch = max_batch
        self.out_cols = classes + (1 if mode else 0)
        self.h = ctc.ctc_net_create(ctc.ops_from_layers(layers), in_shape[0],
                                    in_shape[1], in_shape[2], classes,
                                    ctc.DTYPES[dtype], mode)
        self.ws_bytes = ctc.ctc_net_workspace_bytes(self.h, max_batch)
        self._ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8,
                               device=device)
        self._ws_off = (-self._ws.data_ptr()) % 256
        self.ws = self._ws[self._ws_off:self._ws_off + self.ws_bytes]
        host = ctc.host_param_list(layers, params)
        ctc.ctc_net_bind(self.h, host, self.ws.data_ptr(), self.ws_bytes,
                         max_batch, stream)

    def __del__(self):
        h = getattr(self, "h", None)
        if h:
            self.h = None
            try:
                ctc.ctc_net_destroy(h)
            except TypeError:
                # interpreter shutdown: the binding module is already torn
                # down and the process is about to release everything
                pass

    def set_fusion(self, kinds):
        """Fusion kinds in effect: a CTC_FUSE_* bit mask; True selects every
        kind, False none (default: every kind)."""
        if kinds is True:
            kinds = (ctc.CTC_FUSE_IR | ctc.CTC_FUSE_BLOCK | ctc.CTC_FUSE_STEM
                     | ctc.CTC_FUSE_POOL)
        ctc.ctc_net_set_fusion(self.h, int(kinds))

    def set_threshold(self, ref, tau):
        ctc.ctc_net_set_threshold(self.h, ref, tau)

    def forward(self, x, out=None, flags=None, reexec=ctc.CTC_REEXEC_NONE,
                stream=None):
        n = x.shape[0]
        if out is None:
            if reexec == ctc.CTC_REEXEC_DEFERRED:
                # the library writes re-executed rows into `out` during
                # later calls: a buffer only this call referenced could be
                # reused by the caching allocator before then
                raise ValueError("deferred re-execution needs a caller-owned "
                                 "`out` that stays alive until the flush")
            out = torch.empty((n, self.out_cols), dtype=torch.float32,
                              device=x.device)
        ctc.ctc_network_forward(self.h, n, x, out, flags, reexec, stream)
        return out

    def flush(self, stream=None):
        ctc.ctc_network_flush(self.h, stream)

    def graph(self, x, batch, out=None, flags=None):
        """Captures x.shape[0] / batch one-pass inferences as a HIP graph
        (ctc_graph_create); returns a CtcGraph that keeps x, out and flags
        alive."""
        n = x.shape[0]
        if batch < 1 or n % batch:
            raise ValueError("%d images are not a whole number of %d-image "
                             "passes" % (n, batch))
        if out is None:
            out = torch.empty((n, self.out_cols), dtype=torch.float32,
                              device=x.device)
        return CtcGraph(self, x, batch, out, flags)

    def inject(self, faults, stream=None):
        ctc.ctc_inject_bitflip(self.h, faults, stream)

    def clear_faults(self, stream=None):
        ctc.ctc_clear_faults(self.h, stream)

    def fault_sites(self, with_acts=False):
        return ctc.ctc_net_fault_sites(self.h, with_acts)

    def role(self, i):
        return ctc.ctc_net_role(self.h, i)

    def tensor(self, t, n):
        """Device view of tensor t for the first n images: (n, h, w, c)."""
        dev, cs, h, w, dt = ctc.ctc_net_tensor(self.h, t)
        tdt = torch.float16 if dt == ctc.CTC_F16 else torch.float32
        off = dev - self.ws.data_ptr()
        nbytes = n * h * w * cs * (2 if dt == ctc.CTC_F16 else 4)
        return self.ws[off:off + nbytes].view(tdt).reshape(n, h, w, cs)

    def weight_bits(self, layer, index):
        """The stored bit pattern (int) of deployed weight `index` of op
        `layer`, read from the device workspace."""
        dev, bits = ctc.ctc_net_weight_address(self.h, layer, index)
        off = dev - self.ws.data_ptr()
        b = self.ws[off:off + bits // 8].cpu().numpy()
        return int.from_bytes(b.tobytes(), "little")


class CtcGraph:
    """A captured run of passes of one CtcNet (ctc_graph_*)."""

    def __init__(self, net, x, batch, out, flags):
        self.net, self.x, self.out, self.flags = net, x, out, flags
        self.h = ctc.ctc_graph_create(net.h, batch, x.shape[0] // batch, x,
                                      out, flags)

    def launch(self, reexec=ctc.CTC_REEXEC_NONE, stream=None):
        """Replays the graph; with CTC_REEXEC_SYNC re-runs the flagged images
        and returns how many there were."""
        return ctc.ctc_graph_launch(self.h, reexec, stream)

    def __del__(self):
        h = getattr(self, "h", None)
        if h:
            self.h = None
            try:
                ctc.ctc_graph_destroy(h)
            except TypeError:
                pass
