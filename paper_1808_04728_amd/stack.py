"""The CosmoFlow-shaped conv stack driven through the C ABI.

One training step of the hot path (the order of a TensorFlow forward and
backward pass over the network's convolution part, Section III-A):

  forward,  layer 1..L:  conv -> bias + leaky ReLU (in place) -> [2^3 avg-pool]
  backward, layer L..1:  [pool backward] -> leaky-ReLU backward (+ bias grad)
                         -> weight grad -> data grad (skipped for layer 1,
                            whose input needs no gradient)

PyTorch only allocates device memory and supplies the stream; every step is
one call of ``binding`` (a HIP kernel).  Buffers are allocated once, so a
step launches kernels and nothing else.

Parameters live in flat buffers, one parameter group per tensor (layer l's
weights, then its biases): fp32 master values ``flat_param`` (the weights of
an fp32 stack and every bias are views of it), the bf16 copy ``flat_w16``
the convolutions of a bf16 stack read, and the gradient ``flat_grad`` that
the backward pass writes.  ``update`` applies the paper's Adam + LARC rule
(Section III-B) to all groups in one call.
"""
from __future__ import annotations

import torch

from . import binding as B


def _t(dtype):
    return torch.bfloat16 if dtype == "bf16" else torch.float32


class ConvStack:
    def __init__(self, layers, size, batch, dtype="f32", alpha=0.01, device="cuda", skip_first_dgrad=True,
                 fused=True, defer_reductions=True, overlap_wgrad=None, pooled_dz_pass=True, fused_from=0,
                 dz_pass_layers=None):
        """fused: run a pooled layer through the fused entry points (forward
        epilogue writes pooled output + slope mask; backward rebuilds dz from
        them) wherever the library has fused kernels for the layer.
        defer_reductions: batch all gradient sums of a backward pass into one
        cf_reduce_partials launch.
        overlap_wgrad: in the backward pass of a layer below the first two, run
        the weight gradient on a second stream (default priority) concurrently
        with the data gradient; both only read dz (or its sources), and the
        small deep layers leave most of the GPU idle when run one after the
        other.  None (default) = on for bf16 stacks, off for fp32 ones (measured
        on the 128^3 stacks: bf16 batch 8 0.718 -> 0.709 ms with it; fp32 batch
        1 0.808 -> 0.815 ms, its narrow deep-layer kernels already spread over
        the machine).
        fused_from: layers before this index only are eligible for fusion when it
        is > 0 (an A/B switch: e.g. 2 runs the deep layers unfused).
        pooled_dz_pass: a fused pooled layer without a dz-storing weight-gradient
        kernel forms dz in one pass from the pooled gradient and the mask
        (cf_avgpool3d_lrelu_bwd) for the plain gradient kernels; False runs the
        fused backward kernels, which form dz as they load it.
        dz_pass_layers: indices of fused pooled layers that form dz in that one
        pass even where a dz-storing weight-gradient kernel exists (None: every
        such layer of an fp32 stack)."""
        self.fused = fused
        self.pooled_dz_pass = pooled_dz_pass
        self.dz_pass_layers = dz_pass_layers
        self.fused_from = fused_from
        self.defer_reductions = defer_reductions
        self.reduce_bytes = 0
        self.layers = layers
        self.batch = batch
        self.dtype = dtype
        self.tdt = _t(dtype)
        self.alpha = float(alpha)
        self.device = device
        self.skip_first_dgrad = skip_first_dgrad
        self.timer = None  # optional: {op name: [(start event, end event), ...]}
        self.timed_ops = None  # None = every op, else the set of op names to time
        import torch as _torch
        if overlap_wgrad is None:
            overlap_wgrad = dtype == "bf16"
        self.side = _torch.cuda.Stream(device=device) if overlap_wgrad else None
        self.L = []
        dhw = (size, size, size)
        for i, spec in enumerate(layers):
            desc = B.make_desc(batch, dhw, spec["cin"], spec["cout"], spec["k"], spec["stride"],
                               spec.get("pad", "same"), dtype)
            od = B.cf_conv3d_out_shape(desc)
            pdhw = tuple(t // 2 for t in od) if spec["pool"] else od
            self.L.append(dict(spec=spec, desc=desc, in_dhw=dhw, out_dhw=od, pool_dhw=pdhw,
                               nvox=batch * od[0] * od[1] * od[2]))
            dhw = pdhw
        self.out_dhw = dhw
        self._alloc()

    # ------------------------------------------------------------------
    def _alloc_params(self):
        """Flat parameter / gradient buffers; every group starts on a multiple
        of 16 elements (64 bytes), padding (zeros) belongs to the group before."""
        dev = self.device
        off, shapes = [0], []
        for l in self.L:
            s = l["spec"]
            for shape in (((s["k"],) * 3 + (s["cin"], s["cout"])), (s["cout"],)):
                n = 1
                for t in shape:
                    n *= t
                shapes.append(shape)
                off.append(off[-1] + (n + 15) // 16 * 16)
        self.param_offsets = off
        total = off[-1]
        self.flat_param = torch.zeros(total, dtype=torch.float32, device=dev)
        self.flat_grad = torch.zeros(total, dtype=torch.float32, device=dev)
        self.flat_w16 = torch.zeros(total, dtype=torch.bfloat16, device=dev) if self.dtype == "bf16" else None
        wsrc = self.flat_w16 if self.flat_w16 is not None else self.flat_param

        def view(buf, g):
            shape = shapes[g]
            n = 1
            for t in shape:
                n *= t
            return buf[off[g]:off[g] + n].view(shape)

        for i, l in enumerate(self.L):
            l["w"] = view(wsrc, 2 * i)
            l["w32"] = view(self.flat_param, 2 * i)
            l["b"] = view(self.flat_param, 2 * i + 1)
            l["dw"] = view(self.flat_grad, 2 * i)
            l["db"] = view(self.flat_grad, 2 * i + 1)
        self.opt_m = self.opt_s = self.opt_ws = None
        self.opt_t = 0

    def _alloc(self):
        dev, tdt, n = self.device, self.tdt, self.batch
        self._alloc_params()
        for i, l in enumerate(self.L):
            s = l["spec"]
            needs_dgrad = i > 0 or not self.skip_first_dgrad
            sup = B.cf_conv3d_fused_supported(l["desc"], B.CF_FUSE_POOL2) if s["pool"] else 0
            # fused needs both fused kernels; a layer whose data gradient is needed keeps dz
            both = B.FUSED_FWD | B.FUSED_BWD_WEIGHT
            # a layer whose data gradient is needed also needs a fused backward-data, or a
            # backward-weights that stores dz for the unfused backward-data
            fz = self.fused and (self.fused_from <= 0 or i < self.fused_from)
            l["fused"] = bool(fz and (sup & both) == both and
                              (not needs_dgrad or sup & (B.FUSED_BWD_DATA | B.FUSED_BWD_WEIGHT_DZ)))
            # otherwise conv + bias + leaky ReLU may still share one kernel (y written once)
            sup0 = B.cf_conv3d_fused_supported(l["desc"], 0) if not s["pool"] else 0
            l["fused_act"] = bool(fz and not l["fused"] and sup0 & B.FUSED_FWD)
            # and its backward may take (dy, y) straight into the weight and data
            # gradients (dz formed inside both, no separate leaky-ReLU backward)
            l["fused_y"] = bool(l["fused_act"] and sup0 & B.FUSED_BWD_WEIGHT and
                                (not needs_dgrad or sup0 & B.FUSED_BWD_DATA))
            l["p"] = torch.empty((n,) + l["pool_dhw"] + (s["cout"],), dtype=tdt, device=dev) if s["pool"] else None
            l["gout"] = torch.empty((n,) + l["pool_dhw"] + (s["cout"],), dtype=tdt, device=dev)
            l["dx"] = None
            if l["fused"]:
                l["z"] = l["dy"] = l["dz"] = None
                # a layer whose data gradient is needed may take dz from its weight-gradient
                # pass and run the unfused backward-data on it (same dx bits, faster there)
                # (in fp32 the stride-2 layer takes the one-pass dz below instead: its
                # two plain products then share one launch)
                if self.dz_pass_layers is None:
                    # fp32: the plain weight gradient on a stored dz beats the one that
                    # rebuilds it per load (the 16 -> 32 layer: 189 -> 171 us, with an
                    # 12 us dz pass), and the stride-2 layer's two products share a launch
                    pair_pass = self.dtype == "f32" and self.pooled_dz_pass
                else:
                    pair_pass = i in self.dz_pass_layers and self.pooled_dz_pass
                l["dz_emit"] = bool(needs_dgrad and sup & B.FUSED_BWD_WEIGHT_DZ and not pair_pass)
                # or, without that kernel, form dz in one pooled-gradient pass and run the
                # plain weight and data gradients on it side by side: the data gradient
                # gathers every dz element k^3 times, so forming dz once beats forming it
                # inside every gather (the stride-2 layer: 4 + 26 us against 47 us)
                od = l["out_dhw"]
                l["dz_pass"] = bool(needs_dgrad and not l["dz_emit"] and self.pooled_dz_pass and
                                    B.cf_avgpool3d_lrelu_bwd_workspace_size(n, *od, s["cout"]) > 0 and
                                    self._pool_lrelu_ok(n, od, s["cout"]))
                if l["dz_emit"] or l["dz_pass"]:
                    l["dz"] = torch.empty((n,) + l["out_dhw"] + (s["cout"],), dtype=tdt, device=dev)
                l["mask"] = torch.empty(max(16, B.cf_conv3d_mask_bytes(l["desc"])), dtype=torch.uint8, device=dev)
                if l["dz_pass"]:
                    wsw = B.cf_conv3d_bwd_weight_workspace_size(l["desc"])
                    wsb = B.cf_avgpool3d_lrelu_bwd_workspace_size(n, *od, s["cout"])
                    l["ws_w"] = torch.empty(max(wsw, 16), dtype=torch.uint8, device=dev)
                    l["ws_b"] = torch.empty(max(wsb, 16), dtype=torch.uint8, device=dev)
                    continue
                wsf = B.cf_conv3d_bwd_weight_fused_workspace_size(l["desc"], B.CF_FUSE_POOL2)
                l["ws_w"] = torch.empty(max(wsf, 16), dtype=torch.uint8, device=dev)
                l["ws_b"] = None
                continue
            l["z"] = torch.empty((n,) + l["out_dhw"] + (s["cout"],), dtype=tdt, device=dev)  # z, then y in place
            l["dy"] = torch.empty_like(l["z"]) if s["pool"] else None
            if l["fused_y"]:
                l["dz"] = None
                wsf = B.cf_conv3d_bwd_weight_fused_workspace_size(l["desc"], 0)
                l["ws_w"] = torch.empty(max(wsf, 16), dtype=torch.uint8, device=dev)
                l["ws_b"] = None
                continue
            l["dz"] = torch.empty_like(l["z"])
            wsw = B.cf_conv3d_bwd_weight_workspace_size(l["desc"])
            wsb = B.cf_bias_lrelu_bwd_workspace_size(l["nvox"], s["cout"])
            l["ws_w"] = torch.empty(max(wsw, 16), dtype=torch.uint8, device=dev)
            l["ws_b"] = torch.empty(max(wsb, 16), dtype=torch.uint8, device=dev)
        for i in range(1, len(self.L)):
            self.L[i]["dx"] = self.L[i - 1]["gout"]
        if not self.skip_first_dgrad:
            s = self.L[0]["spec"]
            self.L[0]["dx"] = torch.empty((n,) + self.L[0]["in_dhw"] + (s["cin"],), dtype=tdt, device=dev)
        self.x = torch.empty((n,) + self.L[0]["in_dhw"] + (self.L[0]["spec"]["cin"],), dtype=tdt, device=dev)

    def _pool_lrelu_ok(self, n, od, c):
        # the one-pass kernel's channel rule (whole 16-byte vectors, a power of two of
        # them, at most 64, c <= 256); the call itself rejects anything else
        v = 8 if self.dtype == "bf16" else 4
        g = c // v
        return c % v == 0 and g > 0 and (g & (g - 1)) == 0 and g <= 64 and c <= 256

    def set_params(self, weights, biases):
        """Weights are rounded to the stack's dtype; the fp32 master copy holds
        exactly those values.  Resets the optimizer state."""
        for l, w, b in zip(self.L, weights, biases):
            l["w"].copy_(torch.as_tensor(w).to(self.tdt))
            if l["w32"].data_ptr() != l["w"].data_ptr():
                l["w32"].copy_(l["w"].float())
            l["b"].copy_(torch.as_tensor(b).float())
        self.reset_optimizer()

    def reset_optimizer(self):
        self.opt_t = 0
        if self.opt_m is not None:
            self.opt_m.zero_()
            self.opt_s.zero_()

    def update(self, hp, stream=None):
        """One parameter update from the gradient of the last backward pass
        (Adam + LARC + linear decay, one group per tensor); hp is a
        binding.cf_adam_larc_hparams.  Writes the master values and, for a
        bf16 stack, the bf16 weights the next forward pass reads."""
        if self.opt_m is None:
            self.opt_m = torch.zeros_like(self.flat_param)
            self.opt_s = torch.zeros_like(self.flat_param)
            nws = B.cf_adam_larc_workspace_size(self.param_offsets)
            self.opt_ws = torch.empty(max(nws, 16), dtype=torch.uint8, device=self.device)
            self._opt_off = B.adam_offsets(self.param_offsets)
        self._call("L0.adam_larc_update", B.cf_adam_larc_step, self._opt_off, self.opt_t, hp, self.flat_param,
                   self.flat_grad, self.opt_m, self.opt_s, self.flat_w16, self.opt_ws, None, stream)
        self.opt_t += 1

    def update_bytes(self):
        """Algorithmic HBM bytes of one update: v, g, m, s read, v, m, s (and
        the bf16 copy) written."""
        n = self.param_offsets[-1]
        return n * (7 * 4 + (2 if self.flat_w16 is not None else 0))

    def set_input(self, x):
        self.x.copy_(torch.as_tensor(x).to(self.tdt))

    def output(self):
        l = self.L[-1]
        return l["p"] if l["spec"]["pool"] else l["z"]

    def _call(self, name, fn, *args, rec=None):
        """fn(*args), bracketed by timing events on stream rec (None: the
        current stream) when the op is timed."""
        if self.timer is None or (self.timed_ops is not None and name not in self.timed_ops):
            return fn(*args)
        import torch as _torch
        e0 = _torch.cuda.Event(enable_timing=True)
        e1 = _torch.cuda.Event(enable_timing=True)
        e0.record(rec)
        r = fn(*args)
        e1.record(rec)
        self.timer.setdefault(name, []).append((e0, e1))
        return r

    # ------------------------------------------------------------------
    def forward(self, stream=None):
        h = self.x
        for i, l in enumerate(self.L):
            s = l["spec"]
            c = self._call
            if l["fused"]:
                c(f"L{i+1}.conv_fwd_fused", B.cf_conv3d_fwd_fused, l["desc"], h, l["w"], l["b"], self.alpha,
                  B.CF_FUSE_POOL2, l["p"], l["mask"], stream)
                h = l["p"]
                continue
            if l["fused_act"]:
                c(f"L{i+1}.conv_bias_lrelu_fwd", B.cf_conv3d_fwd_fused, l["desc"], h, l["w"], l["b"], self.alpha, 0,
                  l["z"], None, stream)
            else:
                c(f"L{i+1}.conv_fwd", B.cf_conv3d_fwd, l["desc"], h, l["w"], l["z"], stream)
                c(f"L{i+1}.bias_lrelu_fwd", B.cf_bias_lrelu_fwd, l["nvox"], s["cout"], self.dtype, l["z"], l["b"],
                  self.alpha, l["z"], stream)
            if s["pool"]:
                d, hh, w = l["out_dhw"]
                c(f"L{i+1}.avgpool_fwd", B.cf_avgpool3d_fwd, self.batch, d, hh, w, s["cout"], 2, 2, self.dtype,
                  l["z"], l["p"], stream)
                h = l["p"]
            else:
                h = l["z"]
        return h

    def backward(self, dout, stream=None):
        """dout: gradient w.r.t. the last layer's output (not modified).

        With defer_reductions (the default) every layer's weight- and
        bias-gradient calls leave their fixed-order partial sums pending and
        one cf_reduce_partials call at the end writes all dW and db (the same
        bits as the plain calls)."""
        g = dout
        pend = []
        d = self.defer_reductions
        side_used = False
        for i in range(len(self.L) - 1, -1, -1):
            l = self.L[i]
            s = l["spec"]
            c = self._call
            # a fused layer's backward runs on one stream when its data gradient
            # follows from the dz its weight gradient stores, or when it has none
            # (the first two layers: their kernels fill the GPU by themselves);
            # it starts after the side stream's weight gradients have finished
            one_stream = l["fused"] and (l["dz_emit"] or l["dx"] is None)
            if l["fused"] and l["dz_pass"]:
                # dz (and db) in one pass from the pooled gradient and the mask, then
                # the plain weight gradient (side stream) beside the data gradient
                od = l["out_dhw"]
                if d:
                    pend += c(f"L{i+1}.pool_lrelu_bwd", B.cf_avgpool3d_lrelu_bwd_deferred, self.batch, *od,
                              s["cout"], self.dtype, g, l["mask"], self.alpha, l["dz"], l["db"], l["ws_b"], None,
                              stream)
                else:
                    c(f"L{i+1}.pool_lrelu_bwd", B.cf_avgpool3d_lrelu_bwd, self.batch, *od, s["cout"], self.dtype, g,
                      l["mask"], self.alpha, l["dz"], l["db"], l["ws_b"], None, stream)
                if self.side is None and s["stride"] > 1:
                    # both plain products from dz in one call (the stride-2 layer's share
                    # one launch)
                    if d:
                        pend += c(f"L{i+1}.conv_bwd", B.cf_conv3d_bwd_deferred, l["desc"], self.layer_input(i),
                                  l["dz"], l["w"], l["dw"], l["dx"], l["ws_w"], None, stream)
                    else:
                        c(f"L{i+1}.conv_bwd", B.cf_conv3d_bwd, l["desc"], self.layer_input(i), l["dz"], l["w"],
                          l["dw"], l["dx"], l["ws_w"], None, stream)
                    g = l["dx"]
                    continue
                ws_ = stream
                if self.side is not None:
                    main = stream if stream is not None else torch.cuda.current_stream()
                    ev = torch.cuda.Event()
                    ev.record(main)
                    self.side.wait_event(ev)
                    ws_ = self.side
                    side_used = True
                if d:
                    pend += c(f"L{i+1}.conv_bwd_weight", B.cf_conv3d_bwd_weight_deferred, l["desc"],
                              self.layer_input(i), l["dz"], l["dw"], l["ws_w"], None, ws_, rec=ws_)
                else:
                    c(f"L{i+1}.conv_bwd_weight", B.cf_conv3d_bwd_weight, l["desc"], self.layer_input(i), l["dz"],
                      l["dw"], l["ws_w"], None, ws_, rec=ws_)
                c(f"L{i+1}.conv_bwd_data", B.cf_conv3d_bwd_data, l["desc"], l["dz"], l["w"], l["dx"], stream)
                g = l["dx"]
                continue
            if one_stream and side_used:
                self._join_side(stream)
                side_used = False
            if l["fused"] and l["dz_emit"]:
                if d:
                    pend += c(f"L{i+1}.conv_bwd_weight_fused_dz", B.cf_conv3d_bwd_weight_fused_deferred, l["desc"],
                              self.layer_input(i), g, l["mask"], self.alpha, B.CF_FUSE_POOL2, l["dw"], l["db"],
                              l["dz"], l["ws_w"], None, stream)
                else:
                    c(f"L{i+1}.conv_bwd_weight_fused_dz", B.cf_conv3d_bwd_weight_fused_dz, l["desc"],
                      self.layer_input(i), g, l["mask"], self.alpha, B.CF_FUSE_POOL2, l["dw"], l["db"], l["dz"],
                      l["ws_w"], None, stream)
                c(f"L{i+1}.conv_bwd_data", B.cf_conv3d_bwd_data, l["desc"], l["dz"], l["w"], l["dx"], stream)
                g = l["dx"]
                continue
            if l["fused"]:
                # with a fused data gradient to follow, the weight gradient goes to the
                # side stream (both form dz from the pooled gradient and the mask)
                ws_ = stream
                if self.side is not None and l["dx"] is not None:
                    main = stream if stream is not None else torch.cuda.current_stream()
                    ev = torch.cuda.Event()
                    ev.record(main)
                    self.side.wait_event(ev)
                    ws_ = self.side
                    side_used = True
                if d:
                    pend += c(f"L{i+1}.conv_bwd_weight_fused", B.cf_conv3d_bwd_weight_fused_deferred, l["desc"],
                              self.layer_input(i), g, l["mask"], self.alpha, B.CF_FUSE_POOL2, l["dw"], l["db"],
                              None, l["ws_w"], None, ws_, rec=ws_)
                else:
                    c(f"L{i+1}.conv_bwd_weight_fused", B.cf_conv3d_bwd_weight_fused, l["desc"], self.layer_input(i),
                      g, l["mask"], self.alpha, B.CF_FUSE_POOL2, l["dw"], l["db"], l["ws_w"], None, ws_, rec=ws_)
                if l["dx"] is not None:
                    c(f"L{i+1}.conv_bwd_data_fused", B.cf_conv3d_bwd_data_fused, l["desc"], g, l["mask"], l["w"],
                      self.alpha, B.CF_FUSE_POOL2, l["dx"], stream)
                    g = l["dx"]
                continue
            if l["fused_y"] and self.side is None and l["dx"] is not None:
                # (dy, y): dW, db and dx in one call (one launch where the kernels allow)
                if d:
                    pend += c(f"L{i+1}.conv_bwd_fused", B.cf_conv3d_bwd_fused_deferred, l["desc"],
                              self.layer_input(i), g, l["z"], l["w"], self.alpha, 0, l["dw"], l["db"], l["dx"],
                              l["ws_w"], None, stream)
                else:
                    c(f"L{i+1}.conv_bwd_fused", B.cf_conv3d_bwd_fused, l["desc"], self.layer_input(i), g, l["z"],
                      l["w"], self.alpha, 0, l["dw"], l["db"], l["dx"], l["ws_w"], None, stream)
                g = l["dx"]
                continue
            if l["fused_y"]:
                # (dy, y): the weight gradient (and db) on the side stream, the data
                # gradient on the main stream, both forming dz from dy and y
                ws_ = stream
                if self.side is not None and l["dx"] is not None:
                    main = stream if stream is not None else torch.cuda.current_stream()
                    ev = torch.cuda.Event()
                    ev.record(main)
                    self.side.wait_event(ev)
                    ws_ = self.side
                    side_used = True
                if d:
                    pend += c(f"L{i+1}.conv_bwd_weight_fused", B.cf_conv3d_bwd_weight_fused_deferred, l["desc"],
                              self.layer_input(i), g, l["z"], self.alpha, 0, l["dw"], l["db"], None, l["ws_w"],
                              None, ws_, rec=ws_)
                else:
                    c(f"L{i+1}.conv_bwd_weight_fused", B.cf_conv3d_bwd_weight_fused, l["desc"], self.layer_input(i),
                      g, l["z"], self.alpha, 0, l["dw"], l["db"], l["ws_w"], None, ws_, rec=ws_)
                if l["dx"] is not None:
                    c(f"L{i+1}.conv_bwd_data_fused", B.cf_conv3d_bwd_data_fused, l["desc"], g, l["z"], l["w"],
                      self.alpha, 0, l["dx"], stream)
                    g = l["dx"]
                continue
            if s["pool"]:
                c(f"L{i+1}.avgpool_bwd", B.cf_avgpool3d_bwd, self.batch, *l["out_dhw"], s["cout"], 2, 2, self.dtype,
                  g, l["dy"], stream)
                dy = l["dy"]
            else:
                dy = g
            # weight gradient on the side stream when a data gradient follows
            ws_ = stream
            if self.side is not None and l["dx"] is not None:
                main = stream if stream is not None else torch.cuda.current_stream()
                ev = torch.cuda.Event()
            if d:
                pend += c(f"L{i+1}.bias_lrelu_bwd", B.cf_bias_lrelu_bwd_deferred, l["nvox"], s["cout"], self.dtype,
                          dy, l["z"], self.alpha, l["dz"], l["db"], l["ws_b"], None, stream)
            else:
                c(f"L{i+1}.bias_lrelu_bwd", B.cf_bias_lrelu_bwd, l["nvox"], s["cout"], self.dtype, dy, l["z"],
                  self.alpha, l["dz"], l["db"], l["ws_b"], None, stream)
            if self.side is not None and l["dx"] is not None:
                ev.record(main)
                self.side.wait_event(ev)
                ws_ = self.side
                side_used = True
            if d:
                pend += c(f"L{i+1}.conv_bwd_weight", B.cf_conv3d_bwd_weight_deferred, l["desc"],
                          self.layer_input(i), l["dz"], l["dw"], l["ws_w"], None, ws_, rec=ws_)
            else:
                c(f"L{i+1}.conv_bwd_weight", B.cf_conv3d_bwd_weight, l["desc"], self.layer_input(i), l["dz"],
                  l["dw"], l["ws_w"], None, ws_, rec=ws_)
            if l["dx"] is not None:
                c(f"L{i+1}.conv_bwd_data", B.cf_conv3d_bwd_data, l["desc"], l["dz"], l["w"], l["dx"], stream)
                g = l["dx"]
        if side_used:
            # join: everything after the backward pass sees the weight gradients
            self._join_side(stream)
        if pend:
            self.reduce_bytes = sum(j.rows * j.cols * 4 + j.cols * 4 for j in pend)
            self._call("L0.reduce_partials", B.cf_reduce_partials, pend, stream)

    def _join_side(self, stream):
        """Work queued on `stream` (None: the current stream) after this call
        waits for everything queued on the side stream so far."""
        ev = torch.cuda.Event()
        ev.record(self.side)
        (stream if stream is not None else torch.cuda.current_stream()).wait_event(ev)

    def layer_input(self, i):
        if i == 0:
            return self.x
        p = self.L[i - 1]
        return p["p"] if p["spec"]["pool"] else p["z"]

    def output_tensors(self, i):
        """(pooled-or-activated output, y or None) of layer i, for checks."""
        l = self.L[i]
        return (l["p"] if l["spec"]["pool"] else l["z"]), l["z"]

    def op_flops(self, name):
        """Algorithmic FLOPs of one call of a conv op (2 * MACs), else 0."""
        if ".conv_" not in name:
            return 0
        i = int(name[1:name.index(".")]) - 1
        l = self.L[i]
        s = l["spec"]
        f = 2 * l["nvox"] * s["cout"] * s["k"] ** 3 * s["cin"]
        return 2 * f if name.endswith((".conv_bwd_fused", ".conv_bwd")) else f  # weight and data gradients

    def op_bytes(self, name):
        """Algorithmic HBM bytes of one call (every tensor read once, written once)."""
        if name.endswith(".reduce_partials"):
            return self.reduce_bytes
        if name.endswith(".adam_larc_update"):
            return self.update_bytes()
        i = int(name[1:name.index(".")]) - 1
        l = self.L[i]
        s = l["spec"]
        es = 2 if self.dtype == "bf16" else 4
        vin = self.batch * l["in_dhw"][0] * l["in_dhw"][1] * l["in_dhw"][2]
        xb = vin * s["cin"] * es
        zb = l["nvox"] * s["cout"] * es
        wb = s["k"] ** 3 * s["cin"] * s["cout"] * es
        pb = zb // 8
        op = name.split(".")[1]
        mb = l["nvox"] * s["cout"] // 8
        if op in ("conv_bwd_weight_fused", "conv_bwd_data_fused", "conv_bwd_fused") and not s["pool"]:
            # the (dy, y) form reads dy and y in place of the pooled gradient and mask
            pb = mb = zb
        return {"conv_fwd_fused": xb + wb + pb + mb, "conv_bwd_weight_fused": xb + pb + mb + wb // es * 4,
                "conv_bwd_weight_fused_dz": xb + pb + mb + wb // es * 4 + zb,
                "conv_bwd_data_fused": pb + mb + wb + xb,
                "conv_bwd_fused": xb + pb + mb + wb // es * 4 + wb + xb,
                "conv_bwd": xb + zb + wb // es * 4 + wb + xb,
                "conv_bias_lrelu_fwd": xb + wb + zb,
                "conv_fwd": xb + wb + zb, "conv_bwd_data": zb + wb + xb,
                "conv_bwd_weight": xb + zb + wb // es * 4, "bias_lrelu_fwd": 2 * zb,
                "bias_lrelu_bwd": 3 * zb, "avgpool_fwd": zb + pb, "avgpool_bwd": zb + pb,
                "pool_lrelu_bwd": pb + mb + zb}[op]

    # ------------------------------------------------------------------
    def conv_flops(self):
        """Algorithmic conv FLOPs of one step: 2 * MACs for fwd, wgrad and
        (except a skipped first layer) dgrad; padded taps included."""
        f = 0
        for i, l in enumerate(self.L):
            s = l["spec"]
            macs = l["nvox"] * s["cout"] * s["k"] ** 3 * s["cin"]
            f += 2 * macs * (2 if (i == 0 and self.skip_first_dgrad) else 3)
        return f
