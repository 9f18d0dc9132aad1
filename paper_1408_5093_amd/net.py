"""A fixed chain of convolution layers with the glue between them, run
forward and backward through the C ABI (fp32: the weight and bias gradients
on a second stream, next to the data gradients and the glue).

The paper's Sec. 3.3 describes a network as bookkeeping over layers: a
forward sweep from the data to the top, then a backward sweep that hands
each layer the gradient of its output.  ``ConvStack`` is that bookkeeping for
a fixed chain (CaffeNet conv1-5 with max-pool + LRN after conv1 and conv2,
optionally followed by max-pool and the fc6-fc8 inner products; or the LeNet
conv pair with max-pool between), with every blob preallocated
once so that a step allocates nothing.  Every arithmetic step is a library
call; this module only owns buffers and the call order.
"""
import torch

from . import (BACKWARD_BOTTOM_STAGED, BACKWARD_MASK_BOTTOM_DIFF, BACKWARD_POOL_MASK_OFFSETS,
               BACKWARD_TOP_DIFF_MASKED,
               BACKWARD_TOP_STAGED, CAFFE_BF16_F32_BOTTOM, CAFFE_F32, FORWARD_BOTTOM_STAGED,
               caffe_conv_backward_into, conv_stage_below_supported, pool_lrn_stage_supported,
               PASS_BACKWARD, PASS_BACKWARD_POOL_LRN, PASS_BACKWARD_WEIGHTS, PASS_FORWARD,
               POOL_LRN_STAGE_ONLY, POOL_MASK_OFFSETS, POOL_RELU_INPUT, Workspace,
               caffe_conv_backward,
               caffe_conv_backward_pool_lrn,
               caffe_conv_forward, conv_desc, conv_out_shape, lrn_desc,
               conv_workspace_size, lrn_backward, lrn_forward, maxpool_backward, maxpool_forward,
               lrn_pool_backward, pool_desc, pool_lrn_forward, pool_lrn_supported, relu_backward,
               pool_out_shape, sgd_learning_rate, sgd_update, softmax_loss)


class ConvStack:
    """layers: sequence of workloads.ConvLayer.  glue: {l: [("pool", {...}) | ("lrn", {...})]}
    applied in order to the output of layer l.  bf16=True runs the convolutions on
    bfloat16 operands (fp32 accumulation and outputs): bf16 weights, and each
    layer's float input rounded by the library as it stages it
    (CAFFE_BF16_F32_BOTTOM); glue stays fp32."""

    def __init__(self, layers, N, weights, biases, glue=None, bf16=False, device="cuda",
                 fuse_glue=True, split_backward=True, fuse_staging=True, chain_staging=True,
                 lrn_staging=True, lrn_stage_only=True, mask_offsets=True):
        self.layers = list(layers)
        self.N = N
        self.bf16 = bf16
        self.glue = glue or {}
        dev = torch.device(device)
        dt = CAFFE_BF16_F32_BOTTOM if bf16 else CAFFE_F32
        op = torch.bfloat16 if bf16 else torch.float32
        self.descs, self.W, self.b, self.dW, self.db = [], [], [], [], []
        self.top, self.dtop_glue, self.dbottom = [], [], []
        self.stages = []  # per layer: list of glue stage dicts
        # shape of layer l's output after its glue; an inner-product layer (a
        # 1x1 image) takes it flattened, channels (c, h, w) -- a view
        self.out_shape = []
        ws_need = 0
        ws_layer = []
        ws_weights = 0
        for l, L in enumerate(self.layers):
            d = conv_desc((N, L.C, L.H, L.W), (L.K, L.C // L.g, L.k, L.k), L.s, L.p, L.g, L.relu,
                          dt)
            Ho, Wo = conv_out_shape(d)
            self.descs.append(d)
            w = torch.as_tensor(weights[l], dtype=torch.float32).to(dev)
            self.W.append(w.to(op).contiguous())
            self.b.append(torch.as_tensor(biases[l], dtype=torch.float32).to(dev).contiguous())
            self.dW.append(torch.empty(w.shape, dtype=torch.float32, device=dev))
            self.db.append(torch.empty(L.K, dtype=torch.float32, device=dev))
            self.top.append(torch.empty((N, L.K, Ho, Wo), dtype=torch.float32, device=dev))
            self.dbottom.append(torch.empty((N, L.C, L.H, L.W), dtype=torch.float32, device=dev))
            need_l = max(conv_workspace_size(d, PASS_BACKWARD), conv_workspace_size(d, PASS_FORWARD))
            glue_l = [kind for kind, _ in self.glue.get(l, [])]
            if bf16 and fuse_staging and glue_l == ["pool", "lrn"]:
                need_l = max(need_l, conv_workspace_size(d, PASS_BACKWARD_POOL_LRN))
            ws_need = max(ws_need, need_l)
            ws_layer.append(need_l)
            ws_weights = max(ws_weights, conv_workspace_size(d, PASS_BACKWARD_WEIGHTS))
            cur = (N, L.K, Ho, Wo)
            stages = []
            for kind, prm in self.glue.get(l, []):
                st = dict(kind=kind, prm=dict(prm), in_shape=cur)
                if kind == "pool":
                    pd = pool_desc(cur, prm["kernel"], prm["stride"], prm.get("pad", 0))
                    ph, pw = pool_out_shape(pd)
                    cur = (N, cur[1], ph, pw)
                    st["mask"] = torch.empty(cur, dtype=torch.int32, device=dev)
                elif kind != "lrn":
                    raise ValueError(f"unknown glue layer {kind}")
                st["y"] = torch.empty(cur, dtype=torch.float32, device=dev)
                st["dx"] = torch.empty(st["in_shape"], dtype=torch.float32, device=dev)
                stages.append(st)
            self.stages.append(stages)
            self.out_shape.append(cur)
            if l + 1 < len(self.layers):
                nx = self.layers[l + 1]
                flat = nx.H == 1 and nx.W == 1 and cur[1] * cur[2] * cur[3] == nx.C
                if cur != (N, nx.C, nx.H, nx.W) and not flat:
                    raise ValueError(f"layer {l} output {cur} does not feed layer {l + 1}")
        # bf16: a workspace per layer, so that its backward reads the input
        # its forward staged there (BACKWARD_BOTTOM_STAGED); fp32 stages
        # nothing and all layers share one
        if bf16:
            self.ws_of = [Workspace(dev).get(n) for n in ws_layer]
        else:
            self.ws = Workspace(dev).get(ws_need)
            self.ws_of = [self.ws] * len(ws_layer)
        # fp32 backward: a layer whose top gradient arrives masked runs its
        # weight and bias gradients on a side stream (default priority, own
        # workspace) while the data gradient and the glue below it go on in
        # the caller's stream: the GEMMs fill each other's idle compute units
        # and the bandwidth-bound glue hides behind them (CaffeNet conv1-5,
        # N=256: 9.80 -> 9.39 ms per step).  A layer whose top gradient
        # arrives unmasked (the top layer) runs its ReLU's backward as a pass
        # of its own first, so that both calls take the masked gradient.
        # bf16 keeps one call per layer (both passes read the top gradient it
        # stages once) and hands the call the side stream for the weight
        # side (caffe_conv_backward_ex): the weight and bias gradients run
        # there, not joined per layer, beside the next layers' staging, glue
        # and data gradients.
        self.split_backward = split_backward and not bf16
        self.weight_side = split_backward and bf16
        # bf16: a layer whose bottom is the previous layer's top (no glue in
        # between) writes its data gradient straight into that layer's staged
        # top gradient (caffe_conv_backward_into) where the library supports
        # the pair, so the float gradient is neither stored nor staged again
        n_l = len(self.layers)
        self.stage_into = [False] * n_l
        if bf16 and chain_staging:
            for l in range(1, n_l):
                self.stage_into[l] = (not self.glue.get(l - 1) and not self.glue.get(l) and
                                      conv_stage_below_supported(self.descs[l],
                                                                 self.descs[l - 1]))
        self.top_from_above = [l + 1 < n_l and self.stage_into[l + 1] for l in range(n_l)]
        if self.split_backward or self.weight_side:
            self.side = torch.cuda.Stream(device=dev)
        if self.split_backward:
            self.ws_side = Workspace(dev).get(max(ws_weights, 1))
        # serial = True keeps the separate data- and weight-gradient calls but
        # issues both on the caller's stream (measurement: each call then has
        # the device to itself; the results are the same bits)
        self.serial = False
        self.bottom = [None] * len(self.layers)
        # Fused ReLU backward passes.  A ReLU output that feeds a max-pool gets
        # its backward folded into the pool's routing (CAFFE_POOL_RELU_INPUT);
        # one that feeds the next convolution directly gets it folded into
        # that layer's data gradient (CAFFE_BACKWARD_MASK_BOTTOM_DIFF).  Either
        # way the layer then receives an already masked top gradient.
        n = len(self.layers)
        self.pool_flags = [0] * n
        self.mask_bottom = [False] * n
        self.top_masked = [False] * n
        for l, L in enumerate(self.layers):
            if not L.relu:
                continue
            st = self.stages[l]
            if st and st[0]["kind"] == "pool":
                self.pool_flags[l] = POOL_RELU_INPUT
                self.top_masked[l] = True
            elif not st and l + 1 < n:
                self.mask_bottom[l + 1] = True
                self.top_masked[l] = True
        # masked top gradients of the layers whose ReLU backward runs as its
        # own pass (split backward only)
        self.dtop_relu = [torch.empty_like(self.top[l])
                          if self.split_backward and L.relu and not self.top_masked[l] else None
                          for l, L in enumerate(self.layers)]
        # A max-pool directly followed by an LRN runs as one fused pass each
        # way (the pooled gradient never stored) when the kernels take the
        # geometry; the LRN stage then has no "dx".
        self.fused = [False] * n
        for l in range(n):
            st = self.stages[l]
            if (fuse_glue and len(st) == 2 and st[0]["kind"] == "pool" and st[1]["kind"] == "lrn"):
                p, r = st[0]["prm"], st[1]["prm"]
                self.fused[l] = pool_lrn_supported(st[0]["in_shape"], p["kernel"], p["stride"],
                                                   p.get("pad", 0), r["size"], r["alpha"],
                                                   r["beta"], r["k"])
        # bf16: a layer whose output goes through the fused max-pool + LRN
        # hands the glue's backward to its own backward call, which writes
        # the bf16 staging of its top gradient directly (the float gradient
        # is never stored); dbottom of the glue stage is then not written
        self.fuse_staging = [bf16 and fuse_staging and self.fused[l] for l in range(n)]
        # bf16: a fused max-pool + LRN that feeds the next convolution also
        # writes that layer's bf16 staging as it forms the LRN output
        # (caffe_pool_lrn_forward_into), and the layer's forward then skips
        # its own staging pass (CAFFE_FORWARD_BOTTOM_STAGED)
        self.bottom_staged = [False] * n
        if bf16 and lrn_staging:
            for l in range(1, n):
                if self.fused[l - 1]:
                    pst, lst = self.stages[l - 1]
                    p, r = pst["prm"], lst["prm"]
                    self.bottom_staged[l] = pool_lrn_stage_supported(
                        pst["in_shape"], p["kernel"], p["stride"], p.get("pad", 0), r["size"],
                        r["alpha"], r["beta"], r["k"], self.descs[l])
        # ... and then writes only that staging, not its float output, when the
        # glue's backward is the fused one that forms the output again
        self.lrn_stage_only = [lrn_stage_only and l + 1 < n and self.bottom_staged[l + 1] and
                               self.fuse_staging[l] for l in range(n)]
        # A fused max-pool + LRN records each winner as a byte (its offset in
        # the window): only the fused backward passes read the mask
        self.mask_u8 = [False] * n
        for l in range(n):
            if mask_offsets and self.fused[l]:
                pst = self.stages[l][0]
                if pst["prm"]["kernel"] ** 2 <= 255:
                    self.mask_u8[l] = True
                    pst["mask"] = torch.empty(pst["mask"].shape, dtype=torch.uint8, device=dev)
        for l in range(n):
            if self.fuse_staging[l]:
                pst, lst = self.stages[l]
                p, r = pst["prm"], lst["prm"]
                pst["pool_desc"] = pool_desc(pst["in_shape"], p["kernel"], p["stride"],
                                             p.get("pad", 0))
                lst["lrn_desc"] = lrn_desc(pst["y"].shape, r["size"], r["alpha"], r["beta"],
                                           r["k"])
        # when a list, (tag, event) pairs are recorded around every conv call:
        # tag = (kind, layer, "begin" | "end") with kind "fwd" (forward),
        # "bwd" (data gradient), "wgt" (weight and bias gradients) or "both"
        # (both gradients in one call)
        self.events = None
        # with a set of (kind, layer) keys, only those calls are marked
        self.mark_only = None

    def _mark(self, tag, s):
        if self.events is not None and (self.mark_only is None or tag[:2] in self.mark_only):
            ev = torch.cuda.Event(enable_timing=True)
            ev.record(s)
            self.events.append((tag, ev))

    def forward(self, x, stream=None):
        """x: (N, C, H, W) float32 device tensor.  Returns the last layer's top."""
        s = stream or torch.cuda.current_stream()
        cur = x
        n_l = len(self.layers)
        for l in range(n_l):
            L = self.layers[l]
            cur = cur.view(self.N, L.C, L.H, L.W)
            self.bottom[l] = cur
            self._mark(("fwd", l, "begin"), s)
            caffe_conv_forward(self.descs[l], cur, self.W[l], self.b[l], self.top[l], self.ws_of[l],
                               s, flags=FORWARD_BOTTOM_STAGED if self.bottom_staged[l] else 0)
            self._mark(("fwd", l, "end"), s)
            cur = self.top[l]
            if self.fused[l]:
                pst, lst = self.stages[l]
                p, r = pst["prm"], lst["prm"]
                pst["x"], lst["x"] = cur, pst["y"]
                pool_lrn_forward(cur, p["kernel"], p["stride"], p.get("pad", 0), r["size"],
                                 r["alpha"], r["beta"], r["k"], pooled=pst["y"], mask=pst["mask"],
                                 out=lst["y"], stream=s,
                                 flags=self.pool_flags[l] |
                                 (POOL_LRN_STAGE_ONLY if self.lrn_stage_only[l] else 0) |
                                 (POOL_MASK_OFFSETS if self.mask_u8[l] else 0),
                                 stage_for=((self.descs[l + 1], self.ws_of[l + 1])
                                            if l + 1 < n_l and self.bottom_staged[l + 1]
                                            else None))
                cur = lst["y"]
                continue
            for st in self.stages[l]:
                p = st["prm"]
                st["x"] = cur
                if st["kind"] == "pool":
                    flags = self.pool_flags[l] if st is self.stages[l][0] else 0
                    maxpool_forward(cur, p["kernel"], p["stride"], p.get("pad", 0), out=st["y"],
                                    mask=st["mask"], flags=flags, stream=s)
                else:
                    lrn_forward(cur, p["size"], p["alpha"], p["beta"], p["k"], out=st["y"],
                                stream=s)
                cur = st["y"]
        return self.top[-1]

    def backward(self, top_diff, stream=None, data_grad_bottom=True):
        """top_diff: gradient w.r.t. the last top.  Fills dW, db and dbottom
        (dbottom[0] only when data_grad_bottom)."""
        s = stream or torch.cuda.current_stream()
        # (a captured graph keeps to one stream)
        capturing = torch.cuda.is_current_stream_capturing()
        split = self.split_backward and not capturing
        wside = self.side if self.weight_side and not capturing else None
        if split or wside is not None:
            self.side.wait_stream(s)
        g = top_diff
        for l in range(len(self.layers) - 1, -1, -1):
            L = self.layers[l]
            if g is not None:
                g = g.view(self.out_shape[l])
            if self.fuse_staging[l]:
                g = self._backward_pool_lrn(l, g, s, l > 0 or data_grad_bottom, wside)
                continue
            if self.stage_into[l] or self.top_from_above[l]:
                g = self._backward_staged(l, g, s, wside)
                continue
            if self.fused[l]:
                pst, lst = self.stages[l]
                p, r = pst["prm"], lst["prm"]
                g = lrn_pool_backward(pst["in_shape"], pst["y"], lst["y"], g, pst["mask"],
                                      p["kernel"], p["stride"], p.get("pad", 0), r["size"],
                                      r["alpha"], r["beta"], r["k"], out=pst["dx"], stream=s,
                                      flags=BACKWARD_POOL_MASK_OFFSETS if self.mask_u8[l] else 0)
            for st in (reversed(self.stages[l]) if not self.fused[l] else ()):
                p = st["prm"]
                if st["kind"] == "pool":
                    g = maxpool_backward(st["in_shape"], g, st["mask"], p["kernel"], p["stride"],
                                         p.get("pad", 0), out=st["dx"], stream=s)
                else:
                    g = lrn_backward(st["x"], st["y"], g, p["size"], p["alpha"], p["beta"],
                                     p["k"], out=st["dx"], stream=s)
            want_dx = l > 0 or data_grad_bottom
            bottom = self.bottom[l]
            flags = 0
            if self.top_masked[l]:
                flags |= BACKWARD_TOP_DIFF_MASKED
            if self.mask_bottom[l] and want_dx:
                flags |= BACKWARD_MASK_BOTTOM_DIFF
            if self.bf16:
                flags |= BACKWARD_BOTTOM_STAGED
            top = self.top[l] if L.relu else None
            if split and self.dtop_relu[l] is not None:
                g = relu_backward(self.top[l], g, out=self.dtop_relu[l], stream=s)
                flags |= BACKWARD_TOP_DIFF_MASKED
            if split and (flags & BACKWARD_TOP_DIFF_MASKED or not L.relu):
                ready = torch.cuda.Event()
                ready.record(s)
                # the data gradient (on the critical path) goes out first
                if want_dx:
                    self._mark(("bwd", l, "begin"), s)
                    caffe_conv_backward(self.descs[l], g, top, bottom, self.W[l],
                                        self.dbottom[l], None, None, 0, flags, self.ws_of[l], s)
                    self._mark(("bwd", l, "end"), s)
                if self.serial:
                    wstream, wspace = s, self.ws_of[l]
                else:
                    wstream, wspace = self.side, self.ws_side
                    wstream.wait_event(ready)
                self._mark(("wgt", l, "begin"), wstream)
                caffe_conv_backward(self.descs[l], g, top, bottom, self.W[l], None, self.dW[l],
                                    self.db[l], 0, flags, wspace, wstream)
                self._mark(("wgt", l, "end"), wstream)
            else:
                # one call for both gradients ("both"), or for the weight
                # gradient alone ("wgt") when no data gradient is wanted
                tag = "both" if want_dx else "wgt"
                self._mark((tag, l, "begin"), s)
                caffe_conv_backward(self.descs[l], g, top, bottom, self.W[l],
                                    self.dbottom[l] if want_dx else None, self.dW[l], self.db[l],
                                    0, flags, self.ws_of[l], s, weight_stream=wside)
                self._mark((tag, l, "end"), s)
                if wside is not None:  # (the call ends with the later of the two)
                    self._mark((tag, l, "end"), wside)
            g = self.dbottom[l]
        if split or wside is not None:
            # the next forward overwrites what the side stream reads
            s.wait_stream(self.side)
        return self.dbottom[0]

    def _backward_staged(self, l, g, s, wside):
        """bf16 layer l with its top gradient staged by the layer above and/or
        its data gradient staged into the layer below; returns the float top
        gradient of the layer below, or None when it is staged."""
        L = self.layers[l]
        flags = BACKWARD_BOTTOM_STAGED
        if self.top_masked[l]:
            flags |= BACKWARD_TOP_DIFF_MASKED
        if self.top_from_above[l]:
            flags |= BACKWARD_TOP_STAGED
            g = None
        else:
            g = g.view(self.out_shape[l])
        if self.mask_bottom[l]:
            flags |= BACKWARD_MASK_BOTTOM_DIFF
        top = self.top[l] if L.relu else None
        self._mark(("both", l, "begin"), s)
        if self.stage_into[l]:
            caffe_conv_backward_into(self.descs[l], g, top, self.bottom[l], self.W[l], self.dW[l],
                                     self.db[l], 0, flags, self.ws_of[l], self.descs[l - 1],
                                     self.ws_of[l - 1], s, weight_stream=wside)
            out = None
        else:
            caffe_conv_backward(self.descs[l], g, top, self.bottom[l], self.W[l],
                                self.dbottom[l], self.dW[l], self.db[l], 0, flags, self.ws_of[l],
                                s, weight_stream=wside)
            out = self.dbottom[l]
        self._mark(("both", l, "end"), s)
        if wside is not None:  # (the call ends with the later of the two)
            self._mark(("both", l, "end"), wside)
        return out

    def _backward_pool_lrn(self, l, g, s, want_dx, wside=None):
        """Layer l's backward from the gradient g of the LRN after its max-pool
        (one call: the glue's backward staged as the bf16 top gradient)."""
        pst, lst = self.stages[l]
        L = self.layers[l]
        flags = BACKWARD_BOTTOM_STAGED
        if self.mask_u8[l]:
            flags |= BACKWARD_POOL_MASK_OFFSETS
        if self.top_masked[l]:
            flags |= BACKWARD_TOP_DIFF_MASKED
        if self.mask_bottom[l] and want_dx:
            flags |= BACKWARD_MASK_BOTTOM_DIFF
        self._mark(("both" if want_dx else "wgt", l, "begin"), s)
        caffe_conv_backward_pool_lrn(self.descs[l], pst["pool_desc"], lst["lrn_desc"], pst["y"],
                                     lst["y"], g, pst["mask"], self.top[l] if L.relu else None,
                                     self.bottom[l], self.W[l],
                                     self.dbottom[l] if want_dx else None, self.dW[l],
                                     self.db[l], 0, flags, self.ws_of[l], s,
                                     weight_stream=wside)
        self._mark(("both" if want_dx else "wgt", l, "end"), s)
        if wside is not None:  # (the call ends with the later of the two)
            self._mark(("both" if want_dx else "wgt", l, "end"), wside)
        return self.dbottom[l]

    def layer_top_diff(self, l, top_diff_last):
        """Gradient that layer l received in the last backward (after its glue)."""
        if l == len(self.layers) - 1:
            return top_diff_last
        if self.fuse_staging[l] or self.top_from_above[l]:
            raise ValueError(f"layer {l}'s top gradient is staged in bf16 only (fuse_staging, "
                             "chain_staging)")
        st = self.stages[l]
        return st[0]["dx"] if st else self.dbottom[l + 1].view(self.top[l].shape)


class SGDTrainer:
    """Training of a ConvStack that ends in class scores (Sec. 3.4): each
    iteration runs the forward pass, the softmax loss and its gradient, the
    backward pass (no data gradient for the input batch) and one SGD update
    of every weight and bias blob at the schedule's learning rate.  The
    momentum histories start at zero; all blobs share one rate and decay."""

    def __init__(self, net, policy="inv", base_lr=0.01, gamma=1e-4, power=0.75, stepsize=1,
                 momentum=0.9, weight_decay=5e-4):
        if net.bf16:
            raise ValueError("SGDTrainer runs fp32 networks")
        self.net = net
        self.schedule = dict(policy=policy, base_lr=base_lr, gamma=gamma, power=power,
                             stepsize=stepsize)
        self.momentum = momentum
        self.weight_decay = weight_decay
        self.vW = [torch.zeros_like(w) for w in net.W]
        self.vb = [torch.zeros_like(b) for b in net.b]
        dev = net.W[0].device
        top = net.top[-1]
        self.loss = torch.empty(1, dtype=torch.float32, device=dev)
        self.sample_loss = torch.empty(net.N, dtype=torch.float32, device=dev)
        self.scores_diff = torch.empty(top.shape, dtype=torch.float32, device=dev)
        self.iter = 0

    def forward_backward(self, x, labels, stream=None):
        """Loss and every parameter gradient of the batch; returns the loss (1,)."""
        s = stream or torch.cuda.current_stream()
        scores = self.net.forward(x, s)
        softmax_loss(scores, labels, out=(self.loss, self.sample_loss, None, self.scores_diff),
                     stream=s)
        self.net.backward(self.scores_diff, s, data_grad_bottom=False)
        return self.loss

    def update(self, stream=None):
        """One SGD step of every blob at iteration self.iter's rate."""
        s = stream or torch.cuda.current_stream()
        lr = sgd_learning_rate(it=self.iter, **self.schedule)
        for l in range(len(self.net.layers)):
            sgd_update(self.net.W[l], self.net.dW[l], self.vW[l], lr, self.momentum,
                       self.weight_decay, stream=s)
            sgd_update(self.net.b[l], self.net.db[l], self.vb[l], lr, self.momentum,
                       self.weight_decay, stream=s)
        self.iter += 1
        return lr

    def step(self, x, labels, stream=None):
        loss = self.forward_backward(x, labels, stream)
        self.update(stream)
        return loss

    # ------------------------------------------------------------ HIP graph
    def capture(self, x, labels):
        """Record one whole iteration -- forward, loss, backward and the
        updates, with the learning rate read from device memory -- as a HIP
        graph over the static batch buffers x and labels (which must stay
        allocated; refill them in place to train on other batches).  Every
        buffer the iteration touches is preallocated and no call in it
        allocates or records a memset, so replays rerun the same launches."""
        dev = self.net.W[0].device
        self.lr_dev = torch.empty(1, dtype=torch.float32, device=dev)
        # one eager pass first, so every host-side plan query happens before
        # capture (it leaves only gradients behind, which the graph rewrites)
        self.forward_backward(x, labels)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            s = torch.cuda.current_stream()
            self.forward_backward(x, labels, s)
            for l in range(len(self.net.layers)):
                sgd_update(self.net.W[l], self.net.dW[l], self.vW[l], self.lr_dev, self.momentum,
                           self.weight_decay, stream=s)
                sgd_update(self.net.b[l], self.net.db[l], self.vb[l], self.lr_dev, self.momentum,
                           self.weight_decay, stream=s)
        self.graph = g
        return g

    def replay(self):
        """One iteration through the captured graph at iteration self.iter's
        rate (written to device memory before the replay, outside the graph)."""
        lr = sgd_learning_rate(it=self.iter, **self.schedule)
        self.lr_dev.fill_(lr)
        self.graph.replay()
        self.iter += 1
        return self.loss
