"""ResNet18 (BasicBlock) forward pass over ESB codes on one GPU.

Every convolution and the classifier are quantized layers of Sec. 5 (the paper
quantizes all layers of ResNet18, including the first and the last): the
layer input is scaled by DDA (eq. (13)) over the candidate grid
alpha_j = fl32(max|x| * c_j), c_j = fl32((j+1) / (64 C)), j = 0..63 (C the
largest set value, so the grid spans (0, max|x| / C]), projected to ESB codes
(eq. (8)) and contracted with the pre-quantized weights (eq. (15)) into fp32
outputs.  Weights are quantized once, the same way, when the model is built.

Only the library's calls touch the ESB arithmetic.  The ReLUs and the
residual additions run in the convolutions' epilogues (esb_conv2d_post: the
same fp32 operations), which also raise a device scalar to the max |x| of the
next layer's input, so that its DDA grid needs no separate reduction; the
3x3 / stride-2 max pool after conv1 and the global average pool are torch on
the same stream (the pool keeps the maximum: the ReLU'd values are >= 0 and
every element lies in some window).  The average is a float64 sum of the 7x7
window divided by 49 and rounded to fp32 once.  No batch normalization (the
weights are He-initialized).

A downsample conv reads the same block input as the block's first conv, so it
reuses that conv's alpha and codes instead of quantizing the tensor again.

Activations are NHWC fp32; codes NHWC uint8; weights KRSC.

forward_fused(x) is the inference flow of the paper (Alg. 1 at inference, Sec.
4.2): every layer input's scale is fixed beforehand (here: the scales the DDA
chose in the last forward(), the calibration), so each contraction's epilogue
applies the ReLU and the residual sum and writes the next layer's codes
directly (esb_conv2d_post); fp32 activations are written only where the glue
needs them (the max pool input, the identity of the next block, the average
pool input).  On the calibration batch its logits equal forward()'s bit for bit.
"""
import numpy as np

from . import esb, workloads

N_BITS, K_SIG = 5, 3      # ESB(5, 2) for every layer
GRID_POINTS = 64


def value_max(n, k_sig):
    return float(np.max(esb.esb_valueset(n, k_sig)))


def input_side(name):
    """Height (= width) of a layer's input for 224 x 224 images."""
    if name == "conv1":
        return 224
    stage, blk, conv = name.split(".")
    first = {"l1": 56, "l2": 56, "l3": 28, "l4": 14}[stage]   # the stage's input
    inner = {"l1": 56, "l2": 28, "l3": 14, "l4": 7}[stage]    # after its first conv
    return first if (blk == "0" and conv in ("c1", "ds")) else inner


class ResNet18ESB:
    """Pre-quantized ResNet18; forward(x) returns the fp32 logits [batch, 1000]."""

    def __init__(self, weights, batch, n=N_BITS, k_sig=K_SIG, stream=None, record=False):
        import torch
        self.torch = torch
        self.n, self.ks = n, k_sig
        self.batch = batch
        self.stream = stream
        self.sh = stream.cuda_stream if stream is not None else None
        self.record = record
        self.trace = []
        self.calib = {}   # layer name -> device scale of its input, from the last forward()
        dev = "cuda"
        self.cmax = value_max(n, k_sig)
        self.cgrid = torch.from_numpy(workloads.maxabs_grid_factors(self.cmax, GRID_POINTS)).to(dev)
        self.layers = {}
        sizes = {}
        for name, cin, cout, k, st, pd in workloads.RESNET18_CONVS:
            self.layers[name] = dict(cin=cin, cout=cout, k=k, stride=st, pad=pd)
            sizes[name] = batch * input_side(name) ** 2 * cin
        sizes["fc"] = batch * 512
        self.ws = {k: torch.empty(max(esb.esb_dda_workspace_size(v, n, k_sig, GRID_POINTS), 1),
                                  dtype=torch.uint8, device=dev) for k, v in sizes.items()}
        # one contraction workspace for every layer (they run one after the other
        # on one stream): operands decoded once where the layer has the work for it
        need = esb.esb_gemm_workspace_size(batch, 1000, 512, n, k_sig, n, k_sig)
        for name, L in self.layers.items():
            side = input_side(name)
            need = max(need, esb.esb_conv2d_workspace_size(
                (batch, side, side, L["cin"]), (L["cout"], L["k"], L["k"], L["cin"]), n, k_sig, n,
                k_sig, stride=(L["stride"],) * 2, pad=(L["pad"],) * 2))
        self.cws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
        self.amax = torch.zeros(32, dtype=torch.float32, device=dev)   # max |x| per layer input
        # weights, quantized once: every tensor's DDA and projection as one batch
        names = list(self.layers) + ["fc"]
        ws = [torch.from_numpy(np.ascontiguousarray(weights[nm])).to(dev) for nm in names]
        grids = [self.grid(w) for w in ws]
        alphas = [torch.empty(1, dtype=torch.float32, device=dev) for _ in ws]
        codes = [torch.empty(w.shape, dtype=torch.uint8, device=dev) for w in ws]
        jobs = esb.dda_jobs([(w, n, k_sig, g, a_, None) for w, g, a_ in zip(ws, grids, alphas)])
        wsb = torch.empty(max(esb.esb_dda_batch_workspace_size(jobs), 1), dtype=torch.uint8,
                          device=dev)
        esb.esb_dda_align_batch(jobs, wsb, stream=self.sh)
        esb.esb_project_batch(esb.project_jobs([(w, a_, n, k_sig, c) for w, a_, c in
                                                zip(ws, alphas, codes)]), stream=self.sh)
        for nm, a_, c in zip(names, alphas, codes):
            if nm == "fc":
                self.fc_alpha, self.fc_codes = a_, c
            else:
                self.layers[nm]["alpha"], self.layers[nm]["codes"] = a_, c
        torch.cuda.synchronize()

    def grid(self, x, xmax=None):
        """alpha_j = fl32(max|x| * c_j) on the device (one correctly rounded product); xmax:
        a device scalar already holding max|x| (from the producing epilogue)."""
        m = self.torch.linalg.vector_norm(x, float("inf")) if xmax is None else xmax
        return m.reshape(1) * self.cgrid

    def _quantize(self, x, ws, xmax=None):
        torch = self.torch
        alpha = torch.empty(1, dtype=torch.float32, device=x.device)
        if xmax is None:
            g = self.grid(x)
            esb.esb_dda_align(x, self.n, self.ks, g, alpha_out=alpha, D_out=None, workspace=ws,
                              stream=self.sh, want_D=False)
        else:   # the DDA scales the factors by the device max|x| itself (same single rounding)
            jobs = esb.dda_jobs([(x, self.n, self.ks, self.cgrid, alpha, None, xmax)])
            esb.esb_dda_align_batch(jobs, ws, stream=self.sh)
        codes = esb.esb_project(x, alpha, self.n, self.ks, stream=self.sh)
        return alpha, codes

    def conv(self, name, x, quantized=None, xmax=None, residual=None, relu=False, absmax=None):
        """The layer on input x; `quantized` = (alpha, codes) of x when another layer
        already quantized this same tensor (the DDA and the projection depend on x only);
        xmax: device max|x| for the DDA grid.  With residual / relu / absmax the epilogue adds
        the residual, applies the ReLU and raises absmax to the max |output|."""
        L = self.layers[name]
        ax, cx = quantized if quantized is not None else self._quantize(x, self.ws[name], xmax)
        if residual is None and not relu and absmax is None:
            acc, y = esb.esb_conv2d(cx, self.n, self.ks, ax, L["codes"], self.n, self.ks,
                                    L["alpha"], stride=(L["stride"],) * 2, pad=(L["pad"],) * 2,
                                    want_acc=self.record, stream=self.sh, workspace=self.cws)
        else:
            acc, y, _ = esb.esb_conv2d_post(
                cx, self.n, self.ks, ax, L["codes"], self.n, self.ks, L["alpha"], None, self.n,
                self.ks, residual=residual, relu=relu, stride=(L["stride"],) * 2,
                pad=(L["pad"],) * 2, want_codes=False, want_acc=self.record, want_y=True,
                stream=self.sh, workspace=self.cws, absmax=absmax)
        if self.record:
            self.trace.append(dict(name=name, x=x, alpha=ax, codes=cx, acc=acc, y=y))
        self.calib[name] = ax
        self.last_q = (ax, cx)
        return y

    def forward(self, x):
        torch = self.torch
        F = torch.nn.functional
        self.amax.zero_()
        slots = iter(range(self.amax.numel()))

        def slot():
            i = next(slots)
            return self.amax[i:i + 1]

        m = slot()
        a = self.conv("conv1", x, relu=True, absmax=m)
        # 3x3 max pool, stride 2, pad 1 (padding never wins: -inf); max|a| is unchanged
        a = F.max_pool2d(a.permute(0, 3, 1, 2), 3, 2, 1).permute(0, 2, 3, 1).contiguous()
        for stage in (1, 2, 3, 4):
            for blk in (0, 1):
                p = "l%d.%d." % (stage, blk)
                m1 = slot()
                out = self.conv(p + "c1", a, xmax=m, relu=True, absmax=m1)
                qa = self.last_q                     # the block input, quantized for c1
                # the downsample conv reads the same block input: its quantization is reused
                sc = self.conv(p + "ds", a, quantized=qa) if (p + "ds") in self.layers else a
                m = slot()
                a = self.conv(p + "c2", out, xmax=m1, residual=sc, relu=True, absmax=m)
        feat = (a.double().sum(dim=(1, 2)) / float(a.shape[1] * a.shape[2])).float().contiguous()
        af, cf = self._quantize(feat, self.ws["fc"])
        self.calib["fc"] = af
        acc, logits = esb.esb_gemm(cf, self.n, self.ks, af, self.fc_codes, self.n, self.ks,
                                   self.fc_alpha, want_acc=self.record, stream=self.sh,
                                   workspace=self.cws)
        if self.record:
            self.trace.append(dict(name="fc", x=feat, alpha=af, codes=cf, acc=acc, y=logits))
        return logits

    def conv_post(self, name, cx, out_alpha=None, residual=None, relu=False, want_y=False):
        """The layer on input codes cx (scale calib[name]), with the fused epilogue: ReLU,
        residual, and the next layer's codes under out_alpha when it is given."""
        L = self.layers[name]
        _, y, codes = esb.esb_conv2d_post(
            cx, self.n, self.ks, self.calib[name], L["codes"], self.n, self.ks, L["alpha"],
            out_alpha, self.n, self.ks, residual=residual, relu=relu,
            stride=(L["stride"],) * 2, pad=(L["pad"],) * 2, want_codes=out_alpha is not None,
            want_y=want_y, stream=self.sh, workspace=self.cws)
        return y, codes

    def forward_fused(self, x):
        """Forward pass with the scales of the last forward() fixed (see the module notes)."""
        torch = self.torch
        F = torch.nn.functional
        A = self.calib
        if "fc" not in A:
            raise RuntimeError("forward_fused needs the scales of a forward() first")
        cx = esb.esb_project(x, A["conv1"], self.n, self.ks, stream=self.sh)
        a, _ = self.conv_post("conv1", cx, relu=True, want_y=True)
        a = F.max_pool2d(a.permute(0, 3, 1, 2), 3, 2, 1).permute(0, 2, 3, 1).contiguous()
        ca = esb.esb_project(a, A["l1.0.c1"], self.n, self.ks, stream=self.sh)
        blocks = [(s, b) for s in (1, 2, 3, 4) for b in (0, 1)]
        for i, (stage, blk) in enumerate(blocks):
            p = "l%d.%d." % (stage, blk)
            _, mid = self.conv_post(p + "c1", ca, out_alpha=A[p + "c2"], relu=True)
            if (p + "ds") in self.layers:   # reads the block input's codes (scale of c1)
                L = self.layers[p + "ds"]
                _, sc = esb.esb_conv2d(ca, self.n, self.ks, A[p + "c1"], L["codes"], self.n,
                                       self.ks, L["alpha"], stride=(L["stride"],) * 2,
                                       pad=(L["pad"],) * 2, want_acc=False, stream=self.sh,
                                       workspace=self.cws)
            else:
                sc = a
            nxt = None
            if i + 1 < len(blocks):
                nxt = A["l%d.%d.c1" % blocks[i + 1]]
            a, ca = self.conv_post(p + "c2", mid, out_alpha=nxt, residual=sc, relu=True,
                                   want_y=True)
        feat = (a.double().sum(dim=(1, 2)) / float(a.shape[1] * a.shape[2])).float().contiguous()
        cf = esb.esb_project(feat, A["fc"], self.n, self.ks, stream=self.sh)
        _, logits = esb.esb_gemm(cf, self.n, self.ks, A["fc"], self.fc_codes, self.n, self.ks,
                                 self.fc_alpha, want_acc=False, stream=self.sh, workspace=self.cws)
        return logits
