"""ResNet18 (BasicBlock) forward pass over ESB codes on one GPU.

Every convolution and the classifier are quantized layers of Sec. 5 (the paper
quantizes all layers of ResNet18, including the first and the last): the
layer input is scaled by DDA (eq. (13)) over the candidate grid
alpha_j = 2^E c_j, c_j = fl32((j+1) / (64 C)), j = 0..63, with C the largest
set value and E the binary exponent of max|x| (2^(E-1) <= max|x| < 2^E), so
that the grid spans (0, 2^E / C], past max|x| / C by less than a factor of
two; projected to ESB codes (eq. (8)) and contracted with the pre-quantized
weights (eq. (15)) into fp32 outputs.  Scaling every candidate by a power of
two scales its exact thresholds by the same power, so the DDA's grid-only
set-up is built once (esb_dda_plan) and every call only shifts it
(esb_quantize_planned: the planned DDA and the projection in one call).  Weights
are quantized once, the same way, when the model is built.

Every step runs in the library's kernels; torch only holds the buffers (and
clears the running maxima at the start of a pass).  The ReLUs and the residual
additions run in the convolutions' epilogues (esb_conv2d_post: the same fp32
operations), which also raise a device scalar to the max |x| of the next
layer's input, so that its DDA grid (esb_dda_job.grid_scale) needs no separate
reduction; the image's maximum comes from esb_absmax.  conv1, its ReLU and the
3x3 / stride-2 max pool are one call (esb_conv2d_relu_maxpool: only the pooled
output is written; the pool keeps the maximum: the ReLU'd values are >= 0 and
every element lies in some window) and the global average pool
esb_avgpool_global (a float64 sum of the 7x7 positions in order, divided by 49
and rounded to fp32 once), which raises the maximum of the pooled features.
No batch normalization (the weights are He-initialized).

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
        self.units = None
        self.calib = {}   # layer name -> device scale of its input, from the last forward()
        dev = "cuda"
        self.cmax = value_max(n, k_sig)
        self.cgrid = torch.from_numpy(workloads.maxabs_grid_factors(self.cmax, GRID_POINTS)).to(dev)
        self.plan = esb.esb_dda_plan(n, k_sig, self.cgrid, stream=self.sh)
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
        L1 = self.layers["conv1"]
        pneed = esb.esb_conv2d_relu_maxpool_workspace_size(
            (batch, 224, 224, 3), (L1["cout"], L1["k"], L1["k"], 3), n, k_sig, n, k_sig,
            stride=(L1["stride"],) * 2, pad=(L1["pad"],) * 2)
        self.pool_ws = torch.empty(pneed, dtype=torch.uint8, device=dev) if pneed else None
        self.amax = torch.zeros(32, dtype=torch.float32, device=dev)   # max |x| per layer input
        self.spare = torch.zeros(1, dtype=torch.float32, device=dev)   # max |x| for _quantize(x)
        # weights, quantized once: every tensor's DDA and projection as one batch
        names = list(self.layers) + ["fc"]
        ws = [torch.from_numpy(np.ascontiguousarray(weights[nm])).to(dev) for nm in names]
        wmax = torch.zeros(len(ws), dtype=torch.float32, device=dev)
        alphas = [torch.empty(1, dtype=torch.float32, device=dev) for _ in ws]
        codes = [torch.empty(w.shape, dtype=torch.uint8, device=dev) for w in ws]
        wsw = torch.empty(max(max(esb.esb_dda_workspace_size(w.numel(), n, k_sig, GRID_POINTS)
                                  for w in ws), 1), dtype=torch.uint8, device=dev)
        for i, (w, a_) in enumerate(zip(ws, alphas)):
            esb.esb_absmax(w, wmax[i:i + 1], stream=self.sh)
            esb.esb_dda_align_planned(w, n, k_sig, self.plan, GRID_POINTS, wmax[i:i + 1],
                                      alpha_out=a_, workspace=wsw, stream=self.sh, want_D=False)
        esb.esb_project_batch(esb.project_jobs([(w, a_, n, k_sig, c) for w, a_, c in
                                                zip(ws, alphas, codes)]), stream=self.sh)
        for nm, a_, c in zip(names, alphas, codes):
            if nm == "fc":
                self.fc_alpha, self.fc_codes = a_, c
            else:
                self.layers[nm]["alpha"], self.layers[nm]["codes"] = a_, c
        torch.cuda.synchronize()

    def _call(self, kind, label, fn, nbytes=0.0, ops=0.0):
        """Run one library call.  While self.units is a list (a forward run for the bench),
        the call is bracketed by two timing events on the model's stream and kept there with
        its algorithmic bytes and operations; fn writes only into buffers allocated before it,
        so running it again repeats the same work."""
        if self.units is None:
            return fn()
        torch = self.torch
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        st = self.stream if self.stream is not None else torch.cuda.current_stream()
        e0.record(st)
        out = fn()
        e1.record(st)
        self.units.append(dict(kind=kind, label=label, fn=fn, bytes=float(nbytes),
                               ops=float(ops), events=(e0, e1)))
        return out

    def _quantize(self, x, ws, xmax=None, label=""):
        """DDA over alpha_j = 2^E c_j, E the binary exponent of the device scalar xmax (the
        plan's tables shifted by E), then the projection, in one call (esb_quantize_planned).
        xmax: a device scalar already holding max|x| (from the producing epilogue), else
        esb_absmax."""
        torch = self.torch
        alpha = torch.empty(1, dtype=torch.float32, device=x.device)
        codes = torch.empty(x.shape, dtype=torch.uint8, device=x.device)
        nel = x.numel()
        if xmax is None:
            xmax = self.spare
            xmax.zero_()
            self._call("absmax", label, lambda: esb.esb_absmax(x, xmax, stream=self.sh), 4 * nel)
        # one call: the DDA's pass (4 B per element read), then the projection (4 B read,
        # 1 B written), its blocks choosing alpha themselves
        self._call("quantize", label,
                   lambda: esb.esb_quantize_planned(x, self.n, self.ks, self.plan, GRID_POINTS,
                                                    xmax, alpha_out=alpha, codes=codes,
                                                    workspace=ws, stream=self.sh, want_D=False),
                   9 * nel)
        return alpha, codes

    def conv(self, name, x, quantized=None, xmax=None, residual=None, relu=False, absmax=None):
        """The layer on input x; `quantized` = (alpha, codes) of x when another layer
        already quantized this same tensor (the DDA and the projection depend on x only);
        xmax: device max|x| for the DDA grid.  With residual / relu / absmax the epilogue adds
        the residual, applies the ReLU and raises absmax to the max |output|."""
        torch = self.torch
        L = self.layers[name]
        ax, cx = quantized if quantized is not None else self._quantize(x, self.ws[name], xmax,
                                                                        name)
        Nb, H, W, C = cx.shape
        st, pd = (L["stride"],) * 2, (L["pad"],) * 2
        P, Q = esb.conv_out_hw(H, W, L["k"], L["k"], st, pd)
        y = torch.empty((Nb, P, Q, L["cout"]), dtype=torch.float32, device=cx.device)
        acc = (torch.empty((Nb, P, Q, L["cout"]), dtype=torch.int32, device=cx.device)
               if self.record else None)
        ops = 2.0 * Nb * P * Q * L["cout"] * L["k"] * L["k"] * C
        nbytes = cx.numel() + L["codes"].numel() + 4 * y.numel() * (2 if residual is not None else 1)
        if residual is None and not relu and absmax is None:
            fn = lambda: esb.esb_conv2d(cx, self.n, self.ks, ax, L["codes"], self.n, self.ks,
                                        L["alpha"], stride=st, pad=pd, acc=acc, y=y,
                                        want_acc=self.record, stream=self.sh, workspace=self.cws)
        else:
            fn = lambda: esb.esb_conv2d_post(
                cx, self.n, self.ks, ax, L["codes"], self.n, self.ks, L["alpha"], None, self.n,
                self.ks, residual=residual, relu=relu, stride=st, pad=pd, want_codes=False,
                acc=acc, want_acc=self.record, y=y, stream=self.sh, workspace=self.cws,
                absmax=absmax)
        self._call("contraction", name, fn, nbytes, ops)
        if self.record:
            self.trace.append(dict(name=name, x=x, alpha=ax, codes=cx, acc=acc, y=y))
        self.calib[name] = ax
        self.last_q = (ax, cx)
        return y

    def stem(self, x, xmax, absmax, out_alpha=None):
        """conv1 with its ReLU and the 3x3 / stride-2 / pad-1 max pool in one call
        (esb_conv2d_relu_maxpool): only the pooled output is written (and raises absmax),
        as fp32 and, with out_alpha, as the next layer's codes.  xmax: the input's max|x|
        for its DDA, or None when calib["conv1"] already holds the input's scale."""
        torch = self.torch
        L = self.layers["conv1"]
        if xmax is None:
            ax = self.calib["conv1"]
            cx = esb.esb_project(x, ax, self.n, self.ks, stream=self.sh)
        else:
            ax, cx = self._quantize(x, self.ws["conv1"], xmax, "conv1")
        Nb, H, W, C = cx.shape
        st, pd = (L["stride"],) * 2, (L["pad"],) * 2
        P, Q = esb.conv_out_hw(H, W, L["k"], L["k"], st, pd)
        PP, QQ = esb.conv_out_hw(P, Q, 3, 3, (2, 2), (1, 1))
        pooled = torch.empty((Nb, PP, QQ, L["cout"]), dtype=torch.float32, device=cx.device)
        codes = (torch.empty((Nb, PP, QQ, L["cout"]), dtype=torch.uint8, device=cx.device)
                 if out_alpha is not None else None)
        ops = 2.0 * Nb * P * Q * L["cout"] * L["k"] * L["k"] * C
        nbytes = cx.numel() + L["codes"].numel() + 4 * pooled.numel() + (
            codes.numel() if codes is not None else 0)
        self._call("contraction", "conv1",
                   lambda: esb.esb_conv2d_relu_maxpool(
                       cx, self.n, self.ks, ax, L["codes"], self.n, self.ks, L["alpha"],
                       out_alpha=out_alpha, out_n=self.n, out_k_sig=self.ks, stride=st, pad=pd,
                       y=pooled, codes=codes, want_codes=codes is not None, absmax=absmax,
                       workspace=self.pool_ws, stream=self.sh),
                   nbytes, ops)
        if self.record:   # the full-resolution output, for the layer-by-layer comparison
            self.units = None
            acc, y, _ = esb.esb_conv2d_post(cx, self.n, self.ks, ax, L["codes"], self.n, self.ks,
                                            L["alpha"], None, self.n, self.ks, relu=True,
                                            stride=st, pad=pd, want_codes=False, want_acc=True,
                                            want_y=True, stream=self.sh, workspace=self.cws)
            self.trace.append(dict(name="conv1", x=x, alpha=ax, codes=cx, acc=acc, y=y,
                                   pooled=pooled))
        self.calib["conv1"] = ax
        return pooled if codes is None else (pooled, codes)

    def forward(self, x, units=None):
        """The forward pass with per-layer DDA; units: a list that receives every library call
        of the pass (see _call)."""
        torch = self.torch
        self.units = units
        self.amax.zero_()
        slots = iter(range(self.amax.numel()))

        def slot():
            i = next(slots)
            return self.amax[i:i + 1]

        m0 = slot()
        self._call("absmax", "image", lambda: esb.esb_absmax(x, m0, stream=self.sh), 4 * x.numel())
        m = slot()
        a = self.stem(x, m0, m)
        self.units = units
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
        mf = slot()
        feat = torch.empty((a.shape[0], a.shape[3]), dtype=torch.float32, device=a.device)
        a_last = a
        self._call("avgpool", "head",
                   lambda: esb.esb_avgpool_global(a_last, out=feat, absmax=mf, stream=self.sh),
                   4 * (a_last.numel() + feat.numel()))
        af, cf = self._quantize(feat, self.ws["fc"], xmax=mf, label="fc")
        self.calib["fc"] = af
        M, K = cf.shape
        Nf = self.fc_codes.shape[0]
        logits = torch.empty((M, Nf), dtype=torch.float32, device=cf.device)
        acc = torch.empty((M, Nf), dtype=torch.int32, device=cf.device) if self.record else None
        self._call("contraction", "fc",
                   lambda: esb.esb_gemm(cf, self.n, self.ks, af, self.fc_codes, self.n, self.ks,
                                        self.fc_alpha, acc=acc, y=logits, want_acc=self.record,
                                        stream=self.sh, workspace=self.cws),
                   M * K + Nf * K + 4 * M * Nf, 2.0 * M * Nf * K)
        if self.record:
            self.trace.append(dict(name="fc", x=feat, alpha=af, codes=cf, acc=acc, y=logits))
        self.units = None
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
        A = self.calib
        if "fc" not in A:
            raise RuntimeError("forward_fused needs the scales of a forward() first")
        a, ca = self.stem(x, None, None, out_alpha=A["l1.0.c1"])
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
        feat = esb.esb_avgpool_global(a, stream=self.sh)
        cf = esb.esb_project(feat, A["fc"], self.n, self.ks, stream=self.sh)
        _, logits = esb.esb_gemm(cf, self.n, self.ks, A["fc"], self.fc_codes, self.n, self.ks,
                                 self.fc_alpha, want_acc=False, stream=self.sh, workspace=self.cws)
        return logits
