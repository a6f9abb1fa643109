"""A whole MobileNet v1 forward pass on the library's kernels.

Layer sequence (paper Sec. 3.1, Sec. 3.3 and Table 1): the dense 3x3 stride-2
convolution reads the HWC image and writes CHW (``spconv_conv3x3_hwc``,
ReLU6); 13 blocks of depthwise 3x3 -> sparse 1x1 (ReLU6 after each), each
either one fused plan (``spconv_plan_create_fused``) or
``spconv_depthwise3x3`` followed by a plain plan (whose automatic kernel
choice applies); global average pooling (``spconv_global_avg_pool``); the
dense classifier (``spconv_linear``, no activation).

Both forms of a block compute the same fp32 operations in the same order
(the depthwise taps in dy, dx order from zero, bias, clamp; each 1x1 output
summed in ascending channel order), so they give the same bits and the
choice is a matter of speed only.  ``fuse="auto"`` times both forms once on
the device at construction and keeps the faster; ``"always"`` fuses every
block that a fused plan supports (a block whose input strip does not fit in
LDS, the 1024-channel one, is never fused); ``"never"`` runs every block as
two launches.

Every step is one kernel launch on the caller's (torch's current) stream;
nothing is allocated after construction.  ``capture`` records the whole
sequence into one graph (torch.cuda.CUDAGraph over HIP graphs) and
``replay`` launches it.  This module only orders the launches and owns the
buffers; every arithmetic step runs in libspconv's kernels.
"""

from __future__ import annotations

from typing import List, Optional

from .spconv import (E_UNSUPPORTED, Plan, SpconvError, spconv_conv3x3_hwc, spconv_depthwise3x3,
                     spconv_global_avg_pool, spconv_linear, spconv_run)


class MobileNetV1Engine:
    """Device weights, plans and activation buffers for one batch size and
    image size; ``net`` holds host weights laid out as ``synth.MobileNetV1``
    (stem_w [32, 3, 3, 3] as [cout][dy][dx][cin], stem_b, blocks with
    cin/cout/stride/dw_k/dw_b and the pointwise block-CSR arrays in ``pw``,
    fc_w [classes, 1024], fc_b)."""

    def __init__(self, net, batch: int, h: int = 224, w: int = 224, fuse: str = "auto"):
        import torch
        if fuse not in ("auto", "always", "never"):
            raise ValueError("fuse must be 'auto', 'always' or 'never'")
        dev = torch.device("cuda:0")
        f32 = torch.float32

        def put(a):
            return torch.from_numpy(a).to(dev).contiguous()

        self.batch, self.h, self.w = int(batch), int(h), int(w)
        self.x = torch.zeros((batch, h, w, 3), dtype=f32, device=dev)  # the static input (HWC)
        self._keep = []   # device tensors and plans the launches refer to
        self._steps = []  # closures, one launch each
        self.fused_blocks = 0
        self.fusion_times = []  # (block, fused ms, two-launch ms) of each timed choice
        c0 = int(net.stem_w.shape[0])
        hs, ws = (h - 1) // 2 + 1, (w - 1) // 2 + 1
        stem_w, stem_b = put(net.stem_w), put(net.stem_b)
        cur = torch.empty((batch, c0, hs, ws), dtype=f32, device=dev)
        self._keep += [stem_w, stem_b, cur]
        x0, y0 = self.x, cur
        self._steps.append(lambda: spconv_conv3x3_hwc(x0, stem_w, stem_b, "relu6", 2, y0, batch, h, w, 3, c0))
        ch, hh, ww = c0, hs, ws
        self.layers: List[str] = ["conv3x3 s2 3->%d @%dx%d" % (c0, h, w)]
        for blk in net.blocks:
            pw = blk.pw
            ho, wo = (hh - 1) // blk.stride + 1, (ww - 1) // blk.stride + 1
            out = torch.empty((batch, blk.cout, ho, wo), dtype=f32, device=dev)
            fused = None
            if fuse != "never":
                try:
                    fused = Plan.fused(pw.cout, pw.cin, pw.block_rows, pw.row_ptr, pw.col_idx, pw.values, pw.bias,
                                       "relu6", blk.dw_k, blk.dw_b, "relu6", blk.stride)
                except SpconvError as e:
                    if e.status != E_UNSUPPORTED:
                        raise
            split = None
            if fused is None or fuse == "auto":
                k, b = put(blk.dw_k), put(blk.dw_b)
                mid = torch.empty((batch, blk.cin, ho, wo), dtype=f32, device=dev)
                plan = Plan(pw.cout, pw.cin, pw.block_rows, pw.row_ptr, pw.col_idx, pw.values, pw.bias, "relu6")
                split = ([k, b, mid, plan],
                         [self._dw_step(cur, k, b, blk.stride, mid, batch, blk.cin, hh, ww),
                          self._run_step(plan, mid, out, batch, ho, wo)])
            if fused is not None and split is not None:
                f_step = [self._run_step(fused, cur, out, batch, hh, ww)]
                tf, ts = self._time(f_step), self._time(split[1])
                self.fusion_times.append((len(self.fusion_times), round(tf, 4), round(ts, 4)))
                if tf <= ts:
                    split[0][3].close()
                    split = None
                else:
                    fused.close()
                    fused = None
            if fused is not None:
                self._keep += [fused, out]
                self._steps.append(self._run_step(fused, cur, out, batch, hh, ww))
                self.fused_blocks += 1
                self.layers.append("fused dw3x3 s%d + 1x1 %d->%d @%dx%d" % (blk.stride, blk.cin, blk.cout, hh, ww))
            else:
                self._keep += split[0] + [out]
                self._steps += split[1]
                self.layers.append("dw3x3 s%d %d @%dx%d" % (blk.stride, blk.cin, hh, ww))
                self.layers.append("1x1 %d->%d @%dx%d" % (blk.cin, blk.cout, ho, wo))
            cur, ch, hh, ww = out, blk.cout, ho, wo
        pooled = torch.empty((batch, ch), dtype=f32, device=dev)
        self._keep.append(pooled)
        last = cur
        self._steps.append(lambda: spconv_global_avg_pool(last, pooled, batch, ch, hh, ww))
        self.layers.append("global average pool %d @%dx%d" % (ch, hh, ww))
        self.classes = int(net.fc_w.shape[0])
        fc_w, fc_b = put(net.fc_w), put(net.fc_b)
        self.logits = torch.empty((batch, self.classes), dtype=f32, device=dev)
        self._keep += [fc_w, fc_b]
        logits, classes = self.logits, self.classes
        self._steps.append(lambda: spconv_linear(pooled, fc_w, fc_b, "none", logits, batch, ch, classes))
        self.layers.append("dense fc %d->%d" % (ch, self.classes))
        self.graph = None

    @staticmethod
    def _time(steps, reps: int = 5) -> float:
        """Median device time of one pass over ``steps`` (after two warm-up
        passes), in milliseconds."""
        import torch
        for _ in range(2):
            for st in steps:
                st()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in ev:
            a.record()
            for st in steps:
                st()
            b.record()
        torch.cuda.synchronize()
        t = sorted(a.elapsed_time(b) for a, b in ev)
        return t[len(t) // 2]

    @staticmethod
    def _run_step(plan, x, y, n, h, w):
        return lambda: spconv_run(plan.handle, x, y, n, h, w)

    @staticmethod
    def _dw_step(x, k, b, stride, y, n, c, h, w):
        return lambda: spconv_depthwise3x3(x, k, b, "relu6", stride, y, n, c, h, w)

    def launches(self) -> int:
        return len(self._steps)

    def forward(self, x=None):
        """Queue the whole network on torch's current stream (copying x into
        the static input first when given); returns the logits buffer."""
        if x is not None:
            self.x.copy_(x)
        for step in self._steps:
            step()
        return self.logits

    def capture(self):
        """Record the launch sequence into one graph (after one warm-up pass)."""
        import torch
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            self.forward()
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.forward()
        self.graph = g
        return g

    def replay(self):
        if self.graph is None:
            raise RuntimeError("capture() first")
        self.graph.replay()
        return self.logits

    def close(self):
        for obj in self._keep:
            if isinstance(obj, Plan):
                obj.close()
        self._keep = []
        self._steps = []
        self.graph = None
