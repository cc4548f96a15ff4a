"""A VGG-16 convolution stack on the split-FFT convolution.

The paper evaluates the method on the convolution layers of VGG16
(Section 4).  This driver runs the 13 3x3 'same' convolutions with fused
bias and ReLU and a 2x2 stride-2 max-pool after layers 2, 4, 7, 10 and 13,
all through the library's C ABI: each layer has its own plan (tile size
chosen by the plan unless given) and filter spectra, transformed once at
construction; one workspace (the largest any layer needs) and two
activation buffers are shared by all layers.

With method="direct" the same stack runs on the library's spatial
convolution (fftsplit_direct_conv2d), the method the paper compares
against on these layers; the plans then serve only as layer descriptors.

With fuse_pool (the default for the split method) the layers that end a
stage carry FFTSPLIT_MAXPOOL, so their convolution writes the pooled
activation directly and no separate pooling pass runs.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

from . import Plan, maxpool2x2, set_timing_events

POOL_AFTER = (2, 4, 7, 10, 13)


class VGG16Stack:
    def __init__(self, layers: Sequence, batch: int, hw: int = 224, tiles: Optional[Sequence[int]] = None,
                 mode: str = "os", device=None, method: str = "split", fuse_pool: bool = True):
        """`layers`: 13 (w, b) pairs (torch CUDA float32 tensors or arrays);
        `tiles`: optional per-layer tile sizes (0 or None = plan's choice)."""
        import torch
        if len(layers) != 13:
            raise ValueError("VGG-16 has 13 convolution layers")
        if method not in ("split", "direct"):
            raise ValueError("method must be 'split' or 'direct'")
        self.method = method
        self.fuse_pool = fuse_pool and method == "split"
        dev = torch.device("cuda", torch.cuda.current_device() if device is None else int(device))
        self.device = dev
        self.batch = batch
        self.plans: List[Plan] = []
        self.wspecs = []
        self.biases = []
        s = hw
        shapes = []
        for i, (w, b) in enumerate(layers, start=1):
            w = torch.as_tensor(w, dtype=torch.float32, device=dev).contiguous()
            b = torch.as_tensor(b, dtype=torch.float32, device=dev).contiguous()
            cout, cin, k, _ = w.shape
            t = 0 if tiles is None or not tiles[i - 1] else int(tiles[i - 1])
            plan = Plan(batch, cin, s, s, cout, k, tile=t, mode=mode, bias=True, relu=True, device=dev.index,
                        pool=self.fuse_pool and i in POOL_AFTER)
            self.plans.append(plan)
            self.wspecs.append(plan.transform_weights(w) if method == "split" else plan.direct_transform_weights(w))
            self.biases.append(b)
            shapes.append((batch, cout, s, s))
            if i in POOL_AFTER:
                s //= 2
        self.workspace = (torch.empty(max(p.info.workspace_bytes for p in self.plans), dtype=torch.uint8,
                                      device=dev) if method == "split" else None)
        biggest = max(max(n * c * h * w for n, c, h, w in shapes), batch * 3 * hw * hw)
        self._buf = [torch.empty(biggest, dtype=torch.float32, device=dev) for _ in range(2)]

    @property
    def tiles(self):
        return [p.tile for p in self.plans]

    def forward(self, x, keep=False, layer_events=None):
        """Runs the stack on x [batch, 3, hw, hw].  Returns the final
        activation [batch, 512, hw/32, hw/32] (a view of an internal buffer),
        or with keep=True also a list of copies of every layer's post-ReLU
        output (before pooling; needs fuse_pool=False).  layer_events: 13
        (start, stop) torch.cuda.Event pairs that time each layer's
        convolution call from its kernels' dispatch timestamps."""
        if keep and self.fuse_pool:
            raise ValueError("keep=True needs the unpooled outputs: build the stack with fuse_pool=False")
        cur, other = self._buf
        a = x
        outs = []
        for i, plan in enumerate(self.plans, start=1):
            shape = plan.out_shape
            y = other[: plan.n * plan.cout * shape[2] * shape[3]].view(shape)
            if layer_events is not None:
                set_timing_events(*layer_events[i - 1])
            if self.method == "split":
                plan.conv2d(a, self.wspecs[i - 1], self.biases[i - 1], out=y, workspace=self.workspace)
            else:
                plan.direct_conv2d(a, self.wspecs[i - 1], self.biases[i - 1], out=y)
            if layer_events is not None:
                set_timing_events()
            if keep:
                outs.append(y.clone())
            if i in POOL_AFTER and not plan.pool:
                pooled = cur[: plan.n * plan.cout * (plan.h // 2) * (plan.w // 2)].view(
                    plan.n, plan.cout, plan.h // 2, plan.w // 2)
                a = maxpool2x2(y, out=pooled)
            else:
                a = y
                cur, other = other, cur
        return (a, outs) if keep else a
