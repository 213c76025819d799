"""Synthetic multi-view training step around the hot path.

One iteration on one view: gart_bounds -> gart_build_tile_map ->
gart_forward -> gart_l1_loss_grad (L1 against the view's target image) ->
gart_backward -> gart_adam_step per parameter group.  Every step runs in
the library's kernels; this module only orders the calls and owns the
device buffers (parameters are updated in place).

The paper trains with the 3DGS recipe (Adam over L1 plus SSIM for 30K
iterations); here the loss is the L1 sum alone, whose gradient sign(C - C*)
is the upstream gradient used throughout, and each parameter group has its
own Adam learning rate (3DGS-style defaults below).
"""
from __future__ import annotations

import torch

from . import gart

# Per-group Adam learning rates (3DGS-style defaults; SH bands share one rate).
DEFAULT_LR = dict(means=1.6e-4, log_scales=5e-3, quats=1e-3, logits=5e-2, sh=2.5e-3)
GROUPS = ("means", "log_scales", "quats", "logits", "sh")
_PARAM_ATTR = dict(means="means", log_scales="log_scales", quats="quats", logits="opacity_logits", sh="sh")


class Trainer:
    """Adam on the Gaussians of `scene` over a set of views with target images."""

    def __init__(self, scene, cameras, targets, tile=None, mode="gather", lr=None, betas=(0.9, 0.999),
                 eps=1e-15, stream=None):
        if len(cameras) != len(targets) or not cameras:
            raise ValueError("one target image per camera")
        self.g = gart.Gaussians.from_scene(scene)
        self.settings = gart.make_settings(tile or scene.tile, mode)
        self.cams = [gart.make_camera(c) for c in cameras]
        w, h = self.cams[0].width, self.cams[0].height
        if any(c.width != w or c.height != h for c in self.cams):
            raise ValueError("views must share one image size")
        self.targets = [t.contiguous() for t in targets]
        self.stream = stream
        self.frame = None
        dev = self.g.means.device
        self.image = torch.empty((h, w, 3), dtype=torch.float32, device=dev)
        self.dl = torch.empty_like(self.image)
        self.loss = torch.zeros(1, dtype=torch.float64, device=dev)
        self.partial = torch.empty(gart.gart_l1_partials(self.image.numel()), dtype=torch.float64, device=dev)
        self.grads = gart.empty_grads(self.g)
        lr = dict(DEFAULT_LR, **(lr or {}))
        self.adam = {k: gart.gart_adam(lr[k], betas[0], betas[1], eps) for k in GROUPS}
        self.m = {k: torch.zeros_like(self.param(k)) for k in GROUPS}
        self.v = {k: torch.zeros_like(self.param(k)) for k in GROUPS}
        self.t = 0

    def param(self, k):
        return getattr(self.g, _PARAM_ATTR[k])

    def step(self, view: int, events=None):
        """One iteration on view `view`; returns the device fp64 loss.  With
        `events` (6 torch.cuda.Event), records them between the stages."""
        cam, s = self.cams[view], self.stream

        def mark(k):
            if events is not None:
                events[k].record(torch.cuda.current_stream() if s is None else s)

        mark(0)
        self.frame = gart.prepare(self.g, cam, self.settings, self.frame, stream=s)
        mark(1)
        gart.gart_forward(self.g, cam, self.settings, self.frame, self.image, stream=s)
        mark(2)
        gart.gart_l1_loss_grad(self.image, self.targets[view], self.dl, self.loss, self.partial, stream=s)
        mark(3)
        gart.gart_backward(self.g, cam, self.settings, self.frame, self.dl, self.grads, stream=s)
        mark(4)
        self.t += 1
        for k in GROUPS:
            gart.gart_adam_step(self.param(k), self.grads[k], self.m[k], self.v[k], self.adam[k], self.t, stream=s)
        mark(5)
        return self.loss
