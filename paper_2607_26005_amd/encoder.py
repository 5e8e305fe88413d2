"""Consumer of the rendered views: the perspective policy's image encoder, run on
the device straight from the renderer's output tensors, with no host round trip.

The paper couples its rasterizer with the policy inside one training process:
rendered views feed the network on the device (Sec. 3.2), where a small
from-scratch convolution stack encodes each camera view and learned query tokens
cross-attend over its feature map (Sec. 3.3, policy architecture; App. table of
architecture details: 4 cameras at 96x54, 5 convolution layers with 128 output
channels, 16 queries per camera and one cross-attention block, a 512-d scene
embedding).  The paper's views are RGB; here a view is what this renderer writes:
its class image (one channel per class) and its inverse depth (0 for sky).

This module is PyTorch glue around the renderer (weights are random: the paper's
trained weights are not available); it adds nothing to the render path.
"""
from __future__ import annotations

import torch
import torch.nn as nn
import torch.nn.functional as F

NUM_CLASSES = 11   # ground .. light_green (scenegen.CLASS_NAMES)


class ViewEncoder(nn.Module):
    def __init__(self, cams: int = 4, width: int = 128, queries: int = 16, num_classes: int = NUM_CLASSES):
        super().__init__()
        self.cams, self.width, self.num_classes = cams, width, num_classes
        chans = [num_classes + 1, 32, 64, 64, 128, width]
        strides = [2, 2, 1, 2, 1]
        self.convs = nn.ModuleList(nn.Conv2d(chans[i], chans[i + 1], 3, stride=strides[i], padding=1)
                                   for i in range(5))
        self.queries = nn.Parameter(torch.randn(cams, queries, width) * 0.02)
        self.attn = nn.MultiheadAttention(width, 4, batch_first=True)
        self.proj = nn.Linear(width, width)

    def planes(self, cls: torch.Tensor, depth: torch.Tensor) -> torch.Tensor:
        """[V, H, W] uint8 classes and fp32 depths -> [V, classes + 1, H, W] inputs."""
        # (an elementwise comparison: F.one_hot would check the value range on the host)
        ids = torch.arange(self.num_classes, device=cls.device, dtype=torch.int32).view(1, -1, 1, 1)
        onehot = (cls.to(torch.int32).unsqueeze(1) == ids).to(torch.float32)
        inv = torch.reciprocal(depth).unsqueeze(1)   # +inf (sky) -> 0
        return torch.cat([onehot, inv], 1)

    def forward(self, cls: torch.Tensor, depth: torch.Tensor) -> torch.Tensor:
        """cls, depth: [egos * cams, H, W], view v = ego * cams + camera.  Returns the
        [egos, cams * width] scene embedding (mean of each camera's pooled tokens)."""
        x = self.planes(cls, depth)
        for conv in self.convs:
            x = F.relu(conv(x))
        V = x.shape[0]
        tokens = x.flatten(2).transpose(1, 2).contiguous()            # [V, h*w, width]
        q = self.queries.repeat(V // self.cams, 1, 1)                 # camera k's queries for view v
        pooled, _ = self.attn(q, tokens, tokens, need_weights=False)  # [V, queries, width]
        emb = self.proj(pooled.mean(1))                               # [V, width]
        return emb.reshape(V // self.cams, self.cams * self.width)
