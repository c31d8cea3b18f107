"""ResNet-18 encoder on block stacks (the network the paper's block modules
are used in, Method > Block modules; its blocks stay through the downsampling
stages and shrink with the feature map).

Dense 7x7/2 stem with ReLU and 3x3/2 max-pool, split at stride 4 (block side
image_block / 4), four stages of two basic blocks on the high / low stacks
(3x3 convolutions with BlockPad fused into the tile load; a stage's first
block may have stride 2 and a 1x1/2 shortcut), combine at stride 32.  Every
step is one call of libsegblocks.so; torch only holds the tensors.
"""
from __future__ import annotations

import torch

from . import (block_conv3x3, block_conv3x3_workspace_size, block_conv_ex, block_conv_ex_workspace_size, combine,
               conv2d, count, maxpool, split)
from ._binding import SB_NHWC

WIDTHS = (64, 128, 256, 512)
STRIDES = (1, 2, 2, 2)


class BlockEncoder:
    """weights: name -> OIHW tensor as drawn by inputs.encoder_weights (any
    device); they are moved to `device` as channels_last (OHWI memory)."""

    def __init__(self, weights: dict, image_block: int, device="cuda"):
        if image_block % 64:
            raise ValueError("the image block must be a multiple of 64 pixels (block side >= 2 at stride 32)")
        self.image_block = image_block
        cl = torch.channels_last
        self.w = {k: (v.to(device).contiguous(memory_format=cl) if v.dim() == 4 else v.to(device).contiguous())
                  for k, v in weights.items()}

    def stem(self, x: torch.Tensor) -> torch.Tensor:
        h = conv2d(x, self.w["stem.w"], self.w["stem.b"], stride=2, padding=3, relu=True)
        return maxpool(h, 3, 2, 1)

    def workspace_bytes(self, N: int, H: int, W: int, dtype: torch.dtype, counts) -> int:
        """Largest workspace any stage convolution needs for an N x 64 x H x W
        stage-1 map with block counts (n_high, n_low); the convolutions run
        one after the other on one stream, so they share one buffer."""
        nh, nl = counts
        bs, need = self.image_block // 4, 0
        cin = WIDTHS[0]
        for si, (width, stride) in enumerate(zip(WIDTHS, STRIDES)):
            for bi in range(2):
                st = stride if bi == 0 else 1
                if st == 1:
                    need = max(need, block_conv3x3_workspace_size(dtype, SB_NHWC, N, cin, H, W, bs, width, nh, nl))
                else:
                    need = max(need, block_conv_ex_workspace_size(dtype, N, cin, H, W, bs, width, 3, st, nh, nl))
                if st != 1 or cin != width:
                    need = max(need, block_conv_ex_workspace_size(dtype, N, cin, H, W, bs, width, 1, st, nh, nl))
                bs, H, W = bs // st, H // st, W // st
                need = max(need, block_conv3x3_workspace_size(dtype, SB_NHWC, N, width, H, W, bs, width, nh, nl))
                cin = width
        return need

    def stages(self, h: torch.Tensor, mask: torch.Tensor, counts=None) -> torch.Tensor:
        N, C, H, W = h.shape
        bs = self.image_block // 4
        hi, lo = split(h, mask, bs, counts=counts)
        nbytes = self.workspace_bytes(N, H, W, h.dtype, (hi.shape[0], lo.shape[0]))
        ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=h.device) if nbytes else None
        for si, (width, stride) in enumerate(zip(WIDTHS, STRIDES)):
            for bi in range(2):
                st = stride if bi == 0 else 1
                p = f"s{si + 1}.b{bi}."
                w1, b1 = self.w[p + "c1.w"], self.w[p + "c1.b"]
                if st == 1:
                    h1 = block_conv3x3(hi, lo, mask, bs, H, W, w1, b1, relu=True, workspace=ws)
                else:
                    h1 = block_conv_ex(hi, lo, mask, bs, H, W, w1, b1, stride=st, relu=True, workspace=ws)
                if p + "sc.w" in self.w:
                    sc = block_conv_ex(hi, lo, mask, bs, H, W, self.w[p + "sc.w"], self.w[p + "sc.b"], stride=st,
                                       workspace=ws)
                else:
                    sc = (hi, lo)
                bs, H, W = bs // st, H // st, W // st
                hi, lo = block_conv3x3(h1[0], h1[1], mask, bs, H, W, self.w[p + "c2.w"], self.w[p + "c2.b"],
                                       relu=True, residual=sc, workspace=ws)
        return combine(hi, lo, mask, bs, H, W)

    def __call__(self, x: torch.Tensor, mask: torch.Tensor, counts=None) -> torch.Tensor:
        """x [N, 3, H, W] channels_last, mask [N, H/image_block, W/image_block]
        uint8 -> [N, 512, H/32, W/32] channels_last.  counts = (n_high, n_low)
        of the mask, else taken with segblocks_count (one host sync)."""
        if counts is None:
            counts = count(mask)
        return self.stages(self.stem(x), mask, counts)

    def capture(self, x: torch.Tensor, mask: torch.Tensor, counts):
        """Records one forward into a HIP graph, so that a replay costs one
        host call instead of one per kernel.  x and mask stay the graph's
        inputs (write new values into them before a replay; the block counts
        are fixed at capture).  Nothing needs to run before the capture: the
        library allocates nothing, and the workspace and every intermediate
        come from torch's graph memory pool.  Returns (graph, output tensor)."""
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            y = self(x, mask, counts)
        return g, y
