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

from . import block_conv3x3, block_conv_ex, combine, conv2d, count, maxpool, split

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

    def stages(self, h: torch.Tensor, mask: torch.Tensor, counts=None) -> torch.Tensor:
        N, C, H, W = h.shape
        bs = self.image_block // 4
        hi, lo = split(h, mask, bs, counts=counts)
        for si, (width, stride) in enumerate(zip(WIDTHS, STRIDES)):
            for bi in range(2):
                st = stride if bi == 0 else 1
                p = f"s{si + 1}.b{bi}."
                w1, b1 = self.w[p + "c1.w"], self.w[p + "c1.b"]
                if st == 1:
                    h1 = block_conv3x3(hi, lo, mask, bs, H, W, w1, b1, relu=True)
                else:
                    h1 = block_conv_ex(hi, lo, mask, bs, H, W, w1, b1, stride=st, relu=True)
                if p + "sc.w" in self.w:
                    sc = block_conv_ex(hi, lo, mask, bs, H, W, self.w[p + "sc.w"], self.w[p + "sc.b"], stride=st)
                else:
                    sc = (hi, lo)
                bs, H, W = bs // st, H // st, W // st
                hi, lo = block_conv3x3(h1[0], h1[1], mask, bs, H, W, self.w[p + "c2.w"], self.w[p + "c2.b"],
                                       relu=True, residual=sc)
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
        are fixed at capture).  Returns (graph, output tensor)."""
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            self(x, mask, counts)          # first launches set kernel attributes outside the capture
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            y = self(x, mask, counts)
        return g, y
