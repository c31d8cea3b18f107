"""ResNet-18 encoder on block stacks (the network the paper's block modules
are used in, Method > Block modules; its blocks stay through the downsampling
stages and shrink with the feature map).

Dense 7x7/2 stem with ReLU and 3x3/2 max-pool, split at stride 4 (block side
image_block / 4), four stages of two basic blocks on the high / low stacks
(3x3 convolutions with BlockPad fused into the tile load; a stage's first
block may have stride 2 and a 1x1/2 shortcut), combine at stride 32.  Every
step is one call of libsegblocks.so; torch only holds the tensors.

A 3x3 convolution whose implicit GEMM takes a low block's halo beside a high
neighbour from the input's high stack at half resolution gets that stack
from the convolution that wrote its input (its epilogue averages the 2x2
cells), so no launch pads the low stack beforehand (half_stacks=False pads
as segblocks_block_conv_ex does; the results are the same bit for bit).
"""
from __future__ import annotations

import torch

from . import (block_conv3x3, block_conv3x3_workspace_size, block_conv_chain, block_conv_chain_reads_half,
               block_conv_ex, block_conv_ex_workspace_size, combine, conv2d, conv_halo, count, maxpool, maxpool_halo,
               pad_halo, split)
from ._binding import SB_NHWC

WIDTHS = (64, 128, 256, 512)
STRIDES = (1, 2, 2, 2)


class BlockEncoder:
    """weights: name -> OIHW tensor as drawn by inputs.encoder_weights (any
    device); they are moved to `device` as channels_last (OHWI memory)."""

    def __init__(self, weights: dict, image_block: int, device="cuda", blockwise_stem: bool = False,
                 half_stacks: bool = True):
        if image_block % 64:
            raise ValueError("the image block must be a multiple of 64 pixels (block side >= 2 at stride 32)")
        self.image_block = image_block
        # blockwise_stem: split the image itself and run the 7x7/2 stem (3-pixel
        # BlockPad) and the 3x3/2 max-pool (1-pixel BlockPad) on the blocks, so
        # that the blocks persist from the image to the last stage
        self.blockwise_stem = blockwise_stem
        self.half_stacks = half_stacks
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

    def stem_blocks(self, x: torch.Tensor, mask: torch.Tensor, counts):
        """The blockwise stem: image blocks -> stacks at stride 4."""
        N, C, H, W = x.shape
        blk = self.image_block
        hi, lo = split(x, mask, blk, counts=counts)
        hp, lp = pad_halo(hi, lo, mask, blk, H, W, 3)
        sh, sl = conv_halo(hp, lp, mask, blk, H, W, 3, self.w["stem.w"], self.w["stem.b"], stride=2, relu=True)
        ph, pl = pad_halo(sh, sl, mask, blk // 2, H // 2, W // 2, 1)
        return maxpool_halo(ph, pl, mask, blk // 2, H // 2, W // 2, 1, 3, 2)

    def stages(self, h: torch.Tensor, mask: torch.Tensor, counts=None) -> torch.Tensor:
        """h: the stage-1 map [N, 64, H/4, W/4] -> [N, 512, H/32, W/32]."""
        N, C, H, W = h.shape
        hi, lo = split(h, mask, self.image_block // 4, counts=counts)
        return self.stages_on_stacks(hi, lo, mask, H, W)

    def stages_on_stacks(self, hi: torch.Tensor, lo: torch.Tensor, mask: torch.Tensor, H: int, W: int):
        """The four stages on the stage-1 stacks (H x W: the stage-1 map), then
        BlockCombine."""
        N = mask.shape[0]
        bs = self.image_block // 4
        ref = hi if hi.shape[0] else lo
        dt, nh, nl = ref.dtype, hi.shape[0], lo.shape[0]
        nbytes = self.workspace_bytes(N, H, W, dt, (nh, nl))
        ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=ref.device) if nbytes else None

        def reads_half(c_in, h, w, b, c_out, stride):  # does that 3x3 convolution take the half stack?
            return self.half_stacks and block_conv_chain_reads_half(dt, N, c_in, h, w, b, c_out, 3, stride, nh, nl)

        hh = None  # the high input stack at half resolution, when the next convolution reads it
        convs = [(si, bi) for si in range(len(WIDTHS)) for bi in range(2)]
        for idx, (si, bi) in enumerate(convs):
            width = WIDTHS[si]
            st = STRIDES[si] if bi == 0 else 1
            p = f"s{si + 1}.b{bi}."
            w1, b1 = self.w[p + "c1.w"], self.w[p + "c1.b"]
            # c1 feeds c2: 3x3/1 on the map at this block's output resolution
            want = reads_half(width, H // st, W // st, bs // st, width, 1)
            h1 = block_conv_chain(hi, lo, mask, bs, H, W, w1, b1, stride=st, relu=True, hi_half=hh, want_half=want,
                                  workspace=ws)
            if p + "sc.w" in self.w:
                sc = block_conv_ex(hi, lo, mask, bs, H, W, self.w[p + "sc.w"], self.w[p + "sc.b"], stride=st,
                                   workspace=ws)
            else:
                sc = (hi, lo)
            bs, H, W = bs // st, H // st, W // st
            # c2 feeds the next block's c1, if there is one
            want = False
            if idx + 1 < len(convs):
                nsi, nbi = convs[idx + 1]
                nst = STRIDES[nsi] if nbi == 0 else 1
                want = reads_half(width, H, W, bs, WIDTHS[nsi], nst)
            hi, lo, hh = block_conv_chain(h1[0], h1[1], mask, bs, H, W, self.w[p + "c2.w"], self.w[p + "c2.b"],
                                          relu=True, residual=sc, hi_half=h1[2], want_half=want, workspace=ws)
        return combine(hi, lo, mask, bs, H, W)

    def __call__(self, x: torch.Tensor, mask: torch.Tensor, counts=None) -> torch.Tensor:
        """x [N, 3, H, W] channels_last, mask [N, H/image_block, W/image_block]
        uint8 -> [N, 512, H/32, W/32] channels_last.  counts = (n_high, n_low)
        of the mask, else taken with segblocks_count (one host sync)."""
        if counts is None:
            counts = count(mask)
        if self.blockwise_stem:
            hi, lo = self.stem_blocks(x, mask, counts)
            return self.stages_on_stacks(hi, lo, mask, x.shape[2] // 4, x.shape[3] // 4)
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
