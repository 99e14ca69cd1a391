"""A ViT encoder with random weights and MPM insertions, to measure what the merge
saves in the blocks after it: the paper's end-to-end setting (MPM before blocks 2
and 5 of a ViT encoder, the full token grid rebuilt by the gather before the
decoder; Sec. 3.3, Sec. 4, Table 1 and Table 5), with no trained weights.

The blocks are plain torch operations (pre-LN attention and MLP, bfloat16). After a
merge the images have different token counts: the per-token parts of a block
(norms, projections, MLP) run on the packed rows, so only real tokens are
computed. Attention runs either on the packed rows too (attn="varlen": torch's
variable-length flash attention, with the merge's offsets as the cumulative
sequence lengths; the plain encoder uses the same kernel with equal lengths), or
on the padded layout the paper uses (attn="padded", Sec. 4.2): each batch padded
to its longest image with the library's mpm_pad, the padded keys masked, two
batched products around a float32 softmax (both operands of each product
contiguous), and the result unpadded with mpm_unpad. The merges, the map
composition and the gather are the library's kernels (mpm_merge,
mpm_compose_unmerge).
"""
from __future__ import annotations

import math

import torch

from . import api


class Block:
    """One pre-LN transformer block (multi-head attention, 4x MLP) with random weights."""

    def __init__(self, D: int, heads: int, dtype, device, gen: torch.Generator):
        def w(shape, scale):
            return (torch.randn(shape, generator=gen) * scale).to(dtype).to(device)

        self.D, self.H, self.dh = D, heads, D // heads
        self.ln1 = (torch.ones(D, dtype=dtype, device=device), torch.zeros(D, dtype=dtype, device=device))
        self.ln2 = (torch.ones(D, dtype=dtype, device=device), torch.zeros(D, dtype=dtype, device=device))
        self.w_qkv, self.b_qkv = w((D, 3 * D), D ** -0.5), w((3 * D,), 0.02)
        self.w_proj, self.b_proj = w((D, D), D ** -0.5), w((D,), 0.02)
        self.w_fc1, self.b_fc1 = w((D, 4 * D), D ** -0.5), w((4 * D,), 0.02)
        self.w_fc2, self.b_fc2 = w((4 * D, D), (4 * D) ** -0.5), w((D,), 0.02)

    def attention(self, qkv, B: int, P: int, key_valid):
        """qkv [B, P, 3, H, dh] -> [B, P, D]; key_valid [B, P] bool or None (all valid)."""
        H, dh = self.H, self.dh
        q = qkv[:, :, 0].permute(0, 2, 1, 3).reshape(B * H, P, dh).contiguous()
        kt = qkv[:, :, 1].permute(0, 2, 3, 1).reshape(B * H, dh, P).contiguous()
        v = qkv[:, :, 2].permute(0, 2, 1, 3).reshape(B * H, P, dh).contiguous()
        s = torch.bmm(q, kt).float().view(B, H, P, P) * (dh ** -0.5)
        if key_valid is not None:
            s = s.masked_fill(~key_valid[:, None, None, :], float("-inf"))
        p = torch.softmax(s, dim=-1).to(qkv.dtype).view(B * H, P, P)
        o = torch.bmm(p, v)  # [B*H, P, dh]
        return o.view(B, H, P, dh).permute(0, 2, 1, 3).reshape(B, P, self.D)

    def __call__(self, rows, B: int, N: int, off=None, P: int | None = None, key_valid=None, attn: str = "varlen"):
        """rows [R, D]: dense (off None: B images of N rows) or packed by off [B+1]
        (P = the batch's longest image, key_valid its mask [B, P])."""
        h = torch.nn.functional.layer_norm(rows, (self.D,), *self.ln1)
        qkv = torch.addmm(self.b_qkv, h, self.w_qkv)  # [R, 3D]
        if attn == "varlen":
            from torch.nn.attention.varlen import varlen_attn

            cu = off if off is not None else torch.arange(0, (B + 1) * N, N, dtype=torch.int32, device=rows.device)
            mx = P if off is not None else N
            q, k, v = (t.contiguous() for t in qkv.view(-1, 3, self.H, self.dh).unbind(1))
            a = varlen_attn(q, k, v, cu, cu, mx, mx).reshape(-1, self.D)
        elif off is None:
            a = self.attention(qkv.view(B, N, 3, self.H, self.dh), B, N, None).reshape(B * N, self.D)
        else:
            padded = api.pad(qkv, off, P)  # [B, P, 3D]
            o = self.attention(padded.view(B, P, 3, self.H, self.dh), B, P, key_valid)
            a = api.unpad(o.contiguous(), off, rows=rows.shape[0])
        rows = rows + torch.addmm(self.b_proj, a, self.w_proj)
        h = torch.nn.functional.layer_norm(rows, (self.D,), *self.ln2)
        f = torch.nn.functional.gelu(torch.addmm(self.b_fc1, h, self.w_fc1))
        return rows + torch.addmm(self.b_fc2, f, self.w_fc2)


class Encoder:
    """`depth` blocks with MPM before the blocks listed in `merge_before` (0-based),
    then the composed gather back to the full grid. merge_before=() is the plain
    encoder."""

    def __init__(self, D: int = 768, heads: int = 12, depth: int = 12, merge_before=(2, 5),
                 dtype=torch.bfloat16, device="cuda", seed: int = 0, attn: str = "varlen"):
        gen = torch.Generator().manual_seed(seed)
        self.blocks = [Block(D, heads, dtype, device, gen) for _ in range(depth)]
        self.merge_before = tuple(merge_before)
        self.D = D
        self.attn = attn
        self.last_counts = None  # per insertion: token counts per image (host), after a forward

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        B, N, D = x.shape
        rows, off, P, key_valid = x.reshape(B * N, D), None, N, None
        maps, counts = [], []
        for i, blk in enumerate(self.blocks):
            if i in self.merge_before:
                m = api.merge(rows if off is not None else rows.view(B, N, D), off, N=N)
                off_h = m.y_off.cpu()  # one host read per insertion: the packed row count and the longest image
                n = torch.diff(off_h)
                counts.append(n.tolist())
                total, P = int(off_h[-1]), int(n.max())
                rows, off = m.y[:total], m.y_off
                key_valid = torch.arange(P, device=x.device)[None, :] < n.to(x.device)[:, None]
                maps.append(m.map)
            rows = blk(rows, B, N, off, P, key_valid, self.attn)
        self.last_counts = counts
        if not maps:
            return rows.view(B, N, D)
        first = maps[0]
        for m in maps[1:-1]:
            first = api.compose(first, m)
        if len(maps) == 1:
            return api.unmerge(rows, off, first)
        out, _ = api.compose_unmerge(rows, off, first, maps[-1])
        return out
