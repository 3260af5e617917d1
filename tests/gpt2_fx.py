"""A GPT-2 model written for torch.fx tracing (test input of the graph-sharding
checks).  Same block structure as GPT-2: token and position embeddings, pre-LN
blocks of attention and feed-forward halves, each closed by a residual add,
final LayerNorm and a vocabulary head.  The causal mask is built once from the
input's length and used by every block, the kind of node the sharding
algorithm treats as common."""
from __future__ import annotations

import math

import torch
import torch.nn as nn


class Attention(nn.Module):
    def __init__(self, h: int, heads: int):
        super().__init__()
        self.h, self.heads = h, heads
        self.c_attn = nn.Linear(h, 3 * h)
        self.c_proj = nn.Linear(h, h)

    def forward(self, x, mask):
        b, s, h = x.shape
        q, k, v = self.c_attn(x).split(self.h, dim=2)
        d = h // self.heads
        q = q.view(b, s, self.heads, d).transpose(1, 2)
        k = k.view(b, s, self.heads, d).transpose(1, 2)
        v = v.view(b, s, self.heads, d).transpose(1, 2)
        att = (q @ k.transpose(-2, -1)) * (1.0 / math.sqrt(d))
        att = att.masked_fill(mask, float("-inf")).softmax(dim=-1)
        y = (att @ v).transpose(1, 2).reshape(b, s, h)
        return self.c_proj(y)


class MLP(nn.Module):
    def __init__(self, h: int):
        super().__init__()
        self.c_fc = nn.Linear(h, 4 * h)
        self.act = nn.GELU(approximate="tanh")
        self.c_proj = nn.Linear(4 * h, h)

    def forward(self, x):
        return self.c_proj(self.act(self.c_fc(x)))


class Block(nn.Module):
    def __init__(self, h: int, heads: int):
        super().__init__()
        self.ln_1 = nn.LayerNorm(h)
        self.attn = Attention(h, heads)
        self.ln_2 = nn.LayerNorm(h)
        self.mlp = MLP(h)

    def forward(self, x, mask):
        x = x + self.attn(self.ln_1(x), mask)
        return x + self.mlp(self.ln_2(x))


class GPT2(nn.Module):
    def __init__(self, n_layer: int, h: int, heads: int, vocab: int = 50257, n_pos: int = 1024):
        super().__init__()
        self.wte = nn.Embedding(vocab, h)
        self.wpe = nn.Embedding(n_pos, h)
        self.h = nn.ModuleList(Block(h, heads) for _ in range(n_layer))
        self.ln_f = nn.LayerNorm(h)
        self.lm_head = nn.Linear(h, vocab, bias=False)

    def forward(self, input_ids):
        s = input_ids.size(1)
        pos = torch.arange(s, device=input_ids.device)
        mask = pos.unsqueeze(0) > pos.unsqueeze(1)  # key j masked for query i when j > i
        x = self.wte(input_ids) + self.wpe(pos)
        for blk in self.h:
            x = blk(x, mask)
        return self.lm_head(self.ln_f(x))


def traced(n_layer: int, h: int, heads: int, vocab: int = 50257, meta: bool = True):
    """torch.fx GraphModule of a GPT-2 model (parameters on the meta device
    unless meta=False)."""
    import torch.fx as fx
    if meta:
        with torch.device("meta"):
            m = GPT2(n_layer, h, heads, vocab)
    else:
        m = GPT2(n_layer, h, heads, vocab)
    return fx.symbolic_trace(m)
