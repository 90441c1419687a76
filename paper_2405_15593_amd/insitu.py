"""MicroAdam inside a training loop: a small randomly initialised decoder-only
transformer on synthetic tokens, trained with ``MicroAdamW`` and, for
comparison, with torch's dense AdamW.

The tokens follow a fixed random first-order Markov chain (seeded), so the
loss has a floor well below log(V) that a working optimizer approaches.  The
run reports each optimizer's loss curve, optimizer state bytes and the time of
its optimizer step inside the loop.  Everything is float32 (the attention and
its backward stay in float32).

    python -m paper_2405_15593_amd.insitu [--steps 200] [--layers 4] [--dim 256]
"""
from __future__ import annotations

import argparse
import json
import math
import time

import torch
import torch.nn as nn
import torch.nn.functional as F


class Block(nn.Module):
    def __init__(self, dim: int, heads: int):
        super().__init__()
        self.heads = heads
        self.norm1 = nn.LayerNorm(dim)
        self.qkv = nn.Linear(dim, 3 * dim)
        self.proj = nn.Linear(dim, dim)
        self.norm2 = nn.LayerNorm(dim)
        self.fc1 = nn.Linear(dim, 4 * dim)
        self.fc2 = nn.Linear(4 * dim, dim)

    def forward(self, x):
        b, s, d = x.shape
        q, k, v = self.qkv(self.norm1(x)).split(d, dim=-1)
        shape = (b, s, self.heads, d // self.heads)
        q, k, v = (y.reshape(shape).transpose(1, 2).contiguous() for y in (q, k, v))
        y = F.scaled_dot_product_attention(q, k, v, is_causal=True)
        x = x + self.proj(y.transpose(1, 2).reshape(b, s, d))
        return x + self.fc2(F.gelu(self.fc1(self.norm2(x))))


class TinyLM(nn.Module):
    def __init__(self, vocab: int, dim: int, layers: int, heads: int, seq: int):
        super().__init__()
        self.tok = nn.Embedding(vocab, dim)
        self.pos = nn.Embedding(seq, dim)
        self.blocks = nn.ModuleList(Block(dim, heads) for _ in range(layers))
        self.norm = nn.LayerNorm(dim)
        self.head = nn.Linear(dim, vocab, bias=False)

    def forward(self, ids):
        x = self.tok(ids) + self.pos(torch.arange(ids.shape[1], device=ids.device))
        for blk in self.blocks:
            x = blk(x)
        return self.head(self.norm(x))


class MarkovTokens:
    """Batches from a fixed random Markov chain over `vocab` tokens: each token
    has `fanout` likely successors."""

    def __init__(self, vocab: int, seq: int, batch: int, device, seed: int = 0, fanout: int = 4):
        g = torch.Generator(device="cpu").manual_seed(seed)
        logits = torch.full((vocab, vocab), -4.0)
        nxt = torch.randint(0, vocab, (vocab, fanout), generator=g)
        logits.scatter_(1, nxt, torch.rand(vocab, fanout, generator=g) * 4.0)
        self.probs = torch.softmax(logits, dim=1).to(device)
        self.vocab, self.seq, self.batch, self.device = vocab, seq, batch, device
        self.g = torch.Generator(device=device).manual_seed(seed + 1)
        # the chain's entropy rate bounds the achievable loss from below
        p = torch.softmax(logits, dim=1)
        self.entropy = float(-(p * p.log()).sum(1).mean())

    def next(self):
        ids = torch.empty(self.batch, self.seq + 1, dtype=torch.long, device=self.device)
        ids[:, 0] = torch.randint(0, self.vocab, (self.batch,), generator=self.g, device=self.device)
        for i in range(self.seq):
            ids[:, i + 1] = torch.multinomial(self.probs[ids[:, i]], 1, generator=self.g).squeeze(1)
        return ids[:, :-1], ids[:, 1:]


def train(opt_name: str, steps: int, vocab=1024, dim=256, layers=4, heads=4, seq=128, batch=32,
          lr=1e-3, seed=0, device="cuda", log_every=10):
    from .optim import MicroAdamW
    torch.manual_seed(seed)
    model = TinyLM(vocab, dim, layers, heads, seq).to(device)
    params = [p for p in model.parameters()]
    n_params = sum(p.numel() for p in params)
    if opt_name == "microadam":
        opt = MicroAdamW(params, lr=lr)
    else:
        opt = torch.optim.AdamW(params, lr=lr, weight_decay=0.0)
    data = MarkovTokens(vocab, seq, batch, device, seed=seed)
    losses, opt_ms = [], []
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    t0 = time.perf_counter()
    for step in range(steps):
        x, y = data.next()
        loss = F.cross_entropy(model(x).reshape(-1, vocab), y.reshape(-1))
        opt.zero_grad(set_to_none=True)
        loss.backward()
        ev[0].record()
        opt.step()
        ev[1].record()
        if step % log_every == 0 or step == steps - 1:
            torch.cuda.synchronize()
            losses.append((step, float(loss.detach())))
            opt_ms.append(ev[0].elapsed_time(ev[1]))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    if opt_name == "microadam":
        state = opt.state_bytes()
    else:
        state = sum(v.numel() * v.element_size() for st in opt.state.values()
                    for v in st.values() if torch.is_tensor(v))
    return {"optimizer": opt_name, "params": n_params, "steps": steps, "losses": losses,
            "final_loss": losses[-1][1], "opt_step_ms": sum(opt_ms[1:]) / max(1, len(opt_ms) - 1),
            "wall_s": wall, "state_bytes": state, "state_bytes_per_param": state / n_params,
            "loss_floor": data.entropy, "log_vocab": math.log(vocab)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--layers", type=int, default=4)
    ap.add_argument("--dim", type=int, default=256)
    ap.add_argument("--lr", type=float, default=1e-3)
    args = ap.parse_args()
    out = {name: train(name, args.steps, layers=args.layers, dim=args.dim, lr=args.lr)
           for name in ("microadam", "adamw")}
    print(json.dumps(out))


if __name__ == "__main__":
    main()
