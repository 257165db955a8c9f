"""Multi-query associative recall (MQAR): the capacity workload of Section
2.3 ("Capacity in isolation") and Appendix C, scaled down to run in minutes.

Each example holds N key-value pairs followed by the same N keys in random
order; the model must return the value of each queried key.  Keys and values
are drawn without replacement from two vocabularies of 8192 tokens each; a
pair token is the concatenation of its key's and its value's embeddings, a
query token the key's embedding followed by zeros.  Queries are read-only:
they do not write the state (their write strength beta is 0).

The model follows Alg. 1 (the vanilla triadic block): per layer
RMSNorm -> per-head projections q, k, v (dimension D) and q', k' (dimension
E) -> the triadic recurrence S_h <- S_h + k (x) k' (x) v, o_h = S_h x1 q x2 q'
(no forgetting, no delta rule, no convolution or activations: the sGLA
variant of the operator with log-gates 0) -> per-head RMSNorm -> output
projection, then a SwiGLU MLP; an RMSNorm and a linear readout over the
value vocabulary at the query positions.  The recurrence runs in this
library's kernels (tla_fwd / tla_bwd through paper_2609_36529_amd.attention,
bf16 operands, chunk 16); the rest of the model is plain PyTorch.

Readings (the paper gives the architecture and hyperparameters, Appendix C):
d_model 128 (64 + 64 for the key and value embeddings), H = 4 heads, D = 16,
SwiGLU width 384, two layers, AdamW (lr 1e-3, betas (0.9, 0.999), weight
decay 0.1, cosine decay to 0), bf16 operands; the scaled-down run trains
for far fewer tokens than the paper's 12.5 billion (steps and batch are
arguments) and sweeps a few (N, E) cells.
"""
import argparse
import json
import math
import time

import torch
import torch.nn as nn
import torch.nn.functional as F

N_KEYS = N_VALS = 8192


def make_batch(n_seq, N, gen, device="cpu"):
    """(key ids [n_seq, 2N], value ids [n_seq, 2N] (-1 at queries),
    write mask [n_seq, 2N] (1 for pairs, 0 for queries), targets [n_seq, N]
    (the value id of each query)).  gen: a torch.Generator."""
    keys = torch.stack([torch.randperm(N_KEYS, generator=gen)[:N] for _ in range(n_seq)])
    vals = torch.stack([torch.randperm(N_VALS, generator=gen)[:N] for _ in range(n_seq)])
    order = torch.stack([torch.randperm(N, generator=gen) for _ in range(n_seq)])
    qkeys = torch.gather(keys, 1, order)
    targets = torch.gather(vals, 1, order)
    key_ids = torch.cat([keys, qkeys], 1)
    val_ids = torch.cat([vals, torch.full_like(vals, -1)], 1)
    write = torch.cat([torch.ones(n_seq, N), torch.zeros(n_seq, N)], 1)
    return tuple(x.to(device) for x in (key_ids, val_ids, write, targets))


class RMSNorm(nn.Module):
    def __init__(self, d, eps=1e-6):
        super().__init__()
        self.w = nn.Parameter(torch.ones(d))
        self.eps = eps

    def forward(self, x):
        return x * torch.rsqrt(x.pow(2).mean(-1, keepdim=True) + self.eps) * self.w


class Mixer(nn.Module):
    """The vanilla triadic mixer of Alg. 1 for H heads."""

    def __init__(self, d, H, D, E, mixer):
        super().__init__()
        self.H, self.D, self.E = H, D, E
        self.norm = RMSNorm(d)
        self.proj = nn.Linear(d, H * (3 * D + 2 * E), bias=False)
        self.head_norm = RMSNorm(D)
        self.out = nn.Linear(H * D, d, bias=False)
        self.mixer = mixer  # (q, k, v, q2, k2, g, beta) -> o, all [B, T, H, .]

    def forward(self, x, write):
        B, T, _ = x.shape
        H, D, E = self.H, self.D, self.E
        y = self.proj(self.norm(x)).view(B, T, H, 3 * D + 2 * E)
        q, k, v, q2, k2 = torch.split(y, [D, D, D, E, E], dim=-1)
        g = torch.zeros(B, T, H, E, device=x.device, dtype=torch.float32)
        beta = write[:, :, None].expand(B, T, H).contiguous().float()
        o = self.mixer(q, k, v, q2, k2, g, beta)
        return x + self.out(self.head_norm(o.float()).reshape(B, T, H * D))


class SwiGLU(nn.Module):
    def __init__(self, d, width):
        super().__init__()
        self.norm = RMSNorm(d)
        self.gate = nn.Linear(d, width, bias=False)
        self.up = nn.Linear(d, width, bias=False)
        self.down = nn.Linear(width, d, bias=False)

    def forward(self, x):
        u = self.norm(x)
        return x + self.down(F.silu(self.gate(u)) * self.up(u))


class MQARModel(nn.Module):
    def __init__(self, E, mixer, d=128, H=4, D=16, width=384, layers=2):
        super().__init__()
        self.key_emb = nn.Embedding(N_KEYS, d // 2)
        self.val_emb = nn.Embedding(N_VALS, d // 2)
        self.blocks = nn.ModuleList()
        for _ in range(layers):
            self.blocks.append(Mixer(d, H, D, E, mixer))
            self.blocks.append(SwiGLU(d, width))
        self.norm = RMSNorm(d)
        self.readout = nn.Linear(d, N_VALS, bias=False)

    def forward(self, key_ids, val_ids, write):
        ve = self.val_emb(val_ids.clamp(min=0)) * (val_ids >= 0)[..., None]
        x = torch.cat([self.key_emb(key_ids), ve], -1)
        for blk in self.blocks:
            x = blk(x, write) if isinstance(blk, Mixer) else blk(x)
        return self.readout(self.norm(x))

    def loss_acc(self, batch):
        key_ids, val_ids, write, targets = batch
        N = targets.shape[1]
        logits = self(key_ids, val_ids, write)[:, N:]
        loss = F.cross_entropy(logits.reshape(-1, N_VALS).float(), targets.reshape(-1))
        acc = (logits.argmax(-1) == targets).float().mean()
        return loss, acc


def tla_mixer(dtype=torch.bfloat16, chunk=16, out_dtype=None):
    """The recurrence through this library's kernels (sGLA, log-gates 0,
    beta = write mask), operands in `dtype`; the output and the operand
    gradients in out_dtype (default: dtype)."""
    import paper_2609_36529_amd as tla

    def run(q, k, v, q2, k2, g, beta):
        args = [t.to(dtype).contiguous() for t in (q, k, v, q2, k2)]
        o, _ = tla.attention(tla.SGLA, *args, g, beta, None, chunk=chunk, out_dtype=out_dtype)
        return o
    return run


def train(E, N, steps, batch, seed=0, device="cuda", eval_seqs=512, log=None, lr=1e-3, warmup=0.05):
    """Trains one (E, N) cell; returns a dict with the held-out accuracy.
    The learning rate warms up linearly over the first `warmup` fraction of
    the steps, then decays to 0 on a cosine."""
    torch.manual_seed(seed)
    model = MQARModel(E, tla_mixer()).to(device)
    opt = torch.optim.AdamW(model.parameters(), lr=lr, betas=(0.9, 0.999), weight_decay=0.1)
    nw = max(1, int(warmup * steps))
    sched = torch.optim.lr_scheduler.LambdaLR(
        opt, lambda s: (s + 1) / nw if s < nw else 0.5 * (1 + math.cos(math.pi * (s - nw) / max(1, steps - nw))))
    gen = torch.Generator().manual_seed(1000 + seed)
    t0 = time.perf_counter()
    for step in range(steps):
        loss, acc = model.loss_acc(make_batch(batch, N, gen, device))
        opt.zero_grad(set_to_none=True)
        loss.backward()
        opt.step()
        sched.step()
        if log and (step % max(1, steps // 5) == 0 or step == steps - 1):
            log(f"E={E} N={N} step {step}: loss {loss.item():.3f} acc {acc.item():.3f}")
    train_s = time.perf_counter() - t0
    test_gen = torch.Generator().manual_seed(999_999)
    model.eval()
    correct = total = 0
    with torch.no_grad():
        for _ in range(max(1, eval_seqs // batch)):
            _, acc = model.loss_acc(make_batch(batch, N, test_gen, device))
            correct += acc.item() * batch
            total += batch
    n_params = sum(p.numel() for n, p in model.named_parameters() if "emb" not in n and "readout" not in n)
    return {"E": E, "N": N, "steps": steps, "batch": batch, "lr": lr, "test_accuracy": round(correct / total, 4),
            "train_seconds": round(train_s, 1), "non_embedding_params": n_params,
            "state_per_head": f"16 x {E} x 16"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--E", type=int, nargs="+", default=[1, 4, 16])
    ap.add_argument("--N", type=int, nargs="+", default=[32, 64, 128])
    ap.add_argument("--steps", type=int, default=1500)
    ap.add_argument("--batch", type=int, default=64)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--lr", type=float, default=1e-3)
    args = ap.parse_args()
    results = []
    for N in args.N:
        for E in args.E:
            r = train(E, N, args.steps, args.batch, args.seed, log=lambda m: print(m, flush=True), lr=args.lr)
            print(json.dumps(r), flush=True)
            results.append(r)
    print(json.dumps({"mqar": results}), flush=True)


if __name__ == "__main__":
    main()
