"""Seeded synthetic workloads for the tree-replay round.

This module only draws random logits. It holds none of the method's
arithmetic (no softmax, no planning, no sampling of tokens), so both the HIP
path and the CPU oracle may be fed from it. The logits stand in for the
paper's drafter/target outputs at Qwen-scale vocabulary (V = 151936) with the
budgets of its experiments (Section 4, B = 16..64 single-request, batched
serving in Section 4.4); no model, dataset or checkpoint is involved.

Five workloads (sizes, distributions and temperatures):
  1 tiny          R=1,  V=1024,   D=8,  B=16,  K=4,  fp32, T=1.0
                  x = 3 z + 8 on 3 distinct uniform "peak" tokens per position;
                  target noise sd 1.0
  2 small         R=1,  V=32000,  D=16, B=32,  K=8,  bf16, T=1.0
                  x = s z, s ~ U[2,5] per position, plus a Zipf-ranked boost:
                  16 distinct ids drawn without replacement with
                  P(id) ~ (id+1)^-1.1, the i-th drawn gets +6/sqrt(i);
                  target noise sd 0.7
  3 qwen_vocab    R=1,  V=151936, D=16, B=64,  K=8,  bf16, T=0.8, as 2
  4 batched       R=16, V=151936, D=16, B=128, K=10, bf16, T=1.0
                  as 2 with s ~ U[1,6] per (request, position) and target
                  noise sd sigma_r ~ U[0.3, 1.5] per request
  5 large_budget  R=64, V=151936, D=32, B=256, K=16, bf16, T=1.0, as 4

Pool workloads add transition scores between the candidates of consecutive
positions (transitions(): i.i.d. 1.5 * N(0, 1), binary32), as a drafter that
looks its corrections up in a table would hold.

Per request the generator draws D+1 base rows (binary32). Draft row d is base
row d. The target row of tree node n is base row depth(n) (the distribution of
the token that follows node n) plus Gaussian noise, so the target needs the
planned depths. Rows are rounded to the storage dtype by round-to-nearest-even
after the noise is added. Row D only seeds the targets of depth-D nodes.
"""
import torch

CONFIGS = {
    1: dict(name="tiny", R=1, steps=200, V=1024, D=8, B=16, K=4, T=1.0, dtype="f32"),
    2: dict(name="small", R=1, steps=500, V=32000, D=16, B=32, K=8, T=1.0, dtype="bf16"),
    3: dict(name="qwen_vocab", R=1, steps=1000, V=151936, D=16, B=64, K=8, T=0.8, dtype="bf16"),
    4: dict(name="batched", R=16, steps=500, V=151936, D=16, B=128, K=10, T=1.0, dtype="bf16"),
    5: dict(name="large_budget", R=64, steps=200, V=151936, D=32, B=256, K=16, T=1.0, dtype="bf16"),
}

GEN_SEED_BASE = 1000
REPLAY_SEED_BASE = 0x5453_0000_0000_0000

TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}


def replay_seed(cfg_id):
    return REPLAY_SEED_BASE + int(cfg_id)


def config(cfg_id, **over):
    c = dict(CONFIGS[cfg_id])
    c.update(over)
    c["id"] = cfg_id
    return c


def _gen(device, seed):
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def _zipf_ids(rows, V, n, g, device, chunk=256):
    w = torch.arange(1, V + 1, device=device, dtype=torch.float32).pow(-1.1)
    out = torch.empty(rows, n, dtype=torch.int64, device=device)
    for s in range(0, rows, chunk):
        e = min(rows, s + chunk)
        out[s:e] = torch.multinomial(w.expand(e - s, V).contiguous(), n, replacement=False, generator=g)
    return out


def base_rows(cfg, set_idx=0, device="cpu", seed=None):
    """Binary32 base rows [R, D+1, V] and per-request target noise sd [R]."""
    R, D, V = cfg["R"], cfg["D"], cfg["V"]
    seed = GEN_SEED_BASE + cfg.get("id", 0) if seed is None else seed
    g = _gen(device, seed * 1000003 + set_idx)
    rows = R * (D + 1)
    z = torch.randn(rows, V, generator=g, device=device, dtype=torch.float32)
    cid = cfg.get("id", 0)
    if cfg["name"] == "tiny" or cid == 1:
        z.mul_(3.0)
        peaks = torch.multinomial(torch.ones(rows, V, device=device), 3, replacement=False, generator=g)
        z.scatter_add_(1, peaks, torch.full((rows, 3), 8.0, device=device))
        sigma = torch.full((R,), 1.0, device=device)
    else:
        lo, hi = (2.0, 5.0) if cfg["name"] in ("small", "qwen_vocab") else (1.0, 6.0)
        s = lo + (hi - lo) * torch.rand(rows, 1, generator=g, device=device)
        z.mul_(s)
        ids = _zipf_ids(rows, V, 16, g, device)
        boost = 6.0 / torch.sqrt(torch.arange(1, 17, device=device, dtype=torch.float32))
        z.scatter_add_(1, ids, boost.expand(rows, 16).contiguous())
        if cfg["name"] in ("small", "qwen_vocab"):
            sigma = torch.full((R,), 0.7, device=device)
        else:
            sigma = 0.3 + 1.2 * torch.rand(R, generator=g, device=device)
    return z.view(R, D + 1, V), sigma


def draft_from_base(cfg, base):
    """Draft logits [R, D, V] in the storage dtype."""
    return base[:, :cfg["D"]].to(TORCH_DTYPE[cfg["dtype"]]).contiguous()


def target_from_base(cfg, base, sigma, depth, set_idx=0, seed=None, out=None):
    """Target logits [R, B+1, V]: row n of request r = base[r, depth[r, n]] + sigma_r * N(0, 1).

    depth: int tensor [R, B+1]; entries < 0 (nodes the plan did not create)
    read base row 0. The noise does not depend on the depths.
    """
    R, B, V = cfg["R"], cfg["B"], cfg["V"]
    device = base.device
    seed = GEN_SEED_BASE + cfg.get("id", 0) if seed is None else seed
    g = _gen(device, seed * 1000003 + 7919 + set_idx)
    dt = TORCH_DTYPE[cfg["dtype"]]
    if out is None:
        out = torch.empty(R, B + 1, V, dtype=dt, device=device)
    depth = depth.to(device=device, dtype=torch.int64).clamp(min=0)
    for r in range(R):
        noise = torch.randn(B + 1, V, generator=g, device=device, dtype=torch.float32)
        rows = base[r].index_select(0, depth[r])
        out[r].copy_((rows + sigma[r] * noise).to(dt))
    return out


def transitions(cfg, P, scale=1.5, set_idx=0, device="cpu", seed=None):
    """Transition scores [R, D-1, P, P] (binary32): scale * N(0, 1) per entry.

    They stand in for a drafter's precomputed scores between the pool
    candidates of consecutive positions (the correction of pool slot j of
    position d after slot i of position d-1).
    """
    R, D = cfg["R"], cfg["D"]
    seed = GEN_SEED_BASE + cfg.get("id", 0) if seed is None else seed
    g = _gen(device, seed * 1000003 + 104729 + set_idx)
    t = torch.randn(R, max(D - 1, 0), P, P, generator=g, device=device, dtype=torch.float32)
    return t.mul_(scale).contiguous()


def bytes_per_step(cfg):
    """Algorithmic bytes of one round: every draft row and every target row read once."""
    b = 4 if cfg["dtype"] == "f32" else 2
    return cfg["R"] * cfg["D"] * cfg["V"] * b + cfg["R"] * (cfg["B"] + 1) * cfg["V"] * b


def describe(cfg):
    return "R=%d V=%d D=%d B=%d K=%d T=%g %s" % (cfg["R"], cfg["V"], cfg["D"], cfg["B"], cfg["K"],
                                                cfg["T"], cfg["dtype"])


__all__ = ["CONFIGS", "config", "base_rows", "draft_from_base", "target_from_base", "transitions",
           "replay_seed", "bytes_per_step", "describe"]
