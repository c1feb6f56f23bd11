"""Seeded synthetic inputs for Traversal Verification.

This module only draws random numbers and builds tree shapes: it holds none of
the verification arithmetic. It is the one piece of code that both sides of a
parity check share (the HIP library via tests and bench.py, the oracle via
tests); the library itself never imports it.

Recipes (arXiv 2505.12398 runs Llama models on Spec-Bench; these synthetic
inputs stand in for that workload with the same vocabulary sizes, tree shapes
and temperatures):

* logits: target z_b ~ N(0, 3^2) i.i.d. per entry, plus +6 on exactly
  round(0.01 V) distinct token ids per row (peaked distributions); draft
  z_s = z_b + N(0, sigma^2). Rows are independent per node.
* draft tokens: node i's token is drawn from its parent's tempered draft
  distribution softmax(z_s[parent] / T), either i.i.d. per child or without
  replacement across siblings, using Gumbel-max / Gumbel-top-k
  (argmax over z_s / T plus Gumbel noise), so no softmax is formed here.
* uniforms: u = k * 2^-24 with k uniform in [0, 2^24), so float32 and float64
  see the same value.
* shapes: chains, complete binary trees, and irregular BFS trees whose nodes
  draw a branching factor k in {1..4} with P(k) proportional to 2^-k.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

WITHOUT_REPLACEMENT = 0
WITH_REPLACEMENT = 1

U_SCALE = 2.0 ** -24


# ---------------------------------------------------------------------------
# Tree shapes (parents[i] < i, BFS order, children of a node contiguous)
# ---------------------------------------------------------------------------

def chain_parents(depth: int) -> np.ndarray:
    return np.arange(-1, depth, dtype=np.int32)


def binary_parents(levels: int) -> np.ndarray:
    n1 = 2 ** (levels + 1) - 1
    p = (np.arange(n1, dtype=np.int64) - 1) // 2
    p[0] = -1
    return p.astype(np.int32)


def geometric_bfs_parents(rng: np.random.Generator, n_nodes: int, max_depth: int,
                          max_tries: int = 100000) -> np.ndarray:
    """Irregular tree with exactly ``n_nodes`` draft nodes whose deepest node is
    at depth ``max_depth``. Breadth-first: every node above ``max_depth`` draws a
    branching factor k in {1,2,3,4} with P(k) proportional to 2^-k and appends
    that many children until the budget is used up; shapes that miss the budget
    or the depth are redrawn."""
    ks = np.array([1, 2, 3, 4])
    pk = 2.0 ** -ks
    pk /= pk.sum()
    for _ in range(max_tries):
        parents = [-1]
        depth = [0]
        head = 0
        while head < len(parents) and len(parents) - 1 < n_nodes:
            if depth[head] < max_depth:
                k = int(rng.choice(ks, p=pk))
                k = min(k, n_nodes - (len(parents) - 1))
                for _ in range(k):
                    parents.append(head)
                    depth.append(depth[head] + 1)
            head += 1
        if len(parents) - 1 == n_nodes and max(depth) == max_depth:
            return np.asarray(parents, dtype=np.int32)
    raise RuntimeError("could not draw a tree with the requested size and depth")


def node_depths(parents) -> np.ndarray:
    d = np.zeros(len(parents), dtype=np.int32)
    for i in range(1, len(parents)):
        d[i] = d[int(parents[i])] + 1
    return d


def sibling_rank(parents) -> np.ndarray:
    """Position of each node among its parent's children (index order)."""
    r = np.zeros(len(parents), dtype=np.int32)
    count = {}
    for i in range(1, len(parents)):
        j = int(parents[i])
        r[i] = count.get(j, 0)
        count[j] = r[i] + 1
    return r


def uniforms_np(rng: np.random.Generator, shape) -> np.ndarray:
    return (rng.integers(0, 2 ** 24, size=shape) * U_SCALE).astype(np.float32)


# ---------------------------------------------------------------------------
# Context-keyed model for exact checks (every token path has its own rows)
# ---------------------------------------------------------------------------

class ContextModel:
    """A toy autoregressive model pair: for every context (tuple of tokens after
    the root) the target logits are N(0, sigma_target^2) per entry and the draft
    logits add N(0, sigma_noise^2). Rows are keyed by (seed, context) so any
    context can be regenerated on its own."""

    def __init__(self, vocab: int, seed: int = 0, sigma_target: float = 2.0,
                 sigma_noise: float = 1.0):
        self.vocab = vocab
        self.seed = seed
        self.sigma_target = sigma_target
        self.sigma_noise = sigma_noise
        self._cache = {}

    def _rows(self, ctx):
        ctx = tuple(int(x) for x in ctx)
        if ctx not in self._cache:
            ss = np.random.SeedSequence([self.seed, len(ctx)] + list(ctx))
            rng = np.random.default_rng(ss)
            zb = rng.normal(0.0, self.sigma_target, self.vocab)
            zs = zb + rng.normal(0.0, self.sigma_noise, self.vocab)
            self._cache[ctx] = (zb, zs)
        return self._cache[ctx]

    def target(self, ctx):
        return self._rows(ctx)[0]

    def draft(self, ctx):
        return self._rows(ctx)[1]


def gumbel_np(rng, size):
    return -np.log(rng.exponential(1.0, size))


def draw_context_tree(rng: np.random.Generator, model: ContextModel, parents, T: float,
                      mode: int):
    """Draw a draft tree's tokens from the context model (children from the
    parent's tempered draft distribution), and return (tokens, zb, zs) with the
    per-node rows. Gumbel-max per child (i.i.d.) or Gumbel-top-k per parent
    (without replacement)."""
    n1 = len(parents)
    tokens = np.zeros(n1, dtype=np.int32)
    ctx = [()] * n1
    kids = [[] for _ in range(n1)]
    for i in range(1, n1):
        kids[int(parents[i])].append(i)
    for j in range(n1):
        if not kids[j]:
            continue
        zs_j = np.asarray(model.draft(ctx[j])) / np.float64(np.float32(T))
        if mode == WITH_REPLACEMENT:
            for c in kids[j]:
                tokens[c] = int(np.argmax(zs_j + gumbel_np(rng, model.vocab)))
        else:
            order = np.argsort(-(zs_j + gumbel_np(rng, model.vocab)), kind="stable")
            for r, c in enumerate(kids[j]):
                tokens[c] = int(order[r])
        for c in kids[j]:
            ctx[c] = ctx[j] + (int(tokens[c]),)
    zb = np.stack([model.target(c) for c in ctx])
    zs = np.stack([model.draft(c) for c in ctx])
    return tokens, zb, zs


# ---------------------------------------------------------------------------
# The paper's illustrative tree (Sec. 2.1 Table 1 distributions, Sec. 3.2 tree)
# ---------------------------------------------------------------------------

def worked_example():
    """Vocabulary [a, b, c] = [0, 1, 2]; every node has target [.3, .4, .3] and
    draft [.6, .3, .1] (Table 1); the two-layer tree of Fig. 1 with
    [X1..X5] = [a, c, b, c, a] (Sec. 3.2); temperature 1. Logits are the natural
    logarithms of the probabilities."""
    parents = np.array([-1, 0, 0, 1, 1, 2], dtype=np.int32)
    tokens = np.array([0, 0, 2, 1, 2, 0], dtype=np.int32)
    zb = np.tile(np.log(np.array([0.3, 0.4, 0.3])), (6, 1))
    zs = np.tile(np.log(np.array([0.6, 0.3, 0.1])), (6, 1))
    return parents, tokens, zb, zs, 1.0


# ---------------------------------------------------------------------------
# Batched synthetic workloads (torch; runs on the CPU or on the GPU)
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class Config:
    name: str
    batch: int
    shape: str          # "binary", "chain", "geometric"
    n_nodes: int        # draft nodes N (rows per tree = N + 1)
    depth: int
    vocab: int
    dtype: str          # "f32" or "bf16"
    temperature: float
    noise: str          # "const" or "depth"
    noise_sigma: float = 1.5


CONFIGS = {
    # config 1 (tiny exact case) uses ContextModel instead; listed for its shape.
    1: Config("tiny-binary-d2-V8", 1, "binary", 6, 2, 8, "f32", 1.0, "const", 1.0),
    2: Config("chain-d5-B64-V32000", 64, "chain", 5, 5, 32000, "f32", 1.0, "const"),
    3: Config("binary-d4-B32-V128256", 32, "binary", 30, 4, 128256, "bf16", 0.7, "const"),
    4: Config("irregular-N60-d6-B16-V151936", 16, "geometric", 60, 6, 151936, "bf16", 1.0,
              "depth"),
    5: Config("irregular-N64-d7-B256-V128256", 256, "geometric", 64, 7, 128256, "bf16", 1.0,
              "const"),
}


def _seed(*keys) -> int:
    return int(np.random.SeedSequence([int(k) for k in keys]).generate_state(1, np.uint64)[0]
               & np.uint64(0x7FFFFFFFFFFFFFFF))


def make_parents(cfg: Config, batch: int, seed_keys) -> np.ndarray:
    """[B][N+1] int32 parents for a config (every tree its own shape if irregular)."""
    if cfg.shape == "chain":
        one = chain_parents(cfg.depth)
        return np.tile(one, (batch, 1))
    if cfg.shape == "binary":
        one = binary_parents(cfg.depth)
        return np.tile(one, (batch, 1))
    out = np.empty((batch, cfg.n_nodes + 1), dtype=np.int32)
    for b in range(batch):
        rng = np.random.default_rng(np.random.SeedSequence(list(seed_keys) + [1, b]))
        out[b] = geometric_bfs_parents(rng, cfg.n_nodes, cfg.depth)
    return out


def boost_count(vocab: int) -> int:
    return int(round(0.01 * vocab))


def _coprime_strides(vocab: int, count: int = 64) -> np.ndarray:
    """Strides s with gcd(s, V) = 1 spread over [V/7, V/2]: the affine walk
    (o + s*j) mod V then visits distinct ids."""
    out = []
    s = max(3, vocab // 7)
    while len(out) < count and s < vocab:
        if math.gcd(s, vocab) == 1:
            out.append(s)
            s += max(1, vocab // (3 * count))
        else:
            s += 1
    if not out:
        out = [1]
    return np.asarray(out, dtype=np.int64)


def make_logits(cfg: Config, parents: np.ndarray, vocab: int, seed: int, device,
                boost: bool = True):
    """Target and draft logits [B][N+1][V] as float32 torch tensors on device."""
    import torch
    B, n1 = parents.shape
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    zb = torch.randn((B, n1, vocab), generator=g, device=device, dtype=torch.float32)
    zb.mul_(3.0)
    if boost:
        K = boost_count(vocab)
        strides = torch.as_tensor(_coprime_strides(vocab), device=device)
        off = torch.randint(0, vocab, (B, n1, 1), generator=g, device=device)
        pick = torch.randint(0, len(strides), (B, n1, 1), generator=g, device=device)
        j = torch.arange(K, device=device).view(1, 1, K)
        ids = (off + strides[pick] * j) % vocab
        zb.scatter_add_(2, ids, torch.full(ids.shape, 6.0, device=device))
    noise = torch.randn((B, n1, vocab), generator=g, device=device, dtype=torch.float32)
    if cfg.noise == "depth":
        d = torch.as_tensor(np.stack([node_depths(p) for p in parents]), device=device)
        sigma = 0.8 + 1.2 * torch.clamp(d, max=5).to(torch.float32) / 5.0
        noise.mul_(sigma.unsqueeze(-1))
    else:
        noise.mul_(cfg.noise_sigma)
    zs = zb + noise
    del noise
    return zb, zs


def draw_tokens(parents: np.ndarray, draft, temperature: float, mode: int, seed: int,
                chunk: int = 16):
    """Children tokens drawn from the parent's tempered draft distribution.
    ``draft`` is the [B][N+1][V] tensor the verifier will read (its values are
    used after conversion to float32). Gumbel-max for i.i.d. children,
    Gumbel-top-k (one perturbation per parent) without replacement."""
    import torch
    device = draft.device
    B, n1 = parents.shape
    invT = 1.0 / float(np.float32(temperature))
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    tokens = torch.zeros((B, n1), dtype=torch.int32, device=device)
    par = torch.as_tensor(parents, device=device, dtype=torch.int64)
    ranks = torch.as_tensor(np.stack([sibling_rank(p) for p in parents]), device=device,
                            dtype=torch.int64)
    for b0 in range(0, B, chunk):
        b1 = min(B, b0 + chunk)
        rows = draft[b0:b1].to(torch.float32) * invT           # [b, n1, V]
        if mode == WITH_REPLACEMENT:
            pr = rows.gather(1, par[b0:b1, 1:].unsqueeze(-1).expand(-1, -1, rows.shape[-1]))
            gum = torch.empty_like(pr).exponential_(generator=g).log_().neg_()
            tokens[b0:b1, 1:] = torch.argmax(pr + gum, dim=-1).to(torch.int32)
        else:
            gum = torch.empty_like(rows).exponential_(generator=g).log_().neg_()
            kmax = int(ranks.max().item()) + 1
            top = torch.topk(rows + gum, kmax, dim=-1).indices    # [b, n1, kmax]
            pick = top.gather(1, par[b0:b1, 1:].unsqueeze(-1).expand(-1, -1, kmax))
            tokens[b0:b1, 1:] = pick.gather(2, ranks[b0:b1, 1:].unsqueeze(-1)).squeeze(-1) \
                .to(torch.int32)
        del rows
    return tokens


def windowed_parents(rng: np.random.Generator, n_nodes: int, window: int) -> np.ndarray:
    """Random recursive tree of ``n_nodes`` draft nodes: node i's parent is
    uniform over the ``window`` nodes before it (all earlier nodes while
    i <= window), so depth grows about as 2N / window and nodes have a few
    children each."""
    parents = np.empty(n_nodes + 1, dtype=np.int32)
    parents[0] = -1
    for i in range(1, n_nodes + 1):
        parents[i] = rng.integers(max(0, i - window), i)
    return parents


DEEP_NAME = "deep-N767-w64-B8-V128256"


def make_deep_batch(batch: int = 8, n_nodes: int = 767, window: int = 64, vocab: int = 128256,
                    step: int = 0, device="cpu", mode: int = WITHOUT_REPLACEMENT, seed: int = 0,
                    dtype: str = "bf16"):
    """Large, deep trees at the scale of the paper's Sequoia comparison
    (hundreds of nodes, depth above 20): ``windowed_parents`` trees with the
    large-batch workload's logit law (target N(0, 3^2) plus the sparse +6
    boosts, draft = target + N(0, 1.5^2), T = 1), tokens drawn from the
    parent's draft in the given sibling mode, uniforms k * 2^-24."""
    import torch
    cfg = CONFIGS[5]
    keys = (seed, 99, step)
    parents = np.empty((batch, n_nodes + 1), dtype=np.int32)
    for b in range(batch):
        rng = np.random.default_rng(np.random.SeedSequence(list(keys) + [1, b]))
        parents[b] = windowed_parents(rng, n_nodes, window)
    zb, zs = make_logits(cfg, parents, vocab, _seed(*keys, 2), device)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    zb = zb.to(tdt)
    zs = zs.to(tdt)
    tokens = draw_tokens(parents, zs, cfg.temperature, mode, _seed(*keys, 3), chunk=2)
    g = torch.Generator(device=device)
    g.manual_seed(_seed(*keys, 4))
    u = torch.randint(0, 2 ** 24, parents.shape, generator=g, device=device).to(torch.float32)
    u.mul_(U_SCALE)
    return {
        "config": cfg, "parents": torch.as_tensor(parents, device=device),
        "tokens": tokens, "target": zb, "draft": zs, "uniforms": u,
        "temperature": cfg.temperature, "mode": mode, "dtype": dtype,
    }


def make_batch(cfg_id: int, step: int = 0, device="cpu", mode: int = WITHOUT_REPLACEMENT,
               batch: int | None = None, vocab: int | None = None, seed: int = 0):
    """One batch of a config: dict with parents, tokens, target, draft (dtype of
    the config), uniforms, temperature, mode, dtype. ``batch``/``vocab`` shrink
    the config for quick runs; shapes, distributions and temperature stay."""
    import torch
    cfg = CONFIGS[cfg_id]
    B = batch or cfg.batch
    V = vocab or cfg.vocab
    keys = (seed, cfg_id, step)
    parents = make_parents(cfg, B, keys)
    zb, zs = make_logits(cfg, parents, V, _seed(*keys, 2), device)
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    zb = zb.to(tdt)
    zs = zs.to(tdt)
    tokens = draw_tokens(parents, zs, cfg.temperature, mode, _seed(*keys, 3))
    g = torch.Generator(device=device)
    g.manual_seed(_seed(*keys, 4))
    u = torch.randint(0, 2 ** 24, parents.shape, generator=g, device=device).to(torch.float32)
    u.mul_(U_SCALE)
    return {
        "config": cfg, "parents": torch.as_tensor(parents, device=device),
        "tokens": tokens, "target": zb, "draft": zs, "uniforms": u,
        "temperature": cfg.temperature, "mode": mode, "dtype": cfg.dtype,
    }


def tree_numpy(batch: dict, b: int):
    """Host copies of tree b for the oracle: (parents, tokens, target, draft,
    uniforms) with bf16 logits as uint16 bit patterns."""
    import torch

    def rows(t):
        t = t[b].detach().cpu()
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).numpy().view(np.uint16)
        return t.numpy()

    return (batch["parents"][b].cpu().numpy(), batch["tokens"][b].cpu().numpy(),
            rows(batch["target"]), rows(batch["draft"]), batch["uniforms"][b].cpu().numpy())
