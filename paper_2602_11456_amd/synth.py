"""Seeded synthetic weight pairs for the sparse delta checkpoint.

This module only draws inputs.  It holds none of the delta arithmetic (no
compare, compaction or scatter), so both the GPU library's tests and the CPU
oracle's tests consume the same bytes from it.

The paper measures real Qwen3 reinforcement-learning steps (Sec. 3, Sec. 6).
Those checkpoints are not available, so these generators stand in for them:

* ``prev`` is ``bf16(N(0, 0.02))`` (round to nearest even), RMSNorm vectors
  are exactly 1.0.  The weight-magnitude table of the appendix is the
  realism reference for this scale; the extract path compares bits, so the
  values do not change its cost.
* ``new`` equals ``prev`` except at exactly ``K_t = floor(rho * n_t + 1/2)``
  distinct positions per tensor drawn uniformly without replacement, where
  the word is replaced by ``bf16(prev + N(0, 1e-3))``, redrawn up to 64
  times until its bit pattern differs; a position still equal after that
  gets its lowest mantissa bit flipped.  So every planted position differs
  in bits and every other position is identical: the number of changed
  words is known by construction.  ``rho`` of about 1% matches the per-step
  density the paper reports for Qwen3 models (Sec. 3, Eq. 1).
* The clustered variant puts 80% of the changes into randomly chosen rows
  of the embedding, the LM head and the attention projections, covering 5%
  of all elements, and spreads the rest uniformly over the other elements.

Tensor lists follow the public Qwen3 architecture in the canonical order
``embed_tokens``; per layer ``input_layernorm, q_proj, k_proj, v_proj,
o_proj, q_norm, k_norm, post_attention_layernorm, gate_proj, up_proj,
down_proj``; ``norm``; ``lm_head`` (untied models only).  Linear weights are
``[out_features, in_features]``.  q, k and v are adjacent, so their global
offsets coincide with those of a fused ``qkv_proj`` block (Sec. 5.1).

Every tensor has its own seed derived from the base seed and its position,
so any tensor can be regenerated alone.  Draws use ``torch.Generator`` on the
requested device; CPU and GPU draws of the same seed differ, so a test that
compares against the oracle copies the generated tensors to the host.
"""
from __future__ import annotations

import dataclasses
from fractions import Fraction
from typing import List, Optional, Sequence, Tuple

import torch

BASE_SEED = 11456

QWEN3 = {
    # layers, hidden, q heads, kv heads, head dim, MLP width, vocab, tied
    "qwen3-4b": dict(layers=36, hidden=2560, q_heads=32, kv_heads=8,
                     head_dim=128, mlp=9728, vocab=151936, tied=True),
    "qwen3-8b": dict(layers=36, hidden=4096, q_heads=32, kv_heads=8,
                     head_dim=128, mlp=12288, vocab=151936, tied=False),
    "qwen3-14b": dict(layers=40, hidden=5120, q_heads=40, kv_heads=8,
                      head_dim=128, mlp=17408, vocab=151936, tied=False),
    # the same structure at toy sizes, for tests
    "qwen3-tiny": dict(layers=2, hidden=64, q_heads=4, kv_heads=2,
                       head_dim=16, mlp=96, vocab=500, tied=False),
}

NORM_KINDS = ("input_layernorm", "q_norm", "k_norm",
              "post_attention_layernorm", "norm")


def qwen3_tensor_table(model: str) -> List[Tuple[str, Tuple[int, ...]]]:
    """(name, shape) of every parameter tensor in canonical order."""
    c = QWEN3[model]
    h, qd, kvd = c["hidden"], c["q_heads"] * c["head_dim"], c["kv_heads"] * c["head_dim"]
    out = [("model.embed_tokens.weight", (c["vocab"], h))]
    for layer in range(c["layers"]):
        p = f"model.layers.{layer}."
        out += [
            (p + "input_layernorm.weight", (h,)),
            (p + "self_attn.q_proj.weight", (qd, h)),
            (p + "self_attn.k_proj.weight", (kvd, h)),
            (p + "self_attn.v_proj.weight", (kvd, h)),
            (p + "self_attn.o_proj.weight", (h, qd)),
            (p + "self_attn.q_norm.weight", (c["head_dim"],)),
            (p + "self_attn.k_norm.weight", (c["head_dim"],)),
            (p + "post_attention_layernorm.weight", (h,)),
            (p + "mlp.gate_proj.weight", (c["mlp"], h)),
            (p + "mlp.up_proj.weight", (c["mlp"], h)),
            (p + "mlp.down_proj.weight", (h, c["mlp"])),
        ]
    out.append(("model.norm.weight", (h,)))
    if not c["tied"]:
        out.append(("lm_head.weight", (c["vocab"], h)))
    return out


def qwen3_fused_layout(model: str):
    """The inference engine's fused parameter list (Sec. 5.1): per layer
    ``qkv_proj`` stacks the rows of q, k and v and ``gate_up_proj`` those of
    gate and up; every other tensor keeps its own name.  Target order:
    ``embed_tokens``; per layer ``qkv_proj, o_proj, q_norm, k_norm,
    gate_up_proj, down_proj, input_layernorm, post_attention_layernorm``;
    ``norm``; ``lm_head``.

    Returns ``(targets, sources)``: ``targets`` is a list of ``(name,
    numel)`` in target order, ``sources[t] = (target index, word offset of
    its block)`` for every tensor of ``qwen3_tensor_table`` in its order.
    Stacking rows of row-major matrices puts each block's flat words at a
    fixed word offset, so a block offset is a sum of numels."""
    table = qwen3_tensor_table(model)
    size = {name: numel(shape) for name, shape in table}
    c = QWEN3[model]
    targets = [("model.embed_tokens.weight", size["model.embed_tokens.weight"])]
    where = {"model.embed_tokens.weight": (0, 0)}
    for layer in range(c["layers"]):
        p = f"model.layers.{layer}."
        q, k, v = (p + f"self_attn.{x}_proj.weight" for x in "qkv")
        g, u = p + "mlp.gate_proj.weight", p + "mlp.up_proj.weight"

        def add(name, parts):
            off = 0
            for part in parts:
                where[part] = (len(targets), off)
                off += size[part]
            targets.append((name, off))

        add(p + "self_attn.qkv_proj.weight", [q, k, v])
        for single in ("self_attn.o_proj", "self_attn.q_norm", "self_attn.k_norm"):
            add(p + single + ".weight", [p + single + ".weight"])
        add(p + "mlp.gate_up_proj.weight", [g, u])
        for single in ("mlp.down_proj", "input_layernorm", "post_attention_layernorm"):
            add(p + single + ".weight", [p + single + ".weight"])
    where["model.norm.weight"] = (len(targets), 0)
    targets.append(("model.norm.weight", size["model.norm.weight"]))
    if not c["tied"]:
        where["lm_head.weight"] = (len(targets), 0)
        targets.append(("lm_head.weight", size["lm_head.weight"]))
    return targets, [where[name] for name, _ in table]


def is_norm(name: str) -> bool:
    return name.rsplit(".", 2)[-2] in NORM_KINDS


def numel(shape: Sequence[int]) -> int:
    n = 1
    for s in shape:
        n *= int(s)
    return n


def planted_count(n: int, density) -> int:
    """floor(density * n + 1/2), exact in rational arithmetic."""
    d = Fraction(str(density)) if not isinstance(density, Fraction) else density
    return int((2 * n * d.numerator + d.denominator) // (2 * d.denominator))


def tensor_seed(base: int, t: int) -> int:
    """Deterministic 63-bit seed of tensor t (splitmix64 finaliser)."""
    z = (base * 0x9E3779B97F4A7C15 + (t + 1) * 0xBF58476D1CE4E5B9) & ((1 << 64) - 1)
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & ((1 << 64) - 1)
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & ((1 << 64) - 1)
    z ^= z >> 31
    return z & ((1 << 63) - 1)


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def draw_prev(n: int, g: torch.Generator, device, norm: bool = False) -> torch.Tensor:
    """bf16(N(0, 0.02)) flat tensor, or all-ones for a norm vector."""
    if norm:
        return torch.ones(n, dtype=torch.bfloat16, device=device)
    x = torch.randn(n, generator=g, device=device, dtype=torch.float32)
    return x.mul_(0.02).to(torch.bfloat16)


def perturb_words(old: torch.Tensor, g: torch.Generator, rounds: int = 64,
                  sigma: float = 1e-3) -> torch.Tensor:
    """bf16 words that differ in bits from ``old`` (see module doc)."""
    old_bits = old.view(torch.int16)
    out = torch.empty_like(old)
    todo = torch.arange(old.numel(), device=old.device)
    for _ in range(rounds):
        if todo.numel() == 0:
            break
        noise = torch.randn(todo.numel(), generator=g, device=old.device,
                            dtype=torch.float32)
        cand = (old[todo].float() + noise * sigma).to(torch.bfloat16)
        out[todo] = cand
        same = cand.view(torch.int16) == old_bits[todo]
        todo = todo[same]
    if todo.numel():
        out.view(torch.int16)[todo] = old_bits[todo] ^ 1
    return out


def plant(prev: torch.Tensor, positions: torch.Tensor, g: torch.Generator) -> torch.Tensor:
    """Copy of ``prev`` with the words at ``positions`` (distinct) changed."""
    new = prev.clone()
    if positions.numel():
        new[positions] = perturb_words(prev[positions], g)
    return new


def uniform_positions(n: int, k: int, g: torch.Generator, device) -> torch.Tensor:
    """k distinct positions in [0, n), uniform without replacement, sorted."""
    if k == 0 or n == 0:
        return torch.empty(0, dtype=torch.int64, device=device)
    if k > n:
        raise ValueError("more positions than elements")
    pos = torch.randperm(n, generator=g, device=device)[:k]
    return torch.sort(pos).values


def make_pair(n: int, density=0.01, seed: int = BASE_SEED, device="cpu",
              norm: bool = False, k: Optional[int] = None):
    """One flat bf16 pair (prev, new) and the sorted planted positions."""
    g = _gen(seed, device)
    prev = draw_prev(n, g, device, norm=norm)
    kk = planted_count(n, density) if k is None else int(k)
    pos = uniform_positions(n, kk, g, device)
    return prev, plant(prev, pos, g), pos


@dataclasses.dataclass
class WeightSet:
    model: str
    names: List[str]
    shapes: List[Tuple[int, ...]]
    prev: List[torch.Tensor]
    new: List[torch.Tensor]
    planted: List[int]          # number of changed words per tensor

    @property
    def numels(self) -> List[int]:
        return [numel(s) for s in self.shapes]

    @property
    def total(self) -> int:
        return sum(self.numels)

    @property
    def total_planted(self) -> int:
        return sum(self.planted)


def make_weight_set(model: str, density=0.01, seed: int = BASE_SEED,
                    device="cpu", clustered: bool = False,
                    tensors: Optional[Sequence[int]] = None) -> WeightSet:
    """A Qwen3-shaped (prev, new) set.  ``tensors`` restricts generation to
    a subset of tensor positions (seeds stay those of the full set)."""
    table = qwen3_tensor_table(model)
    sel = list(range(len(table))) if tensors is None else list(tensors)
    if clustered:
        return _make_clustered(model, table, density, seed, device, sel)
    ws = WeightSet(model, [], [], [], [], [])
    for t in sel:
        name, shape = table[t]
        n = numel(shape)
        prev, new, pos = make_pair(n, density, tensor_seed(seed, t), device,
                                   norm=is_norm(name))
        ws.names.append(name)
        ws.shapes.append(shape)
        ws.prev.append(prev.view(shape))
        ws.new.append(new.view(shape))
        ws.planted.append(int(pos.numel()))
    return ws


def _hot_candidates(table):
    """(tensor position, rows) of the tensors whose rows may be hot."""
    keys = ("embed_tokens", "lm_head", "q_proj", "k_proj", "v_proj", "o_proj")
    return [(t, shape[0]) for t, (name, shape) in enumerate(table)
            if len(shape) == 2 and any(k in name for k in keys)]


def clustered_plan(model: str, density=0.01, hot_frac=Fraction(1, 20),
                   hot_share=Fraction(4, 5)):
    """Sizes of the clustered variant: (hot row count, hot elements, K, K_hot, K_cold)."""
    table = qwen3_tensor_table(model)
    N = sum(numel(s) for _, s in table)
    row_len = {table[t][1][1] for t, _ in _hot_candidates(table)}
    if len(row_len) != 1:
        raise ValueError("hot candidate rows must share one length")
    L = row_len.pop()
    hot_rows = -(-(N * hot_frac.numerator) // (hot_frac.denominator * L))
    H = hot_rows * L
    K = planted_count(N, density)
    K_hot = planted_count(K, hot_share)
    return hot_rows, H, K, K_hot, K - K_hot


def _make_clustered(model, table, density, seed, device, sel):
    """80% of the changes in randomly chosen rows covering 5% of the
    elements; the rest uniform over all other elements."""
    N = sum(numel(s) for _, s in table)
    hot_rows, H, K, K_hot, K_cold = clustered_plan(model, density)
    cands = _hot_candidates(table)
    L = table[cands[0][0]][1][1]
    g = _gen(tensor_seed(seed, 1_000_000), device)
    total_rows = sum(r for _, r in cands)
    chosen = torch.sort(torch.randperm(total_rows, generator=g, device=device)[:hot_rows]).values
    # global start position of every candidate row, in candidate order
    bases = []
    acc = 0
    for _, shape in table:
        bases.append(acc)
        acc += numel(shape)
    row_starts = torch.cat([
        bases[t] + torch.arange(r, device=device, dtype=torch.int64) * L for t, r in cands])
    hot_start = torch.sort(row_starts[chosen]).values          # [hot_rows]
    # K_hot uniform over the hot elements
    hp = torch.sort(torch.randperm(H, generator=g, device=device)[:K_hot]).values
    hot_pos = hot_start[hp // L] + hp % L
    # K_cold uniform over the N - H other elements: distinct ordinals by
    # oversampling with replacement and keeping a random subset of the
    # unique draws, then mapping ordinal o to the position o + L * (number
    # of hot rows whose non-hot ordinal start is <= o).
    NC = N - H
    cold = torch.empty(0, dtype=torch.int64, device=device)
    m = K_cold + K_cold // 50 + 1024
    while cold.numel() < K_cold:
        draw = torch.randint(0, NC, (m,), generator=g, device=device, dtype=torch.int64)
        cold = torch.unique(torch.cat([cold, draw]))
        m = 2 * m
    keep = torch.randperm(cold.numel(), generator=g, device=device)[:K_cold]
    cold = torch.sort(cold[keep]).values
    c = hot_start - L * torch.arange(hot_rows, device=device, dtype=torch.int64)
    cold_pos = cold + L * torch.searchsorted(c, cold, right=True)
    all_pos = torch.sort(torch.cat([hot_pos, cold_pos])).values
    ws = WeightSet(model, [], [], [], [], [])
    for t in sel:
        name, shape = table[t]
        n = numel(shape)
        gt = _gen(tensor_seed(seed, t), device)
        prev = draw_prev(n, gt, device, norm=is_norm(name))
        lo = torch.searchsorted(all_pos, torch.tensor([bases[t]], device=device))
        hi = torch.searchsorted(all_pos, torch.tensor([bases[t] + n], device=device))
        pos = all_pos[int(lo):int(hi)] - bases[t]
        new = plant(prev, pos, gt)
        ws.names.append(name)
        ws.shapes.append(shape)
        ws.prev.append(prev.view(shape))
        ws.new.append(new.view(shape))
        ws.planted.append(int(pos.numel()))
    return ws


CONFIGS = {
    1: dict(kind="single", n=2048 * 2048, density=0.01, index="int32"),
    2: dict(kind="set", model="qwen3-4b", density=0.01, index="int64"),
    3: dict(kind="set", model="qwen3-8b", density=0.01, index="int64"),
    4: dict(kind="set", model="qwen3-8b", density=0.01, index="int64", clustered=True),
    5: dict(kind="set", model="qwen3-14b", density=0.01, index="int64",
            chunk_elems=1 << 27, num_streams=4),
}


def config_seed(cfg: int) -> int:
    return BASE_SEED + cfg
