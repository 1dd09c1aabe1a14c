"""Seeded synthetic workloads for BSR pruning and BSR x dense products.

This module holds no pruning or product arithmetic: it only draws random tensors with the shapes
and scales of the BERT attention projections, and shapes the per-block-row nonzero counts of the
skewed workload.  Both the GPU tests and the CPU oracle tests take their inputs from here.

Value scales stand in for a trained, pruned BERT (whose weights and data are not available):
weights and biases ~ N(0, 0.02) (BERT's initialiser scale), activations ~ N(0, 1) (post-LayerNorm
hidden states).  Every tensor is drawn as fp64 standard normals from numpy's PCG64 generator with
its own seed, scaled in fp64 and rounded to fp32.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

W_SIGMA = 0.02
B_SIGMA = 0.02
X_SIGMA = 1.0


def draw_normal(seed: int, shape, sigma: float) -> np.ndarray:
    """fp32 tensor of N(0, sigma^2) draws: PCG64(seed) standard normals in fp64, times sigma."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return (rng.standard_normal(shape) * float(sigma)).astype(np.float32)


def item_seed(config: int, item: int) -> int:
    """Seed of item `item` of workload number `config`: 1000 * config + item."""
    return 1000 * int(config) + int(item)


# ---------------------------------------------------------------------------------------------
# Skewed block-row counts (BERT-large stress workload)
# ---------------------------------------------------------------------------------------------


def zipf_counts(nrows: int, cap: int, total: int, s: float = 1.2) -> np.ndarray:
    """Per-rank nonzero-block counts: Zipf(s) shares of `total`, capped at `cap` per row.

    1. rank r (1-based) gets a share proportional to r**-s;
    2. rows over the cap are pinned at the cap and the excess is re-spread, in proportion, over
       the rows not yet pinned, until no row exceeds the cap;
    3. the real shares are rounded to integers summing to `total` by largest remainder, ties to
       the lower rank.
    Returns int64[nrows] in rank order (non-increasing).
    """
    if total > nrows * cap or total < 0:
        raise ValueError("total does not fit under the cap")
    w = np.arange(1, nrows + 1, dtype=np.float64) ** (-float(s))
    share = np.zeros(nrows, dtype=np.float64)
    pinned = np.zeros(nrows, dtype=bool)
    while True:
        free = ~pinned
        left = total - cap * int(pinned.sum())
        share[free] = left * w[free] / w[free].sum()
        share[pinned] = cap
        over = free & (share > cap)
        if not over.any():
            break
        pinned |= over
    base = np.floor(share).astype(np.int64)
    rem = share - base
    short = int(total - base.sum())
    if short > 0:
        order = sorted(range(nrows), key=lambda r: (-rem[r], r))
        for r in order[:short]:
            base[r] += 1
    return base


def zipf_block_mask(counts_by_rank: np.ndarray, Kb: int, seed: int) -> np.ndarray:
    """bool[Nb, Kb] block pattern whose row counts are `counts_by_rank` under a seeded shuffle.

    Ranks are mapped to block-rows by a seeded permutation; within each row the nonzero block
    columns are a seeded uniform choice.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    Nb = counts_by_rank.size
    perm = rng.permutation(Nb)
    mask = np.zeros((Nb, Kb), dtype=bool)
    for rank, row in enumerate(perm):
        cols = rng.choice(Kb, size=int(counts_by_rank[rank]), replace=False)
        mask[row, cols] = True
    return mask


def apply_block_mask(W: np.ndarray, R: int, C: int, mask: np.ndarray) -> np.ndarray:
    """Copy of W with every block outside `mask` set to +0.0 (input shaping only)."""
    N, K = W.shape
    Nb, Kb = N // R, K // C
    m = np.repeat(np.repeat(mask.reshape(Nb, Kb), R, axis=0), C, axis=1)
    out = W.copy()
    out[~m] = 0.0
    return out


# ---------------------------------------------------------------------------------------------
# The five workloads
# ---------------------------------------------------------------------------------------------


@dataclass
class Projection:
    """One weight to prune and multiply: dense W [N, K], bias [N], block shape and density."""
    name: str
    W: np.ndarray
    bias: np.ndarray
    R: int
    C: int
    density: float
    k: int | None = None   # block count when it is fixed by the workload (skewed rows)
    x_index: int = 0        # which activation matrix of the workload it multiplies


@dataclass
class Workload:
    name: str
    X: list[np.ndarray]
    projections: list[Projection]
    bf16: bool = False
    notes: dict = field(default_factory=dict)

    @property
    def tokens(self) -> int:
        return self.X[0].shape[0]


SHAPES_SWEEP = [(1, 1), (8, 1), (16, 1), (32, 1), (1, 32), (4, 4), (8, 8), (16, 16), (32, 32)]
QKV_DENSITIES = [0.05, 0.10, 0.20, 0.40]


def single_768(seed_config: int = 1) -> Workload:
    """One 768x768 weight, 32x1 blocks, density 0.2; X 128x768; bias 768."""
    W = draw_normal(item_seed(seed_config, 0), (768, 768), W_SIGMA)
    b = draw_normal(item_seed(seed_config, 1), (768,), B_SIGMA)
    X = draw_normal(item_seed(seed_config, 2), (128, 768), X_SIGMA)
    return Workload("single_768_32x1_d20_T128", [X], [Projection("W", W, b, 32, 1, 0.2)])


def bert_base_attention(R: int = 32, C: int = 1, density: float = 0.1,
                        tokens: int = 128, seed_config: int = 2) -> Workload:
    """BERT-base attention projections Q, K, V, O (768x768 each), batch 1 x seq 128 tokens.

    One activation matrix feeds all four projections (the O projection would read the attention
    context in a real layer; its shape and cost are the same).
    """
    names = ["Q", "K", "V", "O"]
    Ws = [draw_normal(item_seed(seed_config, n), (768, 768), W_SIGMA) for n in range(4)]
    bs = [draw_normal(item_seed(seed_config, 4 + n), (768,), B_SIGMA) for n in range(4)]
    X = draw_normal(item_seed(seed_config, 8), (tokens, 768), X_SIGMA)
    projs = [Projection(nm, W, b, R, C, density) for nm, W, b in zip(names, Ws, bs)]
    return Workload(f"bert_base_attn_qkvo_768_{R}x{C}_d{int(round(density * 100))}_T{tokens}",
                    [X], projs)


def block_sweep(R: int, C: int, density: float = 0.1, seed_config: int = 3) -> Workload:
    """One 768x768 weight at density 0.1 for a block shape of the sweep; X 128x768."""
    W = draw_normal(item_seed(seed_config, 0), (768, 768), W_SIGMA)
    b = draw_normal(item_seed(seed_config, 1), (768,), B_SIGMA)
    X = draw_normal(item_seed(seed_config, 2), (128, 768), X_SIGMA)
    return Workload(f"sweep_768_{R}x{C}_d{int(round(density * 100))}_T128", [X],
                    [Projection("W", W, b, R, C, density)])


def fused_qkv(R: int, C: int, density: float, bf16: bool = False, tokens: int = 4096,
              seed_config: int = 4) -> Workload:
    """Fused QKV weight 2304x768; X = batch 8 x seq 512 = 4096 tokens x 768."""
    W = draw_normal(item_seed(seed_config, 0), (2304, 768), W_SIGMA)
    b = draw_normal(item_seed(seed_config, 1), (2304,), B_SIGMA)
    X = draw_normal(item_seed(seed_config, 2), (tokens, 768), X_SIGMA)
    tag = "bf16" if bf16 else "fp32"
    return Workload(f"fused_qkv_2304x768_{R}x{C}_d{int(round(density * 100))}_T{tokens}_{tag}",
                    [X], [Projection("QKV", W, b, R, C, density)], bf16=bf16)


def bert_large_zipf(R: int, C: int, k: int, density: float = 0.1, layers: int = 24,
                    tokens: int = 6144, seed_config: int = 5) -> Workload:
    """BERT-large attention: `layers` x four 1024x1024 weights, X 16 x 384 = 6144 tokens.

    `k` is the number of kept blocks of each weight, which the caller derives from `density`
    (the library's or the oracle's count; this module does no pruning arithmetic).  Per-block-row
    nonzero counts follow Zipf(1.2) (capped) with that total: blocks outside the chosen pattern
    are zeroed in W, so top-k pruning with k blocks keeps exactly that pattern (nonzero blocks
    outrank all-zero ones).  `density` only names the workload.
    """
    N = K = 1024
    Nb, Kb = N // R, K // C
    counts = zipf_counts(Nb, Kb, int(k))
    nW = 4 * layers
    projs = []
    names = ["Q", "K", "V", "O"]
    for w in range(nW):
        W = draw_normal(item_seed(seed_config, w), (N, K), W_SIGMA)
        mask = zipf_block_mask(counts, Kb, item_seed(seed_config, 3 * nW + layers + w))
        W = apply_block_mask(W, R, C, mask)
        b = draw_normal(item_seed(seed_config, nW + w), (N,), B_SIGMA)
        projs.append(Projection(f"L{w // 4}.{names[w % 4]}", W, b, R, C, density, k=k,
                                x_index=w // 4))
    X = [draw_normal(item_seed(seed_config, 2 * nW + l), (tokens, K), X_SIGMA)
         for l in range(layers)]
    return Workload(f"bert_large_{layers}x4_1024_{R}x{C}_d{int(round(density * 100))}"
                    f"_T{tokens}_zipf", X, projs, notes={"row_counts_by_rank": counts.tolist()})


def bert_base_ffn(R: int, C: int, density: float = 0.1, tokens: int = 128, bf16: bool = False,
                  seed_config: int = 6) -> Workload:
    """BERT-base feed-forward weights: W1 3072x768 (hidden -> intermediate) and W2 768x3072
    (intermediate -> hidden), batch 1 x seq `tokens`.

    W2 reads its own activation matrix (tokens x 3072), drawn like X; in a real layer it would
    be W1's output after GELU, which has the same shape and cost.
    """
    W1 = draw_normal(item_seed(seed_config, 0), (3072, 768), W_SIGMA)
    W2 = draw_normal(item_seed(seed_config, 1), (768, 3072), W_SIGMA)
    b1 = draw_normal(item_seed(seed_config, 2), (3072,), B_SIGMA)
    b2 = draw_normal(item_seed(seed_config, 3), (768,), B_SIGMA)
    X1 = draw_normal(item_seed(seed_config, 4), (tokens, 768), X_SIGMA)
    X2 = draw_normal(item_seed(seed_config, 5), (tokens, 3072), X_SIGMA)
    tag = "bf16" if bf16 else "fp32"
    return Workload(f"bert_base_ffn_3072x768_{R}x{C}_d{int(round(density * 100))}_T{tokens}_{tag}",
                    [X1, X2], [Projection("W1", W1, b1, R, C, density, x_index=0),
                               Projection("W2", W2, b2, R, C, density, x_index=1)], bf16=bf16)
