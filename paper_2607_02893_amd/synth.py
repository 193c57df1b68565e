"""Seeded synthetic inputs for the VBQ decode workloads.

This module only draws random inputs: bit-width maps, fp16 scales, integer
levels and fp16 activations.  It contains none of the method's arithmetic and
is the one module that both the oracle-based tests and the GPU path consume.

Recipe (stand-ins for trained weights; the paper's models and datasets are not
used):
  * every matrix has its own generator, PCG64(SeedSequence(cfg_seed,
    spawn_key=(layer, proj))), so any matrix can be regenerated alone;
  * draw order inside a matrix: bit map, then scales, then levels;
  * bit map: iid per 64-weight group from a width distribution, e.g. the
    mix {1: .69, 2: .15, 4: .12, 8: .04} (mean 1.79 bits) of the adaptive
    pilot (paper section 5.1), or per-row widths for a tiered head;
  * scales: U(0.01, 0.1) rounded to fp16;
  * levels: uniform over the level set of the group's width,
    {-(2^(b-1)-1) .. 2^(b-1)-1} for b >= 2 and {-1, +1} for b = 1;
  * activations: N(0, 1) rounded to fp16, from key (layer, proj, 1000 + m).

Selection path (paper section 3.2, training time): flat fp32 weights whose
64-weight groups are N(0, sigma_g^2) with sigma_g log-uniform in
[1e-3, 0.1] (groups of very different magnitude, as across a network's
layers), logits N(0, 1.5^2) per (group, candidate) and standard Gumbel noise
-log(-log U) per (group, candidate), drawn in that order from key
(3000, part).  The training-step workload is the flat concatenation of the
131M-class model's linear weights (workload 1's matrices, 137.8M weights).

Recipe variant (paper section 4, the fixed recipe that is deployed): the
first block's MLP (gate, up, down) at 4 bits, every other projection at
2 bits, and the LM head tiered per row by token-frequency rank -- top 0.5% of
rows at 8 bits, the next 1.5% at 4, the next 10% at 2, the rest at 1 (mean
1.18 bits).  No corpus is available, so a row's rank is a seeded random
permutation of the vocabulary (key (layer, proj, 2000)).
"""

from dataclasses import dataclass, field

import numpy as np

G = 64
MIX_PILOT = {1: 0.69, 2: 0.15, 4: 0.12, 8: 0.04}       # mean 1.79 bits
MIX_FIRST_MLP = {1: 0.30, 2: 0.50, 4: 0.10, 8: 0.10}   # mean 2.50 bits
# recipe head: (fraction of rows by frequency rank, bits), most frequent first
RECIPE_HEAD_TIERS = ((0.005, 8), (0.015, 4), (0.10, 2), (0.88, 1))
WIDTHS = (1, 2, 4, 8)


def rng_for(seed, *key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=tuple(key))))


def draw_bits(rng, N, Gc, mix):
    """iid widths per group: uint8[N, Gc]."""
    widths = np.array(sorted(mix), dtype=np.uint8)
    p = np.array([mix[int(b)] for b in widths], dtype=np.float64)
    cdf = np.cumsum(p / p.sum())
    u = rng.random((N, Gc))
    idx = np.searchsorted(cdf, u, side="right")
    return widths[np.minimum(idx, len(widths) - 1)]


def draw_row_bits(rng, N, Gc, row_mix):
    """One width per row (all groups of the row share it): uint8[N, Gc]."""
    return np.repeat(draw_bits(rng, N, 1, row_mix), Gc, axis=1)


def draw_scales(rng, N, Gc, lo=0.01, hi=0.1):
    """fp16 bit patterns of U(lo, hi): uint16[N, Gc]."""
    return rng.uniform(lo, hi, size=(N, Gc)).astype(np.float16).view(np.uint16)


def draw_levels(rng, bits):
    """Levels uniform over each group's level set: int8[N, 64*Gc]."""
    N, Gc = bits.shape
    q = np.zeros((N, Gc, G), dtype=np.int8)
    for b in WIDTHS:
        sel = bits == b
        n = int(np.count_nonzero(sel))
        if n == 0:
            continue
        if b == 1:
            q[sel] = (rng.integers(0, 2, size=(n, G), dtype=np.int8) * 2 - 1).astype(np.int8)
        else:
            m = (1 << (b - 1)) - 1
            q[sel] = rng.integers(-m, m + 1, size=(n, G), dtype=np.int16).astype(np.int8)
    return q.reshape(N, Gc * G)


def draw_x(rng, M, K):
    """fp16 activations N(0, 1): float16[M, K]."""
    return rng.standard_normal((M, K)).astype(np.float16)


def draw_weights(rng, N, K, std=0.02):
    """Dense float32 weights for exercising the quantizer: float32[N, K]."""
    return (rng.standard_normal((N, K)) * std).astype(np.float32)


@dataclass
class MatrixSpec:
    """One packed matrix of a decode step (rows N, columns K)."""
    name: str
    layer: int
    proj: int
    N: int
    K: int
    mix: dict = field(default_factory=lambda: dict(MIX_PILOT))
    row_mix: dict = None          # per-row widths on a random subset of rows
    row_mix_rows: float = 0.0     # fraction of rows that take row_mix
    uniform_bits: int = 0         # 1/2/4/8: every group has this width
    row_tiers: tuple = None       # ((fraction, bits), ...): per-row widths by frequency rank

    @property
    def groups(self):
        return self.N * (self.K // G)


@dataclass
class Workload:
    name: str
    seed: int
    matrices: list
    batch: tuple = (1,)


def _decoder(name, seed, d, layers, mlp, vocab, kv=None, first_mlp_mix=None,
             head=None, uniform_bits=0, recipe=False):
    """Decode-step matrices in call order.  Projections that read the same
    input are stored as one row-concatenated matrix: Q|K|V and gate|up.
    recipe: the deployed recipe's widths (module docstring)."""
    kv = d if kv is None else kv
    mats = []
    for layer in range(layers):
        mlp_mix = first_mlp_mix if (layer == 0 and first_mlp_mix) else MIX_PILOT
        attn_u = 2 if recipe else uniform_bits
        mlp_u = (4 if layer == 0 else 2) if recipe else uniform_bits
        mats.append(MatrixSpec("qkv", layer, 0, d + 2 * kv, d, uniform_bits=attn_u))
        mats.append(MatrixSpec("o", layer, 1, d, d, uniform_bits=attn_u))
        mats.append(MatrixSpec("gate_up", layer, 2, 2 * mlp, d, mix=dict(mlp_mix), uniform_bits=mlp_u))
        mats.append(MatrixSpec("down", layer, 3, d, mlp, mix=dict(mlp_mix), uniform_bits=mlp_u))
    hs = MatrixSpec("head", layers, 4, vocab, d, uniform_bits=0 if recipe else uniform_bits)
    if recipe:
        hs.row_tiers = RECIPE_HEAD_TIERS
    elif head is not None:
        for k, v in head.items():
            setattr(hs, k, v)
    mats.append(hs)
    return Workload(name, seed, mats)


def workload(cfg, uniform_bits=0, recipe=False):
    """The five synthetic decode workloads, by index.

    0: one 512x512 GEMV, mix of the adaptive pilot.
    1: 131M-class step: d=768, 12 layers, MLP 3072, head 32000x768 whose rows
       are 1-bit except a random 10% of rows at 2 bits.
    2: 1.0B-class step: d=2048, 24 layers, MLP 8192, vocab 50304; the first MLP
       block draws widths with mean 2.5 bits.
    3: 9B-class step: d=4096, 32 layers, GQA K/V 1024x4096, MLP 14336,
       vocab 128256.
    4: 1.46B-class shapes: d=2048, 32 layers, MLP 8192, vocab 50304,
       batch M in {1,2,4,8,16}; uniform_bits selects the uniform variants.
    recipe=True (workloads 2, 3, 4): the same shapes with the deployed
    recipe's widths instead of the per-group mixes.
    """
    if recipe:
        if cfg not in (2, 3, 4):
            raise ValueError("the recipe variant exists for the decoder workloads 2, 3 and 4")
        shapes = {2: ("1.0B-class", 2048, 24, 8192, 50304, None), 3: ("9B-class", 4096, 32, 14336, 128256, 1024),
                  4: ("1.46B-class", 2048, 32, 8192, 50304, None)}[cfg]
        name, d, layers, mlp, vocab, kv = shapes
        return _decoder(name + "-recipe", 20260750 + cfg, d, layers, mlp, vocab, kv=kv, recipe=True)
    if cfg == 0:
        return Workload("gemv-512x512", 20260700, [MatrixSpec("w", 0, 0, 512, 512)])
    if cfg == 1:
        return _decoder("131M-class", 20260701, 768, 12, 3072, 32000,
                        head={"mix": {1: 1.0}, "row_mix": {2: 1.0}, "row_mix_rows": 0.10})
    if cfg == 2:
        return _decoder("1.0B-class", 20260702, 2048, 24, 8192, 50304,
                        first_mlp_mix=MIX_FIRST_MLP)
    if cfg == 3:
        return _decoder("9B-class", 20260703, 4096, 32, 14336, 128256, kv=1024)
    if cfg == 4:
        w = _decoder("1.46B-class" + (f"-u{uniform_bits}" if uniform_bits else ""),
                     20260704 + 10 * uniform_bits, 2048, 32, 8192, 50304,
                     uniform_bits=uniform_bits)
        w.batch = (1, 2, 4, 8, 16)
        return w
    raise ValueError(f"no workload {cfg}")


def tier_widths(N, tiers, rng):
    """Per-row widths uint8[N] for frequency tiers ((fraction, bits), ...):
    rows are ranked by a random permutation (rank 0 = most frequent) and the
    tiers take consecutive rank ranges, the last one the remainder."""
    rank_to_row = rng.permutation(N)
    w = np.empty(N, dtype=np.uint8)
    lo = 0
    for i, (frac, b) in enumerate(tiers):
        hi = N if i == len(tiers) - 1 else min(N, lo + int(round(frac * N)))
        w[rank_to_row[lo:hi]] = b
        lo = hi
    return w


def make_bits(spec, seed):
    rng = rng_for(seed, spec.layer, spec.proj)
    Gc = spec.K // G
    if spec.row_tiers is not None:
        w = tier_widths(spec.N, spec.row_tiers, rng_for(seed, spec.layer, spec.proj, 2000))
        bits = np.repeat(w[:, None], Gc, axis=1)
    elif spec.uniform_bits:
        bits = np.full((spec.N, Gc), spec.uniform_bits, dtype=np.uint8)
    else:
        bits = draw_bits(rng, spec.N, Gc, spec.mix)
    if spec.row_mix is not None and spec.row_mix_rows > 0:
        n_rows = int(round(spec.row_mix_rows * spec.N))
        rows = np.sort(rng.choice(spec.N, size=n_rows, replace=False))
        bits[rows] = draw_row_bits(rng, n_rows, Gc, spec.row_mix)
    return bits, rng


def make_matrix(spec, seed):
    """(bits uint8[N,G], q int8[N,K], scales uint16[N,G]) for one matrix."""
    bits, rng = make_bits(spec, seed)
    s = draw_scales(rng, spec.N, spec.K // G)
    q = draw_levels(rng, bits)
    return bits, q, s


def make_x(spec, seed, M=1):
    return draw_x(rng_for(seed, spec.layer, spec.proj, 1000), M, spec.K)


# ---------------------------------------------------- differentiable bit selection

SELECTION_SEED = 20260760


def draw_selection_inputs(rng, n_groups, sigma_lo=1e-3, sigma_hi=0.1, logit_std=1.5):
    """(W float32[n_groups*64], logits float32[n_groups, 4], noise float32[n_groups, 4])."""
    sigma = np.exp(rng.uniform(np.log(sigma_lo), np.log(sigma_hi), size=n_groups)).astype(np.float32)
    W = rng.standard_normal((n_groups, G), dtype=np.float32) * sigma[:, None]
    logits = rng.standard_normal((n_groups, 4), dtype=np.float32) * np.float32(logit_std)
    noise = rng.gumbel(size=(n_groups, 4)).astype(np.float32)
    return W.reshape(-1), logits, noise


def selection_inputs(n_groups, part=0, seed=SELECTION_SEED):
    return draw_selection_inputs(rng_for(seed, 3000, part), n_groups)


def selection_workload(cfg=1):
    """(name, [(matrix name, N, K)], total groups) of a model's linear weights
    laid end to end, the unit of one training step of the selection path."""
    w = workload(cfg)
    mats = [(f"{m.name}{m.layer}", m.N, m.K) for m in w.matrices]
    return w.name, mats, sum(N * K // G for _, N, K in mats)
