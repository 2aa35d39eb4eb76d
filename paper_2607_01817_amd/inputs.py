"""Seeded synthetic workloads shared by the tests, the smoke check and the bench.

This module draws inputs only.  It holds none of the method's arithmetic, and it
imports neither the HIP binding nor the oracle, so both sides can be fed the
same host tensors.

The paper's workload is Wan2.2 latent-video self-attention: 40 heads of
dimension 128 and 60 x 104 latents, i.e. 6240 tokens per latent frame
(Sec. 4.1, model configuration table).  A Ulysses rank with P shards holds
H = 40 / P heads over the whole sequence.  The paper gives no distribution
for the activations, so Q, K and V are i.i.d. Gaussians of the stated scale.
The "planted peak" variant sets each query to twice a chosen key, giving a
softmax dominated by that key.  It stands in for peaked real attention maps
and makes the parity tolerance meaningful.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    S: int
    H: int
    d: int
    dtype: str            # "bf16" or "fp32" storage
    sigma: float          # Q, K, V ~ N(0, 1) * sigma
    P: int                # sequence shards of the Ulysses layout
    chunkings: tuple      # tuple of tuples of head counts
    seed: int
    oracle_rows: int      # query rows per head checked against the oracle (0 = all)

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)

    @property
    def flops(self) -> float:
        """Algorithmic attention FLOPs: two GEMMs of S x S x d per head."""
        return 4.0 * self.S * self.S * self.H * self.d

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4


WORKLOADS = {
    "tiny": Workload("tiny", 512, 4, 64, "fp32", 1.0, 4, ((2, 2), (4,)), 1, 0),
    "small": Workload("small", 4096, 8, 128, "bf16", 1.0, 8,
                      ((8,), (4, 4), (2, 2, 2, 2), (3, 3, 2)), 2, 0),
    # Wan2.2-14B shape, rank share at P=4: 21 latent frames x 1560 tokens.
    "wan_p4": Workload("wan_p4", 32760, 10, 128, "bf16", 0.5, 4,
                       ((10,), (5, 5), (4, 3, 3)), 3, 256),
    # Wan2.2-14B shape, rank share at P=8: 36 latent frames x 1560 tokens.
    "wan_p8": Workload("wan_p8", 56160, 5, 128, "bf16", 0.5, 8,
                       ((5,), (2, 2, 1), (1, 1, 1, 1, 1)), 4, 256),
    # All 40 heads of one layer on one GPU, 100k tokens.
    "stress": Workload("stress", 100000, 40, 128, "bf16", 0.5, 8,
                       ((40,), (10, 10, 10, 10), (14, 13, 13)), 5, 128),
}


def torch_dtype(w: Workload):
    return torch.bfloat16 if w.dtype == "bf16" else torch.float32


def make_qkv(w: Workload, planted: bool = False, seed: int | None = None):
    """Q, K, V as host tensors of shape [S][H][d] (= [P][S/P][H][d]).

    Drawn as fp32 ``randn`` in the order Q, K, V from a CPU generator seeded
    with ``seed`` (default ``w.seed``), multiplied by ``sigma`` and rounded to
    the storage dtype (round-to-nearest-even for bf16).

    With ``planted=True``, K is drawn with unit scale and each query row of
    head h is replaced by ``2 * K[π_h(i)]`` for a seeded permutation π_h of the
    keys (the doubling is exact in bf16).  With scale 1/sqrt(d) the planted
    logit is then about 2*sqrt(d) (22.6 at d = 128) while the other logits
    have standard deviation 2, so the softmax puts nearly all of its weight on
    one key and |O| is of the order of |V|.
    """
    seed = w.seed if seed is None else seed
    g = torch.Generator(device="cpu").manual_seed(seed)
    dt = torch_dtype(w)
    shape = (w.S, w.H, w.d)
    k_sigma = 1.0 if planted else w.sigma
    q = (torch.randn(shape, generator=g, dtype=torch.float32) * w.sigma).to(dt)
    k = (torch.randn(shape, generator=g, dtype=torch.float32) * k_sigma).to(dt)
    v = (torch.randn(shape, generator=g, dtype=torch.float32) * w.sigma).to(dt)
    if planted:
        q = torch.empty_like(k)
        for h in range(w.H):
            perm = torch.from_numpy(planted_permutation(w, h, seed))
            q[:, h, :] = k[perm, h, :] * 2
    return q, k, v


def make_dout(w: Workload, seed: int | None = None):
    """The output gradient dL/dO of a training step as a host tensor [S][H][d]:
    fp32 ``randn`` from a CPU generator seeded with ``seed + 2000`` (default
    ``w.seed + 2000``), unit scale, rounded to the storage dtype."""
    seed = (w.seed if seed is None else seed) + 2000
    g = torch.Generator(device="cpu").manual_seed(seed)
    return torch.randn((w.S, w.H, w.d), generator=g, dtype=torch.float32).to(torch_dtype(w))


def planted_permutation(w: Workload, h: int, seed: int | None = None) -> np.ndarray:
    """The key index each query of head ``h`` is planted on (a permutation)."""
    seed = w.seed if seed is None else seed
    return np.random.default_rng(seed * 7919 + h).permutation(w.S)


def sample_rows(w: Workload, n: int | None = None, seed: int | None = None):
    """Sorted query indices per head for oracle checks on the large shapes."""
    n = w.oracle_rows if n is None else n
    seed = w.seed if seed is None else seed
    if n == 0 or n >= w.S:
        return [np.arange(w.S, dtype=np.int64) for _ in range(w.H)]
    rng = np.random.default_rng(seed + 1000)
    return [np.sort(rng.choice(w.S, size=n, replace=False)).astype(np.int64)
            for _ in range(w.H)]



# ---------------------------------------------------------------------------
# Layer workloads: the attention layer around the chunk loop
# ---------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class LayerWorkload:
    """One GPU's share of an attention layer: S tokens of width D, H local
    heads of dimension d (the QKV projection produces 3 H d features per
    token, the output projection maps the H d concatenated head features
    back to D), the tokens laid on a latent grid for the rotary embedding,
    whose d/2 pairs split into the groups ``axis_pairs`` (one per axis)."""
    name: str
    grid: tuple
    axis_pairs: tuple
    H: int
    d: int
    D: int
    dtype: str
    P: int
    chunkings: tuple
    seed: int
    oracle_rows: int      # token rows checked against the oracle (0 = all)
    base: float = 10000.0

    @property
    def S(self) -> int:
        return int(np.prod(self.grid))

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)

    @property
    def flops(self) -> dict:
        """Algorithmic FLOPs of the three steps (2 per multiply-add)."""
        S, H, d, D = self.S, self.H, self.d, self.D
        return {"qkv_projection": 2.0 * S * D * 3 * H * d,
                "attention": 4.0 * S * S * H * d,
                "output_projection": 2.0 * S * H * d * D}


LAYERS = {
    # Small enough for the whole layer in the oracle.
    "layer_small": LayerWorkload("layer_small", (4, 6, 10), (12, 10, 10), 4, 64, 256, "bf16", 4,
                                 ((4,), (2, 2), (3, 1)), 11, 0),
    # Odd grid, tails in every dimension of the tiles.
    "layer_ragged": LayerWorkload("layer_ragged", (3, 7, 13), (22, 21, 21), 3, 128, 192, "bf16",
                                  3, ((3,), (2, 1)), 12, 0),
    # fp32 storage.
    "layer_fp32": LayerWorkload("layer_fp32", (2, 8, 16), (12, 10, 10), 2, 64, 128, "fp32", 2,
                                ((2,), (1, 1)), 13, 0),
    # Wan2.2-14B-shaped rank share at P = 8: 36 latent frames of 30 x 52 patch
    # tokens (1560 per frame), 5 of the 40 heads, model width 5120.
    "layer_wan_p8": LayerWorkload("layer_wan_p8", (36, 30, 52), (22, 21, 21), 5, 128, 5120,
                                  "bf16", 8, ((5,), (2, 2, 1)), 14, 32),
}


def make_layer(w: LayerWorkload, seed: int | None = None):
    """Host tensors of a layer: x [S][D] ~ N(0, 1), the QKV weight [3 H d][D]
    and the output weight [D][H d], each ~ N(0, 1) divided by the square root
    of its input width (so every projected feature has unit variance), all
    stored [out][in], drawn in that order as fp32 ``randn`` from a CPU
    generator seeded with ``seed`` (default ``w.seed``) and rounded to the
    storage dtype."""
    seed = w.seed if seed is None else seed
    g = torch.Generator(device="cpu").manual_seed(seed)
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    S, H, d, D = w.S, w.H, w.d, w.D
    x = torch.randn((S, D), generator=g, dtype=torch.float32).to(dt)
    w_qkv = (torch.randn((3 * H * d, D), generator=g, dtype=torch.float32) / math.sqrt(D)).to(dt)
    w_o = (torch.randn((D, H * d), generator=g, dtype=torch.float32) / math.sqrt(H * d)).to(dt)
    return x, w_qkv, w_o


def sample_tokens(w: LayerWorkload, n: int | None = None, seed: int | None = None) -> np.ndarray:
    """Sorted token rows for oracle checks of a layer (all when n is 0)."""
    n = w.oracle_rows if n is None else n
    seed = w.seed if seed is None else seed
    if n == 0 or n >= w.S:
        return np.arange(w.S, dtype=np.int64)
    rng = np.random.default_rng(seed + 1000)
    return np.sort(rng.choice(w.S, size=n, replace=False)).astype(np.int64)
