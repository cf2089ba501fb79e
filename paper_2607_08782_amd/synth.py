"""Seeded synthetic inputs for one GPU's share of an MoE layer.

This module draws random numbers and lays out the benchmark's fixed rules
(layer shapes, popularity skew, expert-to-GPU placement).  It holds none of
the layer's arithmetic: no routing, no counting, no FFN.  Both the HIP path
and the CPU oracle receive the tensors made here.

Shapes stand in for the models the paper evaluates (Sec. VIII-B: Mixtral
8x7B, DeepSeek-V2-Lite, Qwen3-30B-A3B; Qwen1.5-MoE is cited in Sec. I).  The
paper's prompts and pretrained weights are not used: hidden states are
N(0, 1), weights N(0, 0.02^2), and a router bias skews expert popularity
towards a Zipf law, standing in for the skewed and drifting expert
selection the paper observes (Sec. III, Finding 1; Fig. 8 trace).

Every tensor is drawn from its own torch generator, seeded from
(seed, tensor name, index), so that making only the locally placed experts
gives the same values as making all of them.
"""
from __future__ import annotations

import dataclasses
import hashlib
import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

WEIGHT_STD = 0.02


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    name: str
    dtype: str                      # "f32" or "bf16": element type of X and weights
    d: int                          # hidden size
    E: int                          # routed experts
    k: int                          # experts per token
    f: int                          # routed expert FFN size
    shared_f: Tuple[int, ...] = ()  # FFN sizes of always-on shared experts
    G: int = 1                      # GPUs in the expert-parallel group
    replicas: int = 0               # hottest ranks replicated on GPU 0 and GPU G-r
    zipf: Optional[float] = None    # popularity skew exponent (None: bias 0)
    regimes: Tuple[Tuple[str, int], ...] = (("batch", 64),)
    batches: int = 1                # batches in a drift sequence
    drift_every: int = 0            # popularity re-permuted every this many batches
    coact: bool = False             # also emit the co-activation matrix

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    def T(self, regime: str) -> int:
        return dict(self.regimes)[regime]


CONFIGS: Dict[str, LayerConfig] = {
    "tiny_fp32": LayerConfig(
        name="tiny_fp32", dtype="f32", d=128, E=8, k=2, f=256, G=1,
        zipf=None, regimes=(("batch", 64),)),
    "mixtral_8x7b": LayerConfig(
        name="mixtral_8x7b", dtype="bf16", d=4096, E=8, k=2, f=14336, G=4,
        zipf=1.0, regimes=(("prefill", 4096), ("decode", 64))),
    "deepseek_v2_lite": LayerConfig(
        name="deepseek_v2_lite", dtype="bf16", d=2048, E=64, k=6, f=1408,
        shared_f=(1408, 1408), G=8, replicas=2, zipf=1.2,
        regimes=(("prefill", 8192), ("decode", 256))),
    "qwen15_moe_a27b": LayerConfig(
        name="qwen15_moe_a27b", dtype="bf16", d=2048, E=60, k=4, f=1408,
        shared_f=(5632,), G=8, zipf=1.2, regimes=(("batch", 2048),),
        batches=16, drift_every=4),
    "qwen3_30b_a3b": LayerConfig(
        name="qwen3_30b_a3b", dtype="bf16", d=2048, E=128, k=8, f=768, G=9,
        replicas=2, zipf=1.5, regimes=(("decode", 64), ("prefill", 16384)),
        coact=True),
}


def derived_seed(seed: int, name: str, index: int = 0) -> int:
    h = hashlib.blake2b(("%d/%s/%d" % (seed, name, index)).encode(), digest_size=8).digest()
    return int.from_bytes(h, "little") & ((1 << 63) - 1)


def _gen(device, seed: int, name: str, index: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(derived_seed(seed, name, index))
    return g


def normal(shape, seed: int, name: str, index: int = 0, std: float = 1.0,
           device="cpu", dtype=torch.float32) -> torch.Tensor:
    """N(0, std^2) drawn in fp32 from its own generator, then rounded to `dtype` (RNE)."""
    g = _gen(device, seed, name, index)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    return x.to(dtype)


def popularity_perm(cfg: LayerConfig, seed: int, epoch: int = 0) -> np.ndarray:
    """pi: expert pi[r-1] has popularity rank r (rank 1 = hottest)."""
    g = _gen("cpu", seed, "pi", epoch)
    return torch.randperm(cfg.E, generator=g).numpy().astype(np.int64)


def zipf_bias(cfg: LayerConfig, pi: np.ndarray) -> np.ndarray:
    """Router bias so that selection frequency roughly follows Zipf(s) over ranks.

    b[pi[r-1]] = beta * ln p_r, p_r = r^-s / sum r'^-s, beta = sigma*sqrt(6)/pi
    with sigma = WEIGHT_STD*sqrt(d), the spread of a gate score x.w for
    x ~ N(0, I), w ~ N(0, WEIGHT_STD^2 I) (a Gumbel scale of that spread).
    """
    b = np.zeros(cfg.E, np.float32)
    if cfg.zipf is None:
        return b
    ranks = np.arange(1, cfg.E + 1, dtype=np.float64)
    p = ranks ** (-cfg.zipf)
    p /= p.sum()
    sigma = WEIGHT_STD * math.sqrt(cfg.d)
    beta = sigma * math.sqrt(6.0) / math.pi
    b[pi] = (beta * np.log(p)).astype(np.float32)
    return b


def placement_map(cfg: LayerConfig, pi: np.ndarray) -> np.ndarray:
    """Benchmark placement rule (not the paper's optimizer); GPU 0 is this GPU.

    Ranks 1..R (R = cfg.replicas) are hosted twice, on GPU 0 and on GPU G-r.
    The other ranks are dealt round-robin starting at GPU 0, skipping GPUs
    that already hold C_max experts, where C_max is GPU 0's final slot count.
    Returns uint8 x[E][G] with x[e][j] = 1 iff GPU j hosts expert e.
    """
    E, G, R = cfg.E, cfg.G, cfg.replicas
    x = np.zeros((E, G), np.uint8)
    if G == 1:
        x[:, 0] = 1
        return x
    rest = E - R
    c_max = R + (rest + G - 1) // G
    load = np.zeros(G, np.int64)
    for r in range(1, R + 1):
        e = pi[r - 1]
        for j in {0, G - r}:
            x[e, j] = 1
            load[j] += 1
    j = 0
    for r in range(R + 1, E + 1):
        while load[j] >= c_max:
            j = (j + 1) % G
        x[pi[r - 1], j] = 1
        load[j] += 1
        j = (j + 1) % G
    return x


@dataclasses.dataclass
class LayerInputs:
    cfg: LayerConfig
    T: int
    X: torch.Tensor                 # [T, d]
    Wr: torch.Tensor                # [E, d]
    bias: torch.Tensor              # [E] fp32
    placement: np.ndarray           # [E, G] uint8
    dev: int
    local: List[int]                # experts hosted here, ascending id (slot order)
    w13: List[torch.Tensor]         # per local slot, [2f, d]: f gate rows, then f up rows
    w2: List[torch.Tensor]          # per local slot, [d, f]
    shared: List[Tuple[torch.Tensor, torch.Tensor]]  # (W13 [2fs, d], W2 [d, fs]) each
    pi: np.ndarray


def expert_weights(cfg: LayerConfig, e: int, seed: int, device="cpu", f: Optional[int] = None,
                   name: str = "W") -> Tuple[torch.Tensor, torch.Tensor]:
    f = cfg.f if f is None else f
    w13 = normal((2 * f, cfg.d), seed, name + "13", e, WEIGHT_STD, device, cfg.torch_dtype)
    w2 = normal((cfg.d, f), seed, name + "2", e, WEIGHT_STD, device, cfg.torch_dtype)
    return w13, w2


def make_layer(cfg: LayerConfig, T: int, seed: int = 0, device="cpu", batch: int = 0,
               dev: int = 0, experts: str = "local") -> LayerInputs:
    """All inputs of one layer share: hidden states of batch `batch`, the router,
    the Zipf bias and placement of that batch's popularity epoch, and the
    weights of the experts hosted on `dev` (experts="local"), of every expert
    ("all") or of none ("none")."""
    epoch = batch // cfg.drift_every if cfg.drift_every else 0
    pi = popularity_perm(cfg, seed, epoch)
    X = normal((T, cfg.d), seed, "X", batch, 1.0, device, cfg.torch_dtype)
    Wr = normal((cfg.E, cfg.d), seed, "Wr", 0, WEIGHT_STD, device, cfg.torch_dtype)
    bias = torch.from_numpy(zipf_bias(cfg, pi)).to(device)
    placement = placement_map(cfg, pi)
    local = [int(e) for e in np.nonzero(placement[:, dev])[0]]
    which = {"local": local, "none": [], "all": list(range(cfg.E))}[experts]
    w13, w2 = [], []
    for e in which:
        a, b = expert_weights(cfg, e, seed, device)
        w13.append(a)
        w2.append(b)
    shared = [expert_weights(cfg, u, seed, device, f=fs, name="S")
              for u, fs in enumerate(cfg.shared_f)]
    return LayerInputs(cfg, T, X, Wr, bias, placement, dev, local, w13, w2, shared, pi)


def custom_config(name="custom", dtype="bf16", d=64, E=8, k=2, f=64, shared_f=(), G=1,
                  replicas=0, zipf=None, T=32, coact=False) -> LayerConfig:
    """A small layer shape for tests."""
    return LayerConfig(name=name, dtype=dtype, d=d, E=E, k=k, f=f, shared_f=tuple(shared_f),
                       G=G, replicas=replicas, zipf=zipf, regimes=(("batch", T),), coact=coact)
