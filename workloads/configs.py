"""Named Llama-2-shaped gradient sets and their step schedules.

Shapes follow the Llama-2 family the paper fine-tunes (Evaluation, Table
"Experimental environments": Llama-2-7B and -13B; the 70B shapes extend the
same family).  A linear weight is stored PyTorch-style as [out, in]; its
columns are the input channels the paper scores (Gradient Selection,
"Lightweight Proxy for Gradient Ranking").  Hyperparameters default to the
paper's fine-tuning setup (Experimental Setup: lr 1e-5, AdamW, weight decay
0) and its ZenFlow defaults (S = 4, top-k ratio 10%, Sensitivity section).
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple


@dataclass(frozen=True)
class MatrixSpec:
    name: str
    n: int  # rows = output features
    m: int  # columns = input channels

    @property
    def params(self) -> int:
        return self.n * self.m


@dataclass(frozen=True)
class AdamHyper:
    lr: float = 1e-5
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 0.0


@dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    matrices: Tuple[MatrixSpec, ...]
    sigma: float  # log-std of the per-column lognormal scale
    ratio: float  # top-k ratio per matrix
    steps: int  # T
    refresh: int  # R: selection refresh interval
    accum: int  # S: accumulation interval
    jitter: float  # per-step multiplicative jitter of the column scales (log-std)
    spacing: str  # "all": every sorted adjacent pair; "boundary": the k/k+1 pair only
    master_std: float = 0.02
    hyper: AdamHyper = field(default_factory=AdamHyper)
    sweep_ratios: Optional[Tuple[float, ...]] = None
    sweep_refresh: Optional[Tuple[int, ...]] = None

    @property
    def params(self) -> int:
        return sum(mt.params for mt in self.matrices)

    def with_(self, **kw) -> "Workload":
        d = dict(self.__dict__)
        d.update(kw)
        return Workload(**d)


def llama_layer_shapes(hidden: int, ffn: int, kv: Optional[int] = None,
                       prefix: str = "") -> List[MatrixSpec]:
    """The seven linear weights of one Llama decoder layer, [out, in]."""
    kv = hidden if kv is None else kv
    return [
        MatrixSpec(prefix + "q_proj", hidden, hidden),
        MatrixSpec(prefix + "k_proj", kv, hidden),
        MatrixSpec(prefix + "v_proj", kv, hidden),
        MatrixSpec(prefix + "o_proj", hidden, hidden),
        MatrixSpec(prefix + "gate_proj", ffn, hidden),
        MatrixSpec(prefix + "up_proj", ffn, hidden),
        MatrixSpec(prefix + "down_proj", hidden, ffn),
    ]


def _llama_full(layers: int, hidden: int, ffn: int, vocab: int,
                kv: Optional[int] = None, embeddings: bool = True) -> Tuple[MatrixSpec, ...]:
    mats: List[MatrixSpec] = []
    if embeddings:
        mats.append(MatrixSpec("embed_tokens", vocab, hidden))
    for layer in range(layers):
        mats += llama_layer_shapes(hidden, ffn, kv, prefix=f"layers.{layer}.")
    if embeddings:
        mats.append(MatrixSpec("lm_head", vocab, hidden))
    return tuple(mats)


WORKLOADS = {
    # One 4096x4096 linear weight, one step with a fresh selection and one pack.
    "linear-4096x4096": Workload(
        name="linear-4096x4096", seed=1,
        matrices=(MatrixSpec("q_proj", 4096, 4096),),
        sigma=1.5, ratio=0.10, steps=1, refresh=1, accum=1, jitter=0.0,
        spacing="all"),
    # One Llama-2-7B decoder layer, 4 steps, selection reused, unselected accumulated.
    "llama2-7b-layer": Workload(
        name="llama2-7b-layer", seed=2,
        matrices=tuple(llama_layer_shapes(4096, 11008)),
        sigma=1.5, ratio=0.10, steps=4, refresh=4, accum=4, jitter=0.05,
        spacing="boundary"),
    # Full Llama-2-7B gradient set: embedding, 32 layers, LM head; 16 steps, R = S = 4.
    "llama2-7b-full": Workload(
        name="llama2-7b-full", seed=3,
        matrices=_llama_full(32, 4096, 11008, 32000),
        sigma=1.5, ratio=0.10, steps=16, refresh=4, accum=4, jitter=0.05,
        spacing="boundary"),
    # Llama-2-13B shapes with a sweep of ratio and refresh interval (S = 4).
    "llama2-13b-full": Workload(
        name="llama2-13b-full", seed=4,
        matrices=_llama_full(40, 5120, 13824, 32000),
        sigma=1.5, ratio=0.10, steps=16, refresh=4, accum=4, jitter=0.05,
        spacing="boundary",
        sweep_ratios=(0.01, 0.05, 0.10, 0.25), sweep_refresh=(1, 4, 16)),
    # One GPU's share of Llama-2-70B: 10 decoder layers (GQA k/v 1024x8192),
    # heavy-tailed scales, accumulation interval 8.
    "llama2-70b-10layers": Workload(
        name="llama2-70b-10layers", seed=5,
        matrices=_llama_full(10, 8192, 28672, 32000, kv=1024, embeddings=False),
        sigma=2.0, ratio=0.10, steps=16, refresh=8, accum=8, jitter=0.05,
        spacing="boundary"),
}


def get_workload(name: str) -> Workload:
    try:
        return WORKLOADS[name]
    except KeyError:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(WORKLOADS)}") from None


def shapes(mats: Sequence[MatrixSpec]) -> List[Tuple[int, int]]:
    return [(mt.n, mt.m) for mt in mats]
