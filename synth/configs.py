"""The five workload shapes (sizes, dtypes, temperatures, distributions).

C1  tiny, CPU-checkable: B=1 T=16 N=4 L=3, shared V=1000, fp32,
    X ~ N(0, 2^2), Y = X + N(0, 1).
C2  Vicuna-7B-shaped: B=4 T=256 N=4 L=5, V=32000 bf16,
    Y ~ N(0, 3^2), X = 0.8 Y + N(0, 1.5^2).
C3  LLaMA-3-8B / EAGLE-3-shaped: B=4 T=512 N=8 L=6, target V=128256,
    draft V=32000 with a seeded injective sorted draft->target map,
    Y ~ N(0, 3^2), X = 0.7 Y[map] + sqrt(0.51)*3*eps (correlation 0.7).
C4  low-entropy and ragged: B=8 T=256 N=8 L=8, V=32000 bf16, target rows scaled
    so their top-1 probability is ~U(0.85, 0.99), X = 0.8 Y + N(0, 1.5^2),
    T_q = 0.5, per-path valid depth ~U{1..8}.
C5  fused LM head: B=2 T=512 N=8 L=6, hidden 4096, hidden states N(0,1) bf16,
    LM-head weights N(0, 0.02^2) bf16, target V=128256, draft V=32000 + map.
"""
from dataclasses import dataclass, replace


@dataclass(frozen=True)
class Config:
    name: str
    B: int
    T: int
    N: int
    L: int
    v_draft: int
    v_target: int
    dtype: str            # "f32" or "bf16"
    kind: str             # generator recipe
    temp_draft: float = 1.0
    temp_target: float = 1.0
    mapped: bool = False
    ragged: bool = False
    hidden: int = 0
    w_std: float = 0.02   # fused recipe: LM-head weight standard deviation
    seed: int = 0         # generator seed (inputs)
    philox_seed: int = 0  # sampler seed
    philox_offset: int = 0

    @property
    def P(self):
        return self.B * self.T

    @property
    def R(self):
        return self.B * self.T * self.N * self.L

    @property
    def elem_bytes(self):
        return 4 if self.dtype == "f32" else 2

    def ld(self, v):
        """Row stride in elements: v rounded up to a 16-byte multiple."""
        per16 = 16 // self.elem_bytes
        return (v + per16 - 1) // per16 * per16


CONFIGS = {
    "C1": Config("C1", 1, 16, 4, 3, 1000, 1000, "f32", "gauss_shared", seed=0),
    "C2": Config("C2", 4, 256, 4, 5, 32000, 32000, "bf16", "gauss_corr", seed=2),
    "C3": Config("C3", 4, 512, 8, 6, 32000, 128256, "bf16", "mapped_corr", mapped=True, seed=3),
    "C4": Config("C4", 8, 256, 8, 8, 32000, 32000, "bf16", "peaked_ragged",
                 temp_draft=0.5, ragged=True, seed=4),
    "C5": Config("C5", 2, 512, 8, 6, 32000, 128256, "bf16", "fused", mapped=True,
                 hidden=4096, seed=5),
}


def get_config(name):
    return CONFIGS[name]


def scaled(base_name, **overrides):
    """A config of the same recipe with some fields replaced (smaller B, T ...).

    For the fused recipe a smaller hidden size keeps the logit spread of the
    full shape (std 0.02 * sqrt(4096) = 1.28) unless w_std is given."""
    base = CONFIGS[base_name]
    overrides.setdefault("name", base.name + "-scaled")
    if base.kind == "fused" and "hidden" in overrides and "w_std" not in overrides:
        overrides["w_std"] = base.w_std * (base.hidden / overrides["hidden"]) ** 0.5
    return replace(base, **overrides)
