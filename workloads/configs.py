"""Verify-step workload shapes.

Each shape describes one verifier level's verify step: B sequences, each with
gamma_b drafted tokens and a KV cache that already holds ctx_b context rows
plus this step's gamma_b+1 new rows (so kv_len_b = ctx_b + gamma_b + 1).
Sizes are Llama-family shaped (GQA, head_dim 64/128, vocabulary 128256); the
paper's own evaluation uses Llama-family models in bf16 (Section 5).

Value recipe shared by every shape (Section 2.2 names p as the verifier's and
q as the draft model's distribution):
  * Q, K, V ~ N(0, 1), rounded to bf16 (round-to-nearest-even);
  * verifier logits z_p ~ N(0, p_sigma^2), draft logits z_q = z_p + N(0, s^2)
    with s the per-sequence noise level;
  * draft tokens are exact samples from softmax(z_q) (Gumbel-max);
  * accept/resample uniforms are fp32 in [0, 1).
"""

from __future__ import annotations

from dataclasses import dataclass, field, replace


def _rng_pair(x):
    if isinstance(x, (tuple, list)):
        return (x[0], x[1])
    return (x, x)


@dataclass(frozen=True)
class VerifyShape:
    """One verifier level. Ranges are inclusive; (x, x) means fixed."""

    name: str
    B: int
    Hq: int
    Hkv: int
    D: int
    V: int
    gamma: tuple = (4, 4)
    ctx: tuple = (128, 128)
    noise: tuple = (1.0, 1.0)
    logits: str = "f32"  # "f32" or "bf16"
    p_sigma: float = 3.0
    seed: int = 0
    gamma_max: int | None = None
    L_cap: int | None = None
    note: str = ""

    def __post_init__(self):
        object.__setattr__(self, "gamma", _rng_pair(self.gamma))
        object.__setattr__(self, "ctx", _rng_pair(self.ctx))
        object.__setattr__(self, "noise", _rng_pair(self.noise))
        if self.Hq % self.Hkv:
            raise ValueError("Hq must be a multiple of Hkv")
        if self.logits not in ("f32", "bf16"):
            raise ValueError("logits must be 'f32' or 'bf16'")

    @property
    def gmax(self) -> int:
        return self.gamma[1] if self.gamma_max is None else self.gamma_max

    @property
    def cap(self) -> int:
        """Physical KV capacity per sequence (rounded up to 64 rows)."""
        if self.L_cap is not None:
            return self.L_cap
        need = self.ctx[1] + self.gmax + 1
        return (need + 63) // 64 * 64

    @property
    def group(self) -> int:
        return self.Hq // self.Hkv

    @property
    def ragged(self) -> bool:
        return self.gamma[0] != self.gamma[1] or self.ctx[0] != self.ctx[1] or self.noise[0] != self.noise[1]

    def with_(self, **kw) -> "VerifyShape":
        return replace(self, **kw)


@dataclass(frozen=True)
class ChainShape:
    """Three-level chain on one GPU: draft -> intermediate -> target.

    The intermediate level verifies gamma_int draft tokens; the target level
    verifies the first min(k_int + 1, gamma_tgt) tokens the intermediate
    level emitted, padded to gamma_tgt.
    """

    name: str
    B: int
    ctx: int
    V: int
    draft: tuple  # (Hq, Hkv, D)
    inter: tuple
    target: tuple
    gamma_int: int
    gamma_tgt: int
    sigma_draft_int: float
    sigma_int_tgt: float
    p_sigma: float = 3.0
    seed: int = 0
    logits: str = "f32"
    note: str = ""

    @property
    def cap(self) -> int:
        need = self.ctx + max(self.gamma_int, self.gamma_tgt) + 1
        return (need + 63) // 64 * 64


CONFIGS = {
    1: VerifyShape(
        name="tiny-single-level",
        B=1, Hq=4, Hkv=4, D=64, V=1000,
        gamma=4, ctx=128, noise=1.0, logits="f32", seed=1001,
        note="B=1, gamma=4, 4/4 heads x 64, cache 128, V=1000",
    ),
    2: VerifyShape(
        name="llama3-8b-shaped-b16",
        B=16, Hq=32, Hkv=8, D=128, V=128256,
        gamma=5, ctx=2048, noise=1.5, logits="f32", seed=1002,
        note="B=16, gamma=5, 32/8 heads x 128, cache 2048, V=128256, fp32 logits",
    ),
    3: ChainShape(
        name="three-level-chain-b32",
        B=32, ctx=4096, V=128256,
        draft=(32, 8, 64), inter=(32, 8, 128), target=(64, 8, 128),
        gamma_int=8, gamma_tgt=4,
        sigma_draft_int=2.0, sigma_int_tgt=1.0, seed=1003,
        note="1B/8B/70B-shaped chain, B=32, cache 4096, V=128256, fp32 logits",
    ),
    4: VerifyShape(
        name="long-context-70b-shaped",
        B=4, Hq=64, Hkv=8, D=128, V=128256,
        gamma=8, ctx=32768, noise=1.0, logits="f32", seed=1004,
        note="B=4, gamma=8, 64/8 heads x 128, cache 32768, V=128256, fp32 logits",
    ),
    5: VerifyShape(
        name="ragged-b256",
        B=256, Hq=32, Hkv=8, D=128, V=128256,
        gamma=(1, 8), ctx=(256, 8192), noise=(0.5, 3.0), logits="bf16", seed=1005,
        note="B=256, gamma~U{1..8}, cache~U[256,8192], 32/8 x 128, bf16 logits",
    ),
}


def get_config(i: int):
    return CONFIGS[i]


def small_shape(**kw) -> VerifyShape:
    """A shape the CPU reference finishes in well under a second."""
    base = dict(
        name="small", B=3, Hq=8, Hkv=2, D=128, V=3000,
        gamma=(0, 6), ctx=(40, 700), noise=(0.5, 2.0), logits="f32", seed=7,
    )
    base.update(kw)
    return VerifyShape(**base)
