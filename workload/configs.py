"""Model shapes and workloads (plain data).

The drafting/verification round of the paper (Sec. 3, Sec. 4.2) is exercised
on randomly initialised Qwen3-shaped models.  The drafter has five layers and a
block size of 16 (Sec. 5.1, training and implementation details); the target
feature layers are a fixed set sampled from shallow to deep (Sec. 3, eq.
dflash_context), taken here as evenly spaced decoder-layer outputs.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Tuple


def evenly_spaced_layers(n_layers: int, m: int) -> Tuple[int, ...]:
    """0-based decoder-layer indices floor(i*(L-1)/(m-1)), i = 0..m-1."""
    if m == 1:
        return (n_layers - 1,)
    return tuple((i * (n_layers - 1)) // (m - 1) for i in range(m))


@dataclass(frozen=True)
class ModelDims:
    dtype: str                 # "f32" or "bf16": storage type of weights/activations
    d: int                     # hidden size
    n_layers: int              # target decoder layers L
    n_heads: int               # query heads Hq
    n_kv_heads: int            # key/value heads Hkv
    head_dim: int              # Dh
    ffn: int                   # SwiGLU intermediate size
    vocab: int                 # V
    n_draft_layers: int        # drafter layers Ld
    capture_layers: Tuple[int, ...]   # target layers whose outputs feed W_c
    relay_hidden: int = 0      # MLP_phi hidden width (0 -> d)
    rope_theta: float = 1.0e6
    rms_eps: float = 1.0e-6
    ln_eps: float = 1.0e-5

    @property
    def m(self) -> int:
        return len(self.capture_layers)

    @property
    def d_h(self) -> int:
        return self.relay_hidden or self.d

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim


@dataclass(frozen=True)
class Workload:
    name: str
    dims: ModelDims
    block: int                 # B = anchor + K drafted tokens
    batch: int                 # b sequences
    ctx: Tuple[int, int]       # prompt length range [lo, hi] (lo == hi: fixed)
    rounds: int
    schedule: str              # "bernoulli" or "geometric"
    sched_param: float         # forcing probability, or geometric mean mu
    carry_window: str = "suffix"
    seed_w: int = 1234
    seed_prompt: int = 1235
    seed_sched: int = 1236
    description: str = ""

    @property
    def K(self) -> int:
        return self.block - 1

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


_QWEN3_1P7B = ModelDims("bf16", 2048, 28, 16, 8, 128, 6144, 151936, 5, evenly_spaced_layers(28, 5))
_QWEN3_8B = ModelDims("bf16", 4096, 36, 32, 8, 128, 12288, 151936, 5, evenly_spaced_layers(36, 5))
_QWEN3_32B = ModelDims("bf16", 5120, 64, 64, 8, 128, 25600, 151936, 5, evenly_spaced_layers(64, 5))
_TINY_F32 = ModelDims("f32", 256, 2, 4, 2, 64, 768, 4096, 1, (0, 1))

CONFIGS = {
    # tiny fp32 reference workload, fully checked against the oracle
    "tiny-f32": Workload("tiny-f32", _TINY_F32, block=8, batch=1, ctx=(128, 128), rounds=6,
                         schedule="bernoulli", sched_param=0.7,
                         description="2-layer d=256 fp32 target, 1-layer drafter, ctx 128, B=8"),
    "qwen3-1.7b": Workload("qwen3-1.7b", _QWEN3_1P7B, block=16, batch=1, ctx=(1024, 1024), rounds=64,
                           schedule="geometric", sched_param=5.0,
                           description="Qwen3-1.7B shape bf16, ctx 1024, B=16, b=1"),
    "qwen3-8b": Workload("qwen3-8b", _QWEN3_8B, block=16, batch=1, ctx=(4096, 4096), rounds=128,
                         schedule="geometric", sched_param=6.0,
                         description="Qwen3-8B shape bf16, ctx 4096, B=16, b=1"),
    "qwen3-8b-b8": Workload("qwen3-8b-b8", _QWEN3_8B, block=16, batch=8, ctx=(2048, 8192), rounds=128,
                            schedule="geometric", sched_param=6.0,
                            description="Qwen3-8B shape bf16, b=8 ragged ctx in [2048, 8192], B=16"),
    "qwen3-8b-b32": Workload("qwen3-8b-b32", _QWEN3_8B, block=16, batch=32, ctx=(1024, 2048), rounds=64,
                             schedule="geometric", sched_param=6.0,
                             description="Qwen3-8B shape bf16, b=32 ragged ctx in [1024, 2048], B=16: 512 rows per round"),
    "qwen3-32b": Workload("qwen3-32b", _QWEN3_32B, block=16, batch=4, ctx=(16384, 16384), rounds=64,
                          schedule="geometric", sched_param=6.0,
                          description="Qwen3-32B shape bf16, b=4, ctx 16384, B=16"),
    # Small parity workloads: several GEMM tiles with ragged tails (N not a
    # multiple of the 64-column group, vocab 5008), real head_dim 128, GQA 4,
    # three sequences with ragged contexts spanning several attention chunks.
    "small-bf16": Workload("small-bf16",
                           ModelDims("bf16", 512, 3, 8, 2, 128, 1376, 5008, 2, (0, 1, 2)),
                           block=16, batch=3, ctx=(40, 520), rounds=6,
                           schedule="geometric", sched_param=4.0,
                           description="3-layer d=512 bf16, V=5008, b=3 ragged ctx, B=16"),
    # more rows than the weight-streaming GEMM takes (M = b * B > 128): the
    # tiled GEMM path, checked against the oracle (fp32) and by batch
    # invariance against the same sequences run alone (bf16)
    "tiny-f32-b20": Workload("tiny-f32-b20", _TINY_F32, block=8, batch=20, ctx=(30, 200), rounds=4,
                             schedule="bernoulli", sched_param=0.7,
                             description="tiny fp32 model, b=20 ragged ctx, B=8: 160 rows per round"),
    "small-bf16-b24": Workload("small-bf16-b24",
                               ModelDims("bf16", 512, 3, 8, 2, 128, 1376, 5008, 2, (0, 1, 2)),
                               block=16, batch=24, ctx=(40, 520), rounds=4,
                               schedule="geometric", sched_param=4.0,
                               description="small bf16 model, b=24 ragged ctx, B=16: 384 rows per round"),
    "small-f32": Workload("small-f32",
                          ModelDims("f32", 512, 3, 8, 2, 128, 1376, 5008, 2, (0, 1, 2)),
                          block=16, batch=3, ctx=(40, 520), rounds=6,
                          schedule="geometric", sched_param=4.0,
                          description="fp32 twin of small-bf16"),
}


def get_config(name: str) -> Workload:
    try:
        return CONFIGS[name]
    except KeyError:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(CONFIGS)}") from None
