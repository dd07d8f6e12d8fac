"""Workload presets: model shapes, draft length, batch, prompt and sampling settings.

The five presets are the synthetic random-weight workloads this library is
measured and tested on.  Shapes follow the paper's SwiGLU decoder pairs (the
paper evaluates Vicuna/Qwen3/Llama verifier-drafter pairs, Section "Model
Configurations"); unspecified details (RMSNorm epsilon, RoPE base, untied LM
head, no biases) are fixed here.  Nothing in this module computes anything.
"""
from dataclasses import dataclass, field, replace
from typing import Optional, Tuple


@dataclass(frozen=True)
class Dims:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    d_ff: int
    vocab: int
    rope_theta: float = 1e4
    rms_eps: float = 1e-5

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads


@dataclass(frozen=True)
class Workload:
    name: str
    verifier: Dims
    drafter: Dims
    dtype: str              # "f32" or "bf16": storage type of every weight
    k: int                  # draft length per round
    batch: int
    prompt: Tuple[int, int]  # (lo, hi) prompt length range; lo == hi for fixed length
    new_tokens: int
    temperature: float     # 0 means greedy
    seed: int = 0

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)

    @property
    def max_prompt(self) -> int:
        return self.prompt[1]

    @property
    def max_seq_len(self) -> int:
        # committed prefix + generated tokens + one block of k+1 in flight
        return self.max_prompt + self.new_tokens + self.k + 1


TINY = Workload(
    name="tiny-f32",
    verifier=Dims(4, 256, 8, 8, 1024, 1024, 1e4),
    drafter=Dims(2, 128, 4, 4, 512, 1024, 1e4),
    dtype="f32", k=4, batch=1, prompt=(32, 32), new_tokens=32, temperature=1.0)

SMALL = Workload(
    name="small-bf16-greedy",
    verifier=Dims(12, 768, 12, 12, 3072, 32000, 1e4),
    drafter=Dims(4, 512, 8, 8, 2048, 32000, 1e4),
    dtype="bf16", k=5, batch=1, prompt=(128, 128), new_tokens=128, temperature=0.0)

_V8B = Dims(32, 4096, 32, 8, 14336, 128256, 5e5)
_D1B = Dims(16, 2048, 32, 8, 8192, 128256, 5e5)

LLAMA8B = Workload(
    name="8b-bf16-b1",
    verifier=_V8B, drafter=_D1B,
    dtype="bf16", k=5, batch=1, prompt=(512, 512), new_tokens=256, temperature=1.0)

LLAMA8B_BATCHED = Workload(
    name="8b-bf16-b16-ragged",
    verifier=_V8B, drafter=_D1B,
    dtype="bf16", k=7, batch=16, prompt=(256, 2048), new_tokens=256, temperature=0.7)

LLAMA70B = Workload(
    name="70b-bf16-b4",
    verifier=Dims(80, 8192, 64, 8, 28672, 128256, 5e5), drafter=_D1B,
    dtype="bf16", k=8, batch=4, prompt=(1024, 1024), new_tokens=256, temperature=1.0)

PRESETS = [TINY, SMALL, LLAMA8B, LLAMA8B_BATCHED, LLAMA70B]
BY_NAME = {w.name: w for w in PRESETS}
