"""Shapes of the synthetic workloads.

The paper evaluates LLaDA-8B-Instruct, Dream-v0-Instruct-7B and
DiffuCoder-7B with batch 1 and a 256-token response block (Sec. 6 and
App. G.4, implementation details); its prompt-length study sweeps prompts of
128..2048 tokens at a 256-token response (App. E, table of per-update cost).
No trained weights or benchmark prompts are used here: every workload is a
random-init model of the named architecture fed seeded uniform-random prompt
tokens, which stand in for the paper's code / math prompts.

Readings where the paper is silent (model details are not given; the
backbones are only named): RoPE is rotate-half with theta = 10000, RMSNorm
epsilon is 1e-5, RMSNorm gains are 1, the LM head is untied, and the MASK
token is the last vocabulary id.
"""

from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field


@dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    dtype: str = "bf16"          # "bf16" or "fp32": storage + GEMM operand type
    rms_eps: float = 1e-5
    rope_theta: float = 10000.0
    init_std: float = 0.02
    # bf16 models: projections whose activation operand is a single bf16 value
    # (names from "qkv", "o", "gateup", "down", "head"); the others take the
    # two-term (about 16-bit) activation
    single_term: tuple = ()
    # bf16 models: the gate/up projection multiplies single fp16 operands (its
    # input and w_gate, w_up rounded to fp16) instead of the two-term pair
    gateup_fp16: bool = False

    @property
    def mask_id(self) -> int:
        return self.vocab - 1

    @property
    def qkv_dim(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim


@dataclass(frozen=True)
class DecodeShape:
    batch: int
    prompt_len: int              # fixed prompt length (ignored when ragged)
    resp_len: int                # G
    steps: int                   # T denoising steps (= number of decisions)
    unmask_per_step: int         # k
    remask_threshold: float      # tau
    refresh_every: int           # refresh period / radius K
    ragged: tuple | None = None  # (lo, hi) inclusive prompt-length range


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    decode: DecodeShape
    weight_seed: int = 0
    prompt_seed: int = 1
    length_seed: int = 2
    note: str = ""

    def with_model(self, **kw) -> "Workload":
        return dataclasses.replace(self, model=dataclasses.replace(self.model, **kw))

    def with_decode(self, **kw) -> "Workload":
        return dataclasses.replace(self, decode=dataclasses.replace(self.decode, **kw))


_LLADA = ModelShape(n_layers=32, d_model=4096, n_heads=32, n_kv_heads=32, head_dim=128,
                    d_ff=12288, vocab=126464, dtype="bf16", gateup_fp16=True)
_DREAM = ModelShape(n_layers=28, d_model=3584, n_heads=28, n_kv_heads=4, head_dim=128,
                    d_ff=18944, vocab=152064, dtype="bf16", gateup_fp16=True)

WORKLOADS = {
    "tiny": Workload(
        "tiny",
        ModelShape(n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64,
                   d_ff=1024, vocab=1024, dtype="fp32"),
        DecodeShape(batch=1, prompt_len=64, resp_len=32, steps=32, unmask_per_step=1,
                    remask_threshold=0.1, refresh_every=4),
        note="tiny bidirectional DLM, fp32"),
    "llada_p512": Workload(
        "llada_p512", _LLADA,
        DecodeShape(batch=1, prompt_len=512, resp_len=256, steps=256, unmask_per_step=1,
                    remask_threshold=0.1, refresh_every=8),
        note="LLaDA-8B-shaped, prompt 512, response 256"),
    "llada_p4096": Workload(
        "llada_p4096", _LLADA,
        DecodeShape(batch=1, prompt_len=4096, resp_len=256, steps=128, unmask_per_step=2,
                    remask_threshold=0.1, refresh_every=16),
        note="LLaDA-8B-shaped long-prompt reuse regime"),
    "llada_ragged16": Workload(
        "llada_ragged16", _LLADA,
        DecodeShape(batch=16, prompt_len=2048, resp_len=256, steps=256, unmask_per_step=1,
                    remask_threshold=0.1, refresh_every=8, ragged=(256, 2048)),
        note="LLaDA-8B-shaped batch 16, ragged prompts U[256,2048]"),
    "dream_gqa": Workload(
        "dream_gqa", _DREAM,
        DecodeShape(batch=4, prompt_len=1024, resp_len=512, steps=512, unmask_per_step=1,
                    remask_threshold=0.1, refresh_every=8),
        note="Dream-7B-shaped GQA (28 q heads / 4 kv heads), batch 4"),
}


def get_workload(name: str) -> Workload:
    return WORKLOADS[name]
