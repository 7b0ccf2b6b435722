"""The five workloads: layer shapes and batch recipes.

Shapes are those of the Llama-family dense GQA decoder layers the paper serves
(Llama-70B and CodeLlama-34B in §III, DeepSeek-R1-Llama-70B in the evaluation),
scaled to an 8B-shaped and a 70B-shaped layer, plus a tiny fp32 layer for exact
brute-force cross-checks.
"""
from dataclasses import dataclass, field
from typing import Optional, Tuple

PAGE_TOKENS = 16


@dataclass(frozen=True)
class LayerShape:
    hidden: int
    n_q: int
    n_kv: int
    head_dim: int
    ffn: int
    eps: float
    theta: float
    dtype: str  # "f32" or "bf16": storage type of weights, activations and KV

    @property
    def group(self) -> int:
        return self.n_q // self.n_kv

    @property
    def d_q(self) -> int:
        return self.n_q * self.head_dim

    @property
    def d_kv(self) -> int:
        return self.n_kv * self.head_dim

    @property
    def elt_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


@dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int
    shape: LayerShape
    # prefill: n prompts x prompt tokens (0 = none)
    prefill_seqs: int = 0
    prefill_tokens: int = 0
    # decode: batch, number of steps, context-length law
    decode_batch: int = 0
    decode_steps: int = 0
    ctx_law: str = ""           # "uniform", "lognormal", "fixed", "after_prefill"
    ctx_params: Tuple = ()
    # mixed step: new requests x chunk tokens fused with the decode batch
    mixed_new: int = 0
    mixed_chunk: int = 0
    n_layers: int = 1
    vocab: int = 0
    shuffled_pages: bool = True
    note: str = ""


TINY = LayerShape(256, 4, 2, 64, 1024, 1e-5, 10000.0, "f32")
L8B = LayerShape(4096, 32, 8, 128, 14336, 1e-5, 500000.0, "bf16")
L70B = LayerShape(8192, 64, 8, 128, 28672, 1e-5, 500000.0, "bf16")

CONFIGS = {
    "tiny_f32": Workload(
        "tiny_f32", 1, TINY, prefill_seqs=4, prefill_tokens=128,
        decode_batch=4, decode_steps=16, ctx_law="after_prefill",
        note="tiny fp32 layer: prefill 4x128 then 16 decode steps on a shuffled paged cache"),
    "llama8b_prefill": Workload(
        "llama8b_prefill", 2, L8B, prefill_seqs=8, prefill_tokens=2048,
        note="8B-shaped layer, causal prefill of 8 prompts x 2048 tokens"),
    "llama8b_decode": Workload(
        "llama8b_decode", 3, L8B, decode_batch=64, decode_steps=64,
        ctx_law="uniform", ctx_params=(1024, 4096),
        note="8B-shaped layer, decode batch 64, context U{1024..4096}, 64 steps"),
    "llama8b_think": Workload(
        "llama8b_think", 4, L8B, decode_batch=32, decode_steps=64,
        ctx_law="lognormal", ctx_params=(12288.0, 0.5, 4096, 32768),
        mixed_new=4, mixed_chunk=512,
        note="8B-shaped layer, think decode batch 32 with log-normal contexts "
             "(median 12288, sigma 0.5, clipped to [4096, 32768]) plus a mixed step"),
    "llama70b_model": Workload(
        "llama70b_model", 5, L70B, prefill_seqs=8, prefill_tokens=1024,
        decode_batch=64, decode_steps=64, ctx_law="fixed", ctx_params=(4096,),
        n_layers=80, vocab=128256,
        note="80-layer 70B-shaped model: decode batch 64 at context 4096, prefill 8x1024"),
}


def get(name: str) -> Workload:
    return CONFIGS[name]
