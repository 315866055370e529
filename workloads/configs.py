"""Model shapes and workload definitions.

The paper evaluates Llama2-7B and Llama2-13B served in FP16 with pipeline
parallelism of up to four stages (section 4.1 limits the size to 4; section 8
uses 4 stages, and 2 for the scale-down study). Trained weights and the
request datasets are not available, so every workload here is synthetic: the
model shapes are those of the named models, weights are drawn N(0, 0.02) from
fixed seeds and prompts are uniform token ids.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple


@dataclasses.dataclass(frozen=True)
class ModelCfg:
    """Shape of a Llama-style decoder (pre-norm RMSNorm, rotate-half RoPE,
    SwiGLU FFN, grouped-query attention, no biases, untied LM head)."""
    name: str
    n_layers: int
    hidden: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    rms_eps: float = 1e-5
    rope_base: float = 10000.0

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def group(self) -> int:
        return self.n_heads // self.n_kv_heads


MODELS = {
    # Tiny decoder used for exact end-to-end checks.
    "tiny": ModelCfg("tiny", n_layers=2, hidden=256, n_heads=4, n_kv_heads=4,
                     head_dim=64, ffn=688, vocab=1024),
    "llama2-7b": ModelCfg("llama2-7b", n_layers=32, hidden=4096, n_heads=32,
                          n_kv_heads=32, head_dim=128, ffn=11008, vocab=32000),
    "llama2-13b": ModelCfg("llama2-13b", n_layers=40, hidden=5120, n_heads=40,
                           n_kv_heads=40, head_dim=128, ffn=13824, vocab=32000),
    "llama3-8b": ModelCfg("llama3-8b", n_layers=32, hidden=4096, n_heads=32,
                          n_kv_heads=8, head_dim=128, ffn=14336, vocab=128256,
                          rope_base=500000.0),
}


@dataclasses.dataclass(frozen=True)
class Workload:
    """One serving workload: a model, its stage cuts, the batch and the
    number of greedy decode steps.

    ``stages`` lists contiguous layer ranges [begin, end). ``prompt_lens``
    is either a tuple of per-sequence lengths or None, in which case the
    lengths come from ``ragged`` = (low, high_inclusive, n, seed).
    ``seed`` selects the token stream.
    """
    name: str
    model: str
    stages: Tuple[Tuple[int, int], ...]
    batch: int
    prompt_lens: Optional[Tuple[int, ...]]
    decode_steps: int
    seed: int
    ragged: Optional[Tuple[int, int, int, int]] = None
    bench_stage: Optional[int] = None  # index into stages of the stage timed
    kv_block: int = 16

    @property
    def cfg(self) -> ModelCfg:
        return MODELS[self.model]

    def lengths(self):
        from .gen import ragged_lengths
        if self.prompt_lens is not None:
            return list(self.prompt_lens)
        lo, hi, n, seed = self.ragged
        return ragged_lengths(lo, hi, n, seed)


def _even(n_layers: int, n_stages: int):
    per = n_layers // n_stages
    return tuple((i * per, (i + 1) * per) for i in range(n_stages))


WORKLOADS = {
    # 2 layers split into 2 one-layer stages; batch 1, 32-token prompt,
    # 16 greedy decode steps.
    "tiny-2x1": Workload("tiny-2x1", "tiny", ((0, 1), (1, 2)), batch=1,
                         prompt_lens=(32,), decode_steps=16, seed=1),
    # 7B shape cut into 4 stages; the second stage (layers 8-15) is loaded
    # cold from pinned host memory while it prefills one 512-token prompt.
    "7b-stage8-15-cold": Workload("7b-stage8-15-cold", "llama2-7b",
                                  _even(32, 4), batch=1, prompt_lens=(512,),
                                  decode_steps=0, seed=2, bench_stage=1),
    # 7B shape as one consolidated stage with the LM head: batch 8 x 1024
    # prompt tokens, then 128 greedy decode steps over a paged KV cache.
    "7b-full-b8": Workload("7b-full-b8", "llama2-7b", ((0, 32),), batch=8,
                           prompt_lens=(1024,) * 8, decode_steps=128, seed=3,
                           bench_stage=0),
    # 13B shape cut into 2 stages of 20 layers; batch 4 x 2048, 64 steps.
    "13b-2x20-b4": Workload("13b-2x20-b4", "llama2-13b", _even(40, 2), batch=4,
                            prompt_lens=(2048,) * 4, decode_steps=64, seed=4,
                            bench_stage=0),
    # 8B GQA shape in 4 stages; 16 ragged prompts in [128, 2048], KV export
    # from every stage and import into one merged worker, 256 decode steps.
    "8b-4x8-ragged-merge": Workload("8b-4x8-ragged-merge", "llama3-8b",
                                    _even(32, 4), batch=16, prompt_lens=None,
                                    decode_steps=256, seed=5,
                                    ragged=(128, 2048, 16, 0)),
    # Scaling down (the consolidation study of the evaluation): 13B shape in
    # 4 stages of 10 layers, 512-token prompts, 512 generated tokens. The
    # first stage holds all 40 layers' memory, loads the rest of the model in
    # the background while the pipeline decodes, then absorbs the others'
    # KV cache and decodes alone.
    "13b-4x10-scale-down": Workload("13b-4x10-scale-down", "llama2-13b", _even(40, 4),
                                    batch=4, prompt_lens=(512,) * 4, decode_steps=512,
                                    seed=6),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]
