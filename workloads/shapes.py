"""Parameter tables of the model shapes the synchronisation round is measured on.

A synchronisation round treats the model as one flat vector of parameters, so a
shape only fixes N (the parameter count) and how the flat arena splits into
tensors.  Every tensor size here is a multiple of 4, so packing the tensors back
to back keeps each of them 16-byte aligned inside a 16-byte-aligned arena.

Shapes:
  * GPT-2 small: 12 layers, d=768, vocab 50257, 1024 positions, tied LM head
    (148 tensors, 124,439,808 parameters).
  * Llama-style 1.1B: 22 layers, d=2048, FFN 5632, vocab 32000, 32 query heads
    and 4 key/value heads of width 64, untied head (201 tensors, 1,100,048,384).
  * Llama-style 3B: 26 layers, d=3072, FFN 8192, vocab 32000, full multi-head
    attention, untied head (237 tensors, 3,141,172,224).
  * Llama-style 7B: 32 layers, d=4096, FFN 11008, vocab 32000, full multi-head
    attention, untied head (291 tensors, 6,738,415,616).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Tuple


@dataclass(frozen=True)
class ModelShape:
    name: str
    tensors: Tuple[Tuple[str, Tuple[int, ...]], ...]

    @property
    def n_params(self) -> int:
        total = 0
        for _, shp in self.tensors:
            size = 1
            for s in shp:
                size *= s
            total += size
        return total

    @property
    def n_tensors(self) -> int:
        return len(self.tensors)

    def offsets(self) -> List[Tuple[str, int, int]]:
        """(name, offset, numel) of each tensor inside the flat arena."""
        out = []
        off = 0
        for name, shp in self.tensors:
            size = 1
            for s in shp:
                size *= s
            out.append((name, off, size))
            off += size
        return out


def gpt2_small() -> ModelShape:
    d, vocab, ctx, layers = 768, 50257, 1024, 12
    t: List[Tuple[str, Tuple[int, ...]]] = [("wte", (vocab, d)), ("wpe", (ctx, d))]
    for i in range(layers):
        p = f"h.{i}."
        t += [
            (p + "ln_1.weight", (d,)), (p + "ln_1.bias", (d,)),
            (p + "attn.c_attn.weight", (d, 3 * d)), (p + "attn.c_attn.bias", (3 * d,)),
            (p + "attn.c_proj.weight", (d, d)), (p + "attn.c_proj.bias", (d,)),
            (p + "ln_2.weight", (d,)), (p + "ln_2.bias", (d,)),
            (p + "mlp.c_fc.weight", (d, 4 * d)), (p + "mlp.c_fc.bias", (4 * d,)),
            (p + "mlp.c_proj.weight", (4 * d, d)), (p + "mlp.c_proj.bias", (d,)),
        ]
    t += [("ln_f.weight", (d,)), ("ln_f.bias", (d,))]
    return ModelShape("gpt2-small", tuple(t))


def _llama(name: str, layers: int, d: int, ffn: int, vocab: int, kv_dim: int) -> ModelShape:
    t: List[Tuple[str, Tuple[int, ...]]] = [("embed_tokens", (vocab, d))]
    for i in range(layers):
        p = f"layers.{i}."
        t += [
            (p + "self_attn.q_proj", (d, d)),
            (p + "self_attn.k_proj", (kv_dim, d)),
            (p + "self_attn.v_proj", (kv_dim, d)),
            (p + "self_attn.o_proj", (d, d)),
            (p + "mlp.gate_proj", (ffn, d)),
            (p + "mlp.up_proj", (ffn, d)),
            (p + "mlp.down_proj", (d, ffn)),
            (p + "input_layernorm", (d,)),
            (p + "post_attention_layernorm", (d,)),
        ]
    t += [("norm", (d,)), ("lm_head", (vocab, d))]
    return ModelShape(name, tuple(t))


def llama_1b1() -> ModelShape:
    return _llama("llama-1.1b", 22, 2048, 5632, 32000, 4 * 64)


def llama_3b() -> ModelShape:
    return _llama("llama-3b", 26, 3072, 8192, 32000, 3072)


def llama_7b() -> ModelShape:
    return _llama("llama-7b", 32, 4096, 11008, 32000, 4096)


SHAPES = {
    "gpt2-small": gpt2_small,
    "llama-1.1b": llama_1b1,
    "llama-3b": llama_3b,
    "llama-7b": llama_7b,
}
