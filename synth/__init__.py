"""Seeded synthetic inputs for the SPD step: model shapes, random weights, prompts, acceptance masks.

This module is the only code the CPU oracle and the GPU path share. It holds no arithmetic of the
method itself: it draws numbers, rounds weights to the storage precision a workload states, and
describes shapes. Every tensor comes from its own numpy PCG64 stream keyed by (seed, crc32(name)),
so any single tensor can be regenerated without drawing the others.
"""
from __future__ import annotations

import dataclasses
import zlib
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, Iterator, List, Optional, Tuple

import numpy as np

WEIGHT_STD = 0.02


@dataclasses.dataclass(frozen=True)
class ModelShape:
    """A dense pre-norm GQA decoder plus the SPD width and PDM depth that run it."""

    name: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    dtype: str  # "f32" or "bf16": storage type of weights and KV cache
    n_stages: int  # SPD width n
    pdm_layers: int  # L_s
    rms_eps: float = 1e-6
    rope_base: float = 10000.0
    page_size: int = 16
    pdm_vocab: int = 0  # 0: the PDM shares the target's LM head; else its own head over this many tokens

    def with_(self, **kw) -> "ModelShape":
        return dataclasses.replace(self, **kw)

    @property
    def q_dim(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def layer_shapes(self) -> Dict[str, Tuple[int, ...]]:
        d, f = self.d_model, self.ffn_dim
        return {
            "attn_norm": (d,),
            "wq": (self.q_dim, d),
            "wk": (self.kv_dim, d),
            "wv": (self.kv_dim, d),
            "wo": (d, self.q_dim),
            "mlp_norm": (d,),
            "wg": (f, d),
            "wu": (f, d),
            "wd": (d, f),
        }

    def tensor_shapes(self) -> Dict[str, Tuple[int, ...]]:
        """Every named tensor of the target model and the PDM, with its shape."""
        d = self.d_model
        out: Dict[str, Tuple[int, ...]] = {"embed": (self.vocab, d)}
        for l in range(self.n_layers):
            for k, s in self.layer_shapes().items():
                out[f"layer.{l}.{k}"] = s
        out["final_norm"] = (d,)
        out["lm_head"] = (self.vocab, d)
        out["pdm.in"] = (d, self.n_stages * d)
        for l in range(self.pdm_layers):
            for k, s in self.layer_shapes().items():
                out[f"pdm.layer.{l}.{k}"] = s
        out["pdm.norm"] = (d,)
        if self.pdm_vocab:
            out["pdm.lm_head"] = (self.pdm_vocab, d)
        return out

    def param_bytes(self, names: Optional[List[str]] = None) -> int:
        esz = 2 if self.dtype == "bf16" else 4
        shapes = self.tensor_shapes()
        tot = 0
        for k, s in shapes.items():
            if names is not None and k not in names:
                continue
            n = int(np.prod(s))
            tot += n * (4 if is_norm(k) else esz)
        return tot


def is_norm(name: str) -> bool:
    return name.endswith("norm")


# Workloads. Shapes follow the dense 4B- and 9B-class targets and the tiny CPU-sized model.
TINY = ModelShape("tiny", 4, 256, 4, 2, 64, 704, 1024, "f32", n_stages=2, pdm_layers=1)
B4 = ModelShape("4b", 36, 2560, 32, 8, 128, 9728, 151936, "bf16", n_stages=4, pdm_layers=1)
B9 = ModelShape("9b", 36, 4096, 32, 8, 128, 12288, 151936, "bf16", n_stages=4, pdm_layers=1)
B9_LONG = B9.with_(name="9b-long", n_stages=8, pdm_layers=2)
# A mid-size bf16 model for parity: several GEMV/attention tiles per launch and ragged tails
# (ffn 1000 and vocab 3001 are not multiples of any tile height).
MID = ModelShape("mid", 6, 384, 8, 2, 64, 1000, 3001, "bf16", n_stages=3, pdm_layers=1)
# A bf16 model with the full-size head shape (heads of 128, 4 query heads per KV head) for parity at
# long contexts and wide pipelines: 10 layers split into 5, 6 or 8 ragged stages, a two-layer draft
# module whose feature projection reads n * 1024 anchors, and an FFN of 5120 (eight rows of its down
# projection input do not fit one workgroup's LDS at once).
WIDE = ModelShape("wide", 10, 1024, 8, 2, 128, 5120, 4096, "bf16", n_stages=8, pdm_layers=2)
# bf16 models with other head ratios: eight query heads per KV head (a prefill chunk's 8 rows are then
# 64 queries per KV head) and plain multi-head attention (one query head per KV head).
GQA8 = ModelShape("gqa8", 5, 256, 16, 2, 64, 704, 2000, "bf16", n_stages=4, pdm_layers=1)
MHA = ModelShape("mha", 4, 256, 4, 4, 64, 704, 2000, "bf16", n_stages=3, pdm_layers=1)

WORKLOADS = {
    "tiny": dict(shape=TINY, prompt_len=64, steps=32, p_accept=None),
    "4b": dict(shape=B4, prompt_len=2048, steps=256, p_accept=0.7),
    "9b": dict(shape=B9, prompt_len=4096, steps=256, p_accept=0.7),
    "4b-sweep": dict(shape=B4, prompt_len=8192, steps=256, p_accept=0.7, widths=(2, 4, 6, 8)),
    "9b-long": dict(shape=B9_LONG, prompt_len=32768, steps=512, p_accept=0.6),
}


def _stream(seed: int, name: str) -> np.random.Generator:
    return np.random.default_rng([int(seed), zlib.crc32(name.encode())])


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest even (inputs here are finite)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + r) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)


def tensor(shape: ModelShape, seed: int, name: str) -> np.ndarray:
    """One named tensor as float32 values (already rounded to bf16 for bf16 workloads).

    Norm gains are 1.0; the PDM's own LM head is initialised from the target's, the rows of its
    vocabulary subset (pdm_vocab_map); every other tensor is N(0, 0.02^2)."""
    s = shape.tensor_shapes()[name]
    if is_norm(name):
        return np.ones(s, dtype=np.float32)
    if name == "pdm.lm_head":
        return tensor(shape, seed, "lm_head")[pdm_vocab_map(shape, seed)]
    x = _stream(seed, name).standard_normal(s, dtype=np.float32)
    x *= np.float32(WEIGHT_STD)
    if shape.dtype == "bf16":
        x = bf16_bits_to_f32(bf16_bits(x)).reshape(s)
    return x


def tensor_storage(shape: ModelShape, seed: int, name: str) -> np.ndarray:
    """The same tensor in its storage format: uint16 bf16 bits, or float32 (norms always float32)."""
    s = shape.tensor_shapes()[name]
    if is_norm(name):
        return np.ones(s, dtype=np.float32)
    if name == "pdm.lm_head":
        return np.ascontiguousarray(tensor_storage(shape, seed, "lm_head")[pdm_vocab_map(shape, seed)])
    x = _stream(seed, name).standard_normal(s, dtype=np.float32)
    x *= np.float32(WEIGHT_STD)
    if shape.dtype == "bf16":
        return bf16_bits(x).reshape(s)
    return x


def pdm_vocab_map(shape: ModelShape, seed: int) -> np.ndarray:
    """The PDM vocabulary: pdm_vocab distinct target token ids, ascending (draft id i is target token
    map[i]), drawn uniformly from the target vocabulary."""
    assert 0 < shape.pdm_vocab <= shape.vocab
    ids = np.random.default_rng([int(seed), 13]).choice(shape.vocab, size=shape.pdm_vocab, replace=False)
    return np.sort(ids).astype(np.int32)


def iter_storage(shape: ModelShape, seed: int, threads: int = 8) -> Iterator[Tuple[str, np.ndarray]]:
    """All tensors in storage format, generated on a thread pool (numpy releases the GIL)."""
    names = list(shape.tensor_shapes())
    with ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
        # bounded look-ahead keeps host memory to a few tensors at a time
        window = max(2, threads * 2)
        futs = {}
        for i, nm in enumerate(names):
            futs[i] = ex.submit(tensor_storage, shape, seed, nm)
            if i >= window:
                j = i - window
                yield names[j], futs.pop(j).result()
        for j in sorted(futs):
            yield names[j], futs[j].result()


def prompt(shape: ModelShape, seed: int, length: int) -> np.ndarray:
    """Uniform-random token ids on [0, vocab) from seed+1."""
    return np.random.default_rng([int(seed) + 1, 7]).integers(0, shape.vocab, size=length, dtype=np.int64).astype(np.int32)


def accept_mask(p: float, seed: int, length: int) -> np.ndarray:
    """Bernoulli(p) bits from seed+2: bit i says whether the draft for position i is forced correct."""
    return np.random.default_rng([int(seed) + 2, 11]).random(length) < p


def forced_drafts(reference: np.ndarray, mask: np.ndarray, vocab: int) -> np.ndarray:
    """Per-position draft override: the reference token where the mask bit is set, else a wrong one."""
    ref = np.asarray(reference, dtype=np.int64)
    m = np.asarray(mask[: len(ref)], dtype=bool)
    return np.where(m, ref, (ref + 1) % vocab).astype(np.int32)
