"""Oracle, part 1: the target decoder and plain greedy decoding, in float64 on the CPU.

TEST INFRASTRUCTURE ONLY. Nothing on the product path may import or call this package: only
tests/, the smoke check and the CPU-baseline leg of the benchmark use it.

The paper fixes no architecture for its targets beyond "a decoder with L layers" and a PDM that is a
standard-attention decoder (Section 3.1). The workloads fix the rest: a pre-norm dense decoder with
grouped-query attention, rotary position embedding, RMSNorm and a SwiGLU MLP, without biases, with
untied input embedding and LM head. Greedy decoding picks the lowest index among equal maxima.

Precision: every value is float64. Weights are the workload's stored values (bf16-rounded where the
workload stores bf16). Keys and values are rounded to the workload's KV storage type when they are
written to the cache (bf16 for the 4B/9B-class workloads, unrounded for the fp32 tiny model), since
the workloads define the KV cache in that precision.
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np

import synth


# ----------------------------------------------------------------------------- weights
class Model:
    """Weights of one workload, drawn lazily from the shared seeded generator as float64."""

    def __init__(self, shape: synth.ModelShape, seed: int, overrides: Optional[Dict[str, np.ndarray]] = None):
        self.shape = shape
        self.seed = seed
        self.overrides = dict(overrides or {})
        self._w: Dict[str, np.ndarray] = {}

    def w(self, name: str) -> np.ndarray:
        if name not in self._w:
            if name in self.overrides:
                self._w[name] = np.asarray(self.overrides[name], dtype=np.float64)
            else:
                self._w[name] = synth.tensor(self.shape, self.seed, name).astype(np.float64)
        return self._w[name]

    def layer(self, l: int, prefix: str = "layer") -> Dict[str, np.ndarray]:
        return {k: self.w(f"{prefix}.{l}.{k}") for k in self.shape.layer_shapes()}

    def for_width(self, n: int, pdm_layers: Optional[int] = None) -> "Model":
        """The same target with SPD width n (and PDM depth): target weights are shared, the PDM's
        input projection has width n*d and so is drawn for that shape."""
        ls = self.shape.pdm_layers if pdm_layers is None else pdm_layers
        if n == self.shape.n_stages and ls == self.shape.pdm_layers:
            return self
        m = Model(self.shape.with_(n_stages=n, pdm_layers=ls), self.seed, self.overrides)
        m._w = {k: v for k, v in self._w.items() if not k.startswith("pdm.")}
        return m

    def drop(self, prefix: str) -> None:
        for k in [k for k in self._w if k.startswith(prefix)]:
            del self._w[k]


# ----------------------------------------------------------------------------- primitives
def round_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 value (8 significant bits, ties to even) of each float64 entry."""
    m, e = np.frexp(np.asarray(x, dtype=np.float64))
    return np.ldexp(np.rint(m * 256.0), e - 8)


def round_kv(x: np.ndarray, kv_dtype: str) -> np.ndarray:
    return round_bf16(x) if kv_dtype == "bf16" else np.asarray(x, dtype=np.float64)


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope_angles(pos, head_dim: int, base: float) -> np.ndarray:
    """theta_j = pos * base^(-2j/head_dim) for j < head_dim/2, evaluated in float64."""
    j = np.arange(head_dim // 2, dtype=np.float64)
    inv = np.power(float(base), -2.0 * j / head_dim)
    return np.multiply.outer(np.asarray(pos, dtype=np.float64), inv)


def rope(x: np.ndarray, pos: int, base: float) -> np.ndarray:
    """Rotate-half RoPE: channel j pairs with j + dh/2 and turns by angle theta_j(pos).

    x has shape [heads, dh]."""
    dh = x.shape[-1]
    h = dh // 2
    ang = rope_angles(pos, dh, base)
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :h], x[..., h:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def argmax_first(v: np.ndarray) -> int:
    """Index of the largest entry; the lowest index wins among equal maxima."""
    return int(np.argmax(v))  # numpy returns the first occurrence


# ----------------------------------------------------------------------------- KV cache
class LayerCache:
    """Keys and values of one layer, one row per position, in position order."""

    def __init__(self, n_kv: int, dh: int, cap: int = 64):
        self.k = np.zeros((cap, n_kv, dh))
        self.v = np.zeros((cap, n_kv, dh))
        self.n = 0

    def append(self, pos: int, k: np.ndarray, v: np.ndarray) -> None:
        assert pos == self.n, f"KV append at position {pos} but cache holds {self.n} rows"
        if self.n == self.k.shape[0]:
            self.k = np.concatenate([self.k, np.zeros_like(self.k)])
            self.v = np.concatenate([self.v, np.zeros_like(self.v)])
        self.k[self.n] = k
        self.v[self.n] = v
        self.n += 1

    def truncate(self, n: int) -> None:
        assert 0 <= n <= self.n
        self.n = n

    def clone(self) -> "LayerCache":
        c = LayerCache(self.k.shape[1], self.k.shape[2], 1)
        c.k, c.v, c.n = self.k[: self.n].copy(), self.v[: self.n].copy(), self.n
        return c


def attend(q: np.ndarray, cache: LayerCache, upto: int) -> np.ndarray:
    """Scaled dot-product attention of one position's query heads over cache rows [0, upto].

    q: [Hq, dh]. Query head h reads KV head h // (Hq/Hkv). Softmax is max-subtracted."""
    hq, dh = q.shape
    hkv = cache.k.shape[1]
    grp = hq // hkv
    K = cache.k[: upto + 1]  # [T, Hkv, dh]
    V = cache.v[: upto + 1]
    qg = q.reshape(hkv, grp, dh)
    s = np.einsum("hgd,thd->hgt", qg, K) / np.sqrt(dh)
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=-1, keepdims=True)
    o = np.einsum("hgt,thd->hgd", p, V)
    return o.reshape(hq * dh)


def decoder_layer(shape: synth.ModelShape, lw: Dict[str, np.ndarray], h: np.ndarray, pos: int,
                  cache: LayerCache) -> np.ndarray:
    """One token at position pos through one pre-norm decoder layer; appends its K/V to cache."""
    eps, dh = shape.rms_eps, shape.head_dim
    u = rms_norm(h, lw["attn_norm"], eps)
    q = (lw["wq"] @ u).reshape(shape.n_q_heads, dh)
    k = (lw["wk"] @ u).reshape(shape.n_kv_heads, dh)
    v = (lw["wv"] @ u).reshape(shape.n_kv_heads, dh)
    q = rope(q, pos, shape.rope_base)
    k = rope(k, pos, shape.rope_base)
    cache.append(pos, round_kv(k, shape.dtype), round_kv(v, shape.dtype))
    o = attend(q, cache, pos)
    h = h + lw["wo"] @ o
    u = rms_norm(h, lw["mlp_norm"], eps)
    return h + lw["wd"] @ (silu(lw["wg"] @ u) * (lw["wu"] @ u))


def lm_logits(model: Model, h: np.ndarray, norm: str = "final_norm") -> np.ndarray:
    return model.w("lm_head") @ rms_norm(h, model.w(norm), model.shape.rms_eps)


def embed(model: Model, tok: int) -> np.ndarray:
    return model.w("embed")[int(tok)].copy()


def new_caches(shape: synth.ModelShape, n: int) -> List[LayerCache]:
    return [LayerCache(shape.n_kv_heads, shape.head_dim) for _ in range(n)]


# ----------------------------------------------------------------------------- plain decoding
def run_token(model: Model, caches: List[LayerCache], tok: int, pos: int,
              layers: Optional[range] = None, keep: Optional[List[int]] = None):
    """Embed tok and run it at position pos through `layers` (default: all).

    Returns the final hidden state and, if keep lists layer indices, {l: H^l} for those l
    (H^0 is the embedding; H^l is the output of layer l-1)."""
    L = model.shape.n_layers
    layers = range(L) if layers is None else layers
    h = embed(model, tok)
    kept = {}
    if keep is not None and 0 in keep:
        kept[0] = h.copy()
    for l in layers:
        h = decoder_layer(model.shape, model.layer(l), h, pos, caches[l])
        if keep is not None and (l + 1) in keep:
            kept[l + 1] = h.copy()
    return h, kept


def ar_greedy(model: Model, prompt, n_new: int, return_logits: bool = False):
    """Plain greedy decoding: prefill the prompt one position at a time, then generate.

    Returns n_new tokens; the first is argmax of the logits at the last prompt position."""
    caches = new_caches(model.shape, model.shape.n_layers)
    h = None
    for p, t in enumerate(prompt):
        h, _ = run_token(model, caches, int(t), p)
    out, logs = [], []
    pos = len(prompt)
    for _ in range(n_new):
        lg = lm_logits(model, h)
        x = argmax_first(lg)
        out.append(x)
        logs.append(lg)
        if len(out) == n_new:
            break
        h, _ = run_token(model, caches, x, pos)
        pos += 1
    return (out, logs) if return_logits else out


def forward_full(model: Model, tokens, layers_out=None, free_layers: bool = False) -> Dict[int, np.ndarray]:
    """Brute force without any cache: full causal attention over all rows at every layer.

    Returns {l: H^l [T, d]} for l in layers_out (default: every l in 0..L). free_layers drops each
    layer's weights once the layer is done (same arithmetic; for full-size models, whose float64
    weights do not all fit in memory at once)."""
    H = model.w("embed")[np.asarray(tokens, dtype=np.int64)].copy()
    return forward_rows(model, H, "layer", model.shape.n_layers, layers_out, free_layers)


def forward_rows(model: Model, H0: np.ndarray, prefix: str, n_layers: int, layers_out=None,
                 free_layers: bool = False, caches: Optional[List[LayerCache]] = None) -> Dict[int, np.ndarray]:
    """Layers 0..n_layers-1 named `prefix` ("layer": the target, "pdm.layer": the draft module's)
    over the rows H0 [T, d], row t at position t, each attending causally to rows 0..t, without any
    cache. Returns {l: H^l [T, d]} for l in layers_out (default every l in 0..n_layers; H^0 = H0).
    caches: empty per-layer caches that receive each layer's keys and values of the T rows (as a
    token-by-token pass would have appended them)."""
    sh = model.shape
    dh = sh.head_dim
    H = np.array(H0, dtype=np.float64)
    T = H.shape[0]
    layers_out = list(range(n_layers + 1)) if layers_out is None else list(layers_out)
    res = {0: H.copy()} if 0 in layers_out else {}
    grp = sh.n_q_heads // sh.n_kv_heads
    causal = np.tril(np.ones((T, T), dtype=bool))
    for l in range(n_layers):
        lw = model.layer(l, prefix)
        U = rms_norm(H, lw["attn_norm"], sh.rms_eps)
        Q = (U @ lw["wq"].T).reshape(T, sh.n_q_heads, dh)
        K = (U @ lw["wk"].T).reshape(T, sh.n_kv_heads, dh)
        V = (U @ lw["wv"].T).reshape(T, sh.n_kv_heads, dh)
        Q = np.stack([rope(Q[t], t, sh.rope_base) for t in range(T)])
        K = round_kv(np.stack([rope(K[t], t, sh.rope_base) for t in range(T)]), sh.dtype)
        V = round_kv(V, sh.dtype)
        if caches is not None:
            for t in range(T):
                caches[l].append(t, K[t], V[t])
        O = np.zeros((T, sh.n_q_heads, dh))
        for h in range(sh.n_q_heads):
            kv = h // grp
            S = Q[:, h, :] @ K[:, kv, :].T / np.sqrt(dh)
            S = np.where(causal, S, -np.inf)
            S = S - S.max(axis=1, keepdims=True)
            P = np.exp(S)
            P = P / P.sum(axis=1, keepdims=True)
            O[:, h, :] = P @ V[:, kv, :]
        H = H + O.reshape(T, -1) @ lw["wo"].T
        U = rms_norm(H, lw["mlp_norm"], sh.rms_eps)
        H = H + (silu(U @ lw["wg"].T) * (U @ lw["wu"].T)) @ lw["wd"].T
        if (l + 1) in layers_out:
            res[l + 1] = H.copy()
        if free_layers:
            del lw
            model.drop(f"{prefix}.{l}.")
    return res
