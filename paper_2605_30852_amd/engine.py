"""Device memory and streams for one SPD handle: weights uploaded from the seeded generator, the
workspace, two HIP streams, and the binding's calls bound to the handle.

PyTorch only allocates device memory and streams here; every computation runs in libspd.so."""
from __future__ import annotations

import ctypes as ct
from typing import Dict, List, Optional

import numpy as np
import torch

import synth
from . import binding as B


def make_config(shape: synth.ModelShape, max_tokens: int, n: Optional[int] = None,
                pdm_layers: Optional[int] = None, auto_rollback: bool = True, attn_chunk: int = 0,
                page_seed: int = 0, fused_head: bool = True) -> B.spd_config:
    c = B.spd_config()
    c.n_layers = shape.n_layers
    c.d_model = shape.d_model
    c.n_q_heads = shape.n_q_heads
    c.n_kv_heads = shape.n_kv_heads
    c.head_dim = shape.head_dim
    c.ffn_dim = shape.ffn_dim
    c.vocab = shape.vocab
    c.rms_eps = shape.rms_eps
    c.rope_base = shape.rope_base
    c.dtype = B.SPD_BF16 if shape.dtype == "bf16" else B.SPD_F32
    c.n_stages = shape.n_stages if n is None else n
    c.pdm_layers = shape.pdm_layers if pdm_layers is None else pdm_layers
    c.page_size = shape.page_size
    c.max_tokens = max_tokens
    c.auto_rollback = 1 if auto_rollback else 0
    c.attn_chunk = attn_chunk
    c.page_seed = page_seed
    c.fused_head = 1 if fused_head else 0
    c.pdm_vocab = shape.pdm_vocab
    return c


class DeviceWeights:
    """All tensors of one workload (target + PDM for width n) resident on the GPU."""

    def __init__(self, shape: synth.ModelShape, seed: int, device="cuda", threads: int = 8,
                 overrides: Optional[Dict[str, np.ndarray]] = None):
        self.shape = shape
        self.seed = seed
        self.t: Dict[str, torch.Tensor] = {}
        for name, arr in synth.iter_storage(shape, seed, threads=threads):
            if overrides and name in overrides:
                arr = self._storage(overrides[name], name)
            self.t[name] = self._upload(arr, device)
        if shape.pdm_vocab:
            self.t["pdm.vocab_map"] = self._upload(synth.pdm_vocab_map(shape, seed), device)

    def _storage(self, values: np.ndarray, name: str) -> np.ndarray:
        v = np.asarray(values, dtype=np.float32)
        if synth.is_norm(name) or self.shape.dtype != "bf16":
            return v
        return synth.bf16_bits(v).reshape(v.shape)

    @staticmethod
    def _upload(arr: np.ndarray, device) -> torch.Tensor:
        if arr.dtype == np.uint16:
            return torch.from_numpy(arr.view(np.int16)).to(device).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(arr)).to(device)

    def ptr(self, name: str) -> int:
        return self.t[name].data_ptr()

    def pdm_for_width(self, n: int, pdm_layers: Optional[int] = None, device="cuda") -> "DeviceWeights":
        """A view with the PDM of width n (and depth): the target tensors are shared."""
        ls = self.shape.pdm_layers if pdm_layers is None else pdm_layers
        if n == self.shape.n_stages and ls == self.shape.pdm_layers:
            return self
        other = DeviceWeights.__new__(DeviceWeights)
        other.shape = self.shape.with_(n_stages=n, pdm_layers=ls)
        other.seed = self.seed
        other.t = {k: v for k, v in self.t.items() if not k.startswith("pdm.")}
        for name in other.shape.tensor_shapes():
            if name.startswith("pdm."):
                other.t[name] = self._upload(synth.tensor_storage(other.shape, self.seed, name), device)
        if "pdm.vocab_map" in self.t:
            other.t["pdm.vocab_map"] = self.t["pdm.vocab_map"]
        return other

    def with_pdm_vocab(self, pdm_vocab: int, device="cuda") -> "DeviceWeights":
        """A view whose PDM has its own LM head over pdm_vocab tokens (initialised from the target's
        rows of that vocabulary); every other tensor is shared."""
        other = DeviceWeights.__new__(DeviceWeights)
        other.shape = self.shape.with_(pdm_vocab=pdm_vocab)
        other.seed = self.seed
        other.t = {k: v for k, v in self.t.items() if k not in ("pdm.lm_head", "pdm.vocab_map")}
        if pdm_vocab:
            other.t["pdm.lm_head"] = self._upload(synth.tensor_storage(other.shape, self.seed, "pdm.lm_head"), device)
            other.t["pdm.vocab_map"] = self._upload(synth.pdm_vocab_map(other.shape, self.seed), device)
        return other

    def struct(self):
        sh = self.shape

        def lw(prefix, l):
            s = B.spd_layer_weights()
            for k in ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "wg", "wu", "wd"):
                setattr(s, k, self.ptr(f"{prefix}.{l}.{k}"))
            return s

        layers = (B.spd_layer_weights * sh.n_layers)(*[lw("layer", l) for l in range(sh.n_layers)])
        pdm = (B.spd_layer_weights * sh.pdm_layers)(*[lw("pdm.layer", l) for l in range(sh.pdm_layers)])
        w = B.spd_weights()
        w.embed = self.ptr("embed")
        w.layers = ct.cast(layers, ct.POINTER(B.spd_layer_weights))
        w.final_norm = self.ptr("final_norm")
        w.lm_head = self.ptr("lm_head")
        w.pdm_in = self.ptr("pdm.in")
        w.pdm_layers = ct.cast(pdm, ct.POINTER(B.spd_layer_weights))
        w.pdm_norm = self.ptr("pdm.norm")
        if sh.pdm_vocab:
            w.pdm_lm_head = self.ptr("pdm.lm_head")
            w.pdm_vocab_map = self.ptr("pdm.vocab_map")
        return w, (layers, pdm)


class Engine:
    """One SPD handle on cuda:0 with its own workspace and streams."""

    def __init__(self, weights: DeviceWeights, max_tokens: int, n: Optional[int] = None,
                 pdm_layers: Optional[int] = None, auto_rollback: bool = True, attn_chunk: int = 0,
                 page_seed: int = 0, fused_head: Optional[bool] = None, device="cuda",
                 ws_fill: Optional[int] = None):
        """fused_head: None picks the two-row pass when the PDM shares the target's head.
        ws_fill: a byte value written over the whole workspace before spd_init (0xFF makes every
        float the library has not written a NaN; for tests that nothing stale is read)."""
        if not torch.cuda.is_available():
            raise RuntimeError("Engine needs a GPU: the SPD step has no CPU path")
        n = weights.shape.n_stages if n is None else n
        self.w = weights.pdm_for_width(n, pdm_layers, device)
        self.shape = self.w.shape
        if fused_head is None:
            fused_head = self.shape.pdm_vocab == 0
        self.cfg = make_config(self.shape, max_tokens, n=n, auto_rollback=auto_rollback,
                               attn_chunk=attn_chunk, page_seed=page_seed, fused_head=fused_head)
        self.n = n
        nbytes = B.spd_workspace_size(self.cfg)
        self.ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
        if ws_fill is not None:
            self.ws.fill_(int(ws_fill))
        base = self.ws.data_ptr()
        aligned = (base + 255) // 256 * 256
        # default priority streams only
        self.main = torch.cuda.Stream(device=device)
        self.pdm = torch.cuda.Stream(device=device)
        wstruct, self._keep = self.w.struct()
        torch.cuda.synchronize()  # weights were uploaded on torch's stream
        self.h = B.spd_init(self.cfg, wstruct, aligned, nbytes, self.main.cuda_stream, self.pdm.cuda_stream)
        self.prompt_len = 0

    # thin wrappers with the C names
    def spd_prefill(self, prompt) -> int:
        self.prompt_len = len(prompt)
        return B.spd_prefill(self.h, prompt)

    def spd_step(self, forced_draft: Optional[int] = None) -> B.spd_step_result:
        return B.spd_step(self.h, forced_draft)

    def spd_rollback(self, keep_len: int, reseed: int) -> None:
        B.spd_rollback(self.h, keep_len, reseed)

    def spd_set_forced_drafts(self, table, first_pos: int) -> None:
        B.spd_set_forced_drafts(self.h, table, first_pos)

    def spd_clear_forced_drafts(self) -> None:
        B.spd_clear_forced_drafts(self.h)

    def spd_run_steps(self, count: int, want_log: bool = False):
        return B.spd_run_steps(self.h, count, want_log)

    def spd_sync(self):
        return B.spd_sync(self.h)

    def spd_set_graph(self, on: bool) -> None:
        B.spd_set_graph(self.h, on)

    def spd_set_step_kernel(self, mode: int, grid: int = 0, groups: int = -1) -> None:
        B.spd_set_step_kernel(self.h, mode, grid, groups)

    def spd_set_pdm_placement(self, place: int) -> None:
        B.spd_set_pdm_placement(self.h, place)

    def spd_set_graph_steps(self, steps: int) -> None:
        B.spd_set_graph_steps(self.h, steps)

    def spd_set_pdm_schedule(self, post_step: bool) -> None:
        B.spd_set_pdm_schedule(self.h, post_step)

    def spd_set_sampling(self, top_k: int, temperature: float = 1.0, uniforms=None) -> None:
        B.spd_set_sampling(self.h, top_k, temperature, uniforms)

    def spd_set_pdm_grid(self, wgs: int) -> None:
        B.spd_set_pdm_grid(self.h, wgs)

    def spd_set_debug(self, on: bool) -> None:
        B.spd_set_debug(self.h, on)

    # debug reads
    def resid(self) -> np.ndarray:
        return B.spd_read_debug(self.h, B.SPD_DBG_RESID, self.n * self.shape.d_model).reshape(self.n, -1)

    def anchors(self) -> np.ndarray:
        d = self.shape.d_model
        return B.spd_read_debug(self.h, B.SPD_DBG_ANCHORS, self.n * self.n * d).reshape(self.n, self.n, d)

    def pdm_hidden(self) -> np.ndarray:
        return B.spd_read_debug(self.h, B.SPD_DBG_PDM_HIDDEN, 8 * self.shape.d_model).reshape(8, -1)

    def exit_logits(self) -> np.ndarray:
        return B.spd_read_debug(self.h, B.SPD_DBG_EXIT_LOGITS, self.shape.vocab)

    def pdm_logits(self) -> np.ndarray:
        return B.spd_read_debug(self.h, B.SPD_DBG_PDM_LOGITS, self.shape.pdm_vocab or self.shape.vocab)

    def qdist(self, pos: int):
        """Sampled decoding: (ids, probs) of the draft distribution kept for in-flight position pos."""
        n, K = self.n, B.MAX_TOP_K
        raw = B.spd_read_debug(self.h, B.SPD_DBG_QDIST, n * (1 + 2 * K), np.int32)
        r = pos % n
        cnt = int(raw[r])
        ids = raw[n:n + n * K].reshape(n, K)[r, :cnt].astype(np.int64)
        probs = raw[n + n * K:].view(np.float32).reshape(n, K)[r, :cnt].astype(np.float64)
        return ids, probs

    def tokens(self) -> np.ndarray:
        return B.spd_read_debug(self.h, B.SPD_DBG_TOKENS, self.cfg.max_tokens, np.int32)

    def state(self):
        c, a, p, k = B.spd_read_debug(self.h, B.SPD_DBG_STATE, 4, np.int32)
        return int(c), int(a), int(p), int(k)

    def kv(self, layer: int, pos0: int, count: int, pdm: bool = False):
        k, v = B.spd_read_kv(self.h, 1 if pdm else 0, layer, pos0, count, self.shape.n_kv_heads,
                             self.shape.head_dim, self.shape.dtype == "bf16")
        if self.shape.dtype == "bf16":
            k = synth.bf16_bits_to_f32(k)
            v = synth.bf16_bits_to_f32(v)
        return k, v

    def close(self) -> None:
        if getattr(self, "h", None):
            B.spd_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
