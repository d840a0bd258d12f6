"""ctypes binding of libspd.so: the C ABI of include/spd.h under the same names.

Argument marshalling only. Every step of the decoding path runs in the library's HIP kernels; there
is no Python or CPU fallback. Loading fails loudly if the library has not been built."""
from __future__ import annotations

import ctypes as ct
import os
from typing import Optional

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libspd.so")

SPD_OK, SPD_E_INVAL, SPD_E_STATE, SPD_E_CAPACITY, SPD_E_HIP = 0, 1, 2, 3, 4
SPD_F32, SPD_BF16 = 0, 1
SPD_NONE, SPD_ACCEPT, SPD_REJECT = 0, 1, 2
SPD_DBG_RESID, SPD_DBG_ANCHORS, SPD_DBG_PDM_HIDDEN = 1, 2, 3
SPD_DBG_EXIT_LOGITS, SPD_DBG_PDM_LOGITS, SPD_DBG_TOKENS, SPD_DBG_STATE = 4, 5, 6, 7
SPD_DBG_KTRACE, SPD_DBG_QDIST = 10, 11
MAX_TOP_K = 64
SPD_K_QKV, SPD_K_ATTN, SPD_K_OPROJ, SPD_K_GATEUP, SPD_K_DOWN, SPD_K_HEAD, SPD_K_SPANS = 1, 2, 3, 4, 5, 6, 7


class spd_config(ct.Structure):
    _fields_ = [
        ("n_layers", ct.c_int32), ("d_model", ct.c_int32), ("n_q_heads", ct.c_int32),
        ("n_kv_heads", ct.c_int32), ("head_dim", ct.c_int32), ("ffn_dim", ct.c_int32),
        ("vocab", ct.c_int32), ("rms_eps", ct.c_float), ("rope_base", ct.c_float),
        ("dtype", ct.c_int32), ("n_stages", ct.c_int32), ("pdm_layers", ct.c_int32),
        ("page_size", ct.c_int32), ("max_tokens", ct.c_int32), ("auto_rollback", ct.c_int32),
        ("attn_chunk", ct.c_int32), ("page_seed", ct.c_uint64), ("fused_head", ct.c_int32),
        ("pdm_vocab", ct.c_int32),
    ]


class spd_layer_weights(ct.Structure):
    _fields_ = [(k, ct.c_void_p) for k in
                ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "wg", "wu", "wd")]


class spd_weights(ct.Structure):
    _fields_ = [
        ("embed", ct.c_void_p), ("layers", ct.POINTER(spd_layer_weights)),
        ("final_norm", ct.c_void_p), ("lm_head", ct.c_void_p), ("pdm_in", ct.c_void_p),
        ("pdm_layers", ct.POINTER(spd_layer_weights)), ("pdm_norm", ct.c_void_p),
        ("pdm_lm_head", ct.c_void_p), ("pdm_vocab_map", ct.c_void_p),
    ]


class spd_step_result(ct.Structure):
    _fields_ = [(k, ct.c_int32) for k in
                ("decision", "target_argmax", "draft", "pdm_draft", "exited_pos", "exited_token", "verified_pos",
                 "verified_token", "committed_len", "inflight", "step_index")]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


EXPORTS = [
    "spd_workspace_size", "spd_stage_bounds", "spd_init", "spd_prefill", "spd_step", "spd_rollback",
    "spd_set_forced_drafts", "spd_clear_forced_drafts", "spd_run_steps", "spd_sync", "spd_read_debug",
    "spd_read_kv", "spd_set_debug", "spd_destroy", "spd_status_str", "spd_last_error",
    "spd_set_kernel_timing", "spd_kernel_timing", "spd_set_graph", "spd_span_timing", "spd_set_step_kernel",
    "spd_step_plan_info", "spd_set_kernel_trace", "spd_set_pdm_placement",
    "spd_set_pdm_grid", "spd_set_pdm_enabled", "spd_probe_hbm_read", "spd_set_sampling",
    "spd_set_pdm_schedule", "spd_set_graph_steps", "spd_decode_attention", "spd_decode_attention_noalloc",
]

_lib: Optional[ct.CDLL] = None


class SPDError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn} failed: {status_str(status)} {msg}".strip())
        self.status = status


def lib() -> ct.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(there is no fallback path)")
        L = ct.CDLL(LIB_PATH)
        P = ct.c_void_p
        I = ct.c_int32
        sig = {
            "spd_workspace_size": (I, [ct.POINTER(spd_config), ct.POINTER(ct.c_size_t)]),
            "spd_stage_bounds": (I, [ct.POINTER(spd_config), ct.POINTER(ct.c_int32)]),
            "spd_init": (I, [ct.POINTER(spd_config), ct.POINTER(spd_weights), P, ct.c_size_t, P, P,
                             ct.POINTER(P)]),
            "spd_prefill": (I, [P, ct.POINTER(ct.c_int32), I, ct.POINTER(ct.c_int32)]),
            "spd_step": (I, [P, ct.POINTER(ct.c_int32), ct.POINTER(spd_step_result)]),
            "spd_rollback": (I, [P, I, I]),
            "spd_set_forced_drafts": (I, [P, ct.POINTER(ct.c_int32), I, I]),
            "spd_clear_forced_drafts": (I, [P]),
            "spd_run_steps": (I, [P, I, ct.POINTER(spd_step_result)]),
            "spd_sync": (I, [P, ct.POINTER(spd_step_result)]),
            "spd_read_debug": (I, [P, I, P, ct.c_size_t]),
            "spd_read_kv": (I, [P, I, I, I, I, P, P]),
            "spd_set_debug": (I, [P, I]),
            "spd_set_kernel_timing": (I, [P, I, I]),
            "spd_set_graph": (I, [P, I]),
            "spd_set_step_kernel": (I, [P, I, I, I]),
            "spd_set_kernel_trace": (I, [P, I]),
            "spd_set_pdm_placement": (I, [P, I]),
            "spd_set_pdm_grid": (I, [P, I]),
            "spd_set_pdm_enabled": (I, [P, I]),
            "spd_set_pdm_schedule": (I, [P, I]),
            "spd_set_graph_steps": (I, [P, I]),
            "spd_set_sampling": (I, [P, I, ct.c_float, ct.POINTER(ct.c_float), I]),
            "spd_probe_hbm_read": (I, [P, ct.c_size_t, P, I, P, ct.POINTER(ct.c_double)]),
            "spd_step_plan_info": (I, [P, ct.POINTER(ct.c_int32)]),
            "spd_kernel_timing": (I, [P, ct.POINTER(ct.c_double), ct.POINTER(ct.c_int32)]),
            "spd_span_timing": (I, [P, ct.POINTER(ct.c_double), ct.POINTER(ct.c_double),
                                    ct.POINTER(ct.c_double), ct.POINTER(ct.c_int32)]),
            "spd_decode_attention": (I, [P, P, P, I, ct.POINTER(ct.c_int32), I, I, I, I, I, I, P, P, ct.c_size_t,
                                         P]),
            "spd_decode_attention_noalloc": (I, [P, P, P, I, ct.POINTER(ct.c_int32), I, I, I, I, I, I, P, P]),
            "spd_destroy": (None, [P]),
            "spd_status_str": (ct.c_char_p, [I]),
            "spd_last_error": (ct.c_char_p, [P]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def status_str(s: int) -> str:
    return lib().spd_status_str(int(s)).decode()


def _check(fn: str, st: int, handle=None):
    if st != SPD_OK:
        msg = lib().spd_last_error(handle).decode() if handle is not None or True else ""
        raise SPDError(fn, st, msg)


# ------------------------------------------------------------------------------- raw calls
def spd_workspace_size(cfg: spd_config) -> int:
    b = ct.c_size_t(0)
    _check("spd_workspace_size", lib().spd_workspace_size(ct.byref(cfg), ct.byref(b)))
    return b.value


def spd_stage_bounds(cfg: spd_config):
    out = (ct.c_int32 * (cfg.n_stages + 1))()
    _check("spd_stage_bounds", lib().spd_stage_bounds(ct.byref(cfg), out))
    return list(out)


def spd_init(cfg: spd_config, weights: spd_weights, workspace: int, ws_bytes: int, main_stream: int,
             pdm_stream: int) -> int:
    h = ct.c_void_p(0)
    st = lib().spd_init(ct.byref(cfg), ct.byref(weights), ct.c_void_p(workspace), ws_bytes,
                        ct.c_void_p(main_stream), ct.c_void_p(pdm_stream), ct.byref(h))
    _check("spd_init", st, None)
    return h.value


def spd_prefill(h: int, prompt) -> int:
    p = np.ascontiguousarray(prompt, dtype=np.int32)
    first = ct.c_int32(-1)
    _check("spd_prefill", lib().spd_prefill(h, p.ctypes.data_as(ct.POINTER(ct.c_int32)), len(p),
                                             ct.byref(first)), h)
    return first.value


def spd_step(h: int, forced_draft: Optional[int] = None) -> spd_step_result:
    r = spd_step_result()
    fd = ct.c_int32(int(forced_draft)) if forced_draft is not None else None
    _check("spd_step", lib().spd_step(h, ct.byref(fd) if fd is not None else None, ct.byref(r)), h)
    return r


def spd_rollback(h: int, keep_len: int, reseed_token: int) -> None:
    _check("spd_rollback", lib().spd_rollback(h, int(keep_len), int(reseed_token)), h)


def spd_set_forced_drafts(h: int, table, first_pos: int) -> None:
    t = np.ascontiguousarray(table, dtype=np.int32)
    _check("spd_set_forced_drafts",
           lib().spd_set_forced_drafts(h, t.ctypes.data_as(ct.POINTER(ct.c_int32)), int(first_pos), len(t)), h)


def spd_clear_forced_drafts(h: int) -> None:
    _check("spd_clear_forced_drafts", lib().spd_clear_forced_drafts(h), h)


def spd_run_steps(h: int, count: int, want_log: bool = False):
    if want_log:
        log = (spd_step_result * count)()
        _check("spd_run_steps", lib().spd_run_steps(h, int(count), log), h)
        return [r.as_dict() for r in log]
    _check("spd_run_steps", lib().spd_run_steps(h, int(count), None), h)
    return None


def spd_sync(h: int) -> spd_step_result:
    r = spd_step_result()
    _check("spd_sync", lib().spd_sync(h, ct.byref(r)), h)
    return r


def spd_read_debug(h: int, what: int, count: int, dtype=np.float32) -> np.ndarray:
    out = np.empty(count, dtype=dtype)
    _check("spd_read_debug", lib().spd_read_debug(h, int(what), out.ctypes.data, out.nbytes), h)
    return out


def spd_read_kv(h: int, pdm: int, layer: int, pos0: int, count: int, n_kv: int, dh: int, bf16: bool):
    dt = np.uint16 if bf16 else np.float32
    k = np.empty((count, n_kv, dh), dtype=dt)
    v = np.empty((count, n_kv, dh), dtype=dt)
    _check("spd_read_kv", lib().spd_read_kv(h, int(pdm), int(layer), int(pos0), int(count), k.ctypes.data,
                                            v.ctypes.data), h)
    return k, v


def spd_set_debug(h: int, on: bool) -> None:
    _check("spd_set_debug", lib().spd_set_debug(h, 1 if on else 0), h)


def spd_set_kernel_timing(h: int, kernel: int, first_slot: int = 0) -> None:
    _check("spd_set_kernel_timing", lib().spd_set_kernel_timing(h, int(kernel), int(first_slot)), h)


def spd_kernel_timing(h: int):
    ms = ct.c_double(0.0)
    n = ct.c_int32(0)
    _check("spd_kernel_timing", lib().spd_kernel_timing(h, ct.byref(ms), ct.byref(n)), h)
    return ms.value, n.value


def spd_span_timing(h: int):
    """(stage_ms, pdm_ms, late_ms, steps), sums over the steps timed with SPD_K_SPANS."""
    st, pd, late = ct.c_double(0.0), ct.c_double(0.0), ct.c_double(0.0)
    n = ct.c_int32(0)
    _check("spd_span_timing", lib().spd_span_timing(h, ct.byref(st), ct.byref(pd), ct.byref(late), ct.byref(n)), h)
    return st.value, pd.value, late.value, n.value


def spd_set_graph(h: int, on: bool) -> None:
    _check("spd_set_graph", lib().spd_set_graph(h, 1 if on else 0), h)


def spd_set_step_kernel(h: int, mode: int, grid: int = 0, groups: int = -1) -> None:
    _check("spd_set_step_kernel", lib().spd_set_step_kernel(h, int(mode), int(grid), int(groups)), h)


def spd_step_plan_info(h: int) -> dict:
    info = (ct.c_int32 * 8)()
    _check("spd_step_plan_info", lib().spd_step_plan_info(h, info), h)
    return {"J": info[0], "clock_khz": info[1], "nkslots": info[2], "n": info[3],
            "stage_groups": info[4], "pdm_place": info[5]}


def spd_set_pdm_placement(h: int, place: int) -> None:
    _check("spd_set_pdm_placement", lib().spd_set_pdm_placement(h, place), h)


def spd_set_pdm_enabled(h: int, on: bool) -> None:
    _check("spd_set_pdm_enabled", lib().spd_set_pdm_enabled(h, 1 if on else 0), h)


def spd_set_graph_steps(h: int, steps: int) -> None:
    _check("spd_set_graph_steps", lib().spd_set_graph_steps(h, int(steps)), h)


def spd_set_pdm_schedule(h: int, post_step: bool) -> None:
    """False: the PDM reads pre-step features beside the stage compute; True: post-step, serial."""
    _check("spd_set_pdm_schedule", lib().spd_set_pdm_schedule(h, 1 if post_step else 0), h)


def spd_set_sampling(h: int, top_k: int, temperature: float = 1.0, uniforms=None) -> None:
    """uniforms: float[max_tokens, 3] (u_draft, u_accept, u_resample per position); top_k 0 = greedy."""
    if uniforms is None:
        _check("spd_set_sampling", lib().spd_set_sampling(h, int(top_k), float(temperature), None, 0), h)
        return
    u = np.ascontiguousarray(uniforms, dtype=np.float32)
    assert u.ndim == 2 and u.shape[1] == 3
    _check("spd_set_sampling", lib().spd_set_sampling(h, int(top_k), float(temperature),
                                                      u.ctypes.data_as(ct.POINTER(ct.c_float)), u.shape[0]), h)


def spd_probe_hbm_read(buf: int, nbytes: int, sink: int, reps: int, stream: int) -> float:
    """Mean milliseconds of one streaming read of nbytes at device address buf."""
    ms = ct.c_double(0.0)
    _check("spd_probe_hbm_read", lib().spd_probe_hbm_read(buf, nbytes, sink, reps, stream, ct.byref(ms)), 0)
    return ms.value


def spd_set_pdm_grid(h: int, wgs: int) -> None:
    _check("spd_set_pdm_grid", lib().spd_set_pdm_grid(h, wgs), h)


def spd_set_kernel_trace(h: int, on: bool) -> None:
    _check("spd_set_kernel_trace", lib().spd_set_kernel_trace(h, 1 if on else 0), h)


def spd_kernel_trace(h: int) -> dict:
    """The last traced step's launch spans (see SPD_DBG_KTRACE): `stage` [J][5][n][2] and `extra`
    [4][2] wall-clock stamps (start, end; both 0 where nothing ran)."""
    info = spd_step_plan_info(h)
    J, n, ns = info["J"], info["n"], info["nkslots"]
    raw = spd_read_debug(h, SPD_DBG_KTRACE, 2 * ns, np.uint64).reshape(ns, 2)
    return {"stage": raw[: 5 * J * n].reshape(J, 5, n, 2), "extra": raw[5 * J * n:], **info}


def decode_attention_workspace_bytes(nrows: int, n_kv_heads: int, head_dim: int, lens, chunk: int) -> int:
    """Workspace bytes spd_decode_attention needs (the formula its declaration states)."""
    splits = (max(int(x) for x in lens) + chunk - 1) // chunk
    rec = 4 * nrows * n_kv_heads * splits * 8 * (head_dim + 2)
    return (rec + 255) // 256 * 256 + 4 * nrows * n_kv_heads


def spd_decode_attention(q: int, kv: int, page_table: int, num_pages: int, lens, n_q_heads: int, n_kv_heads: int,
                         head_dim: int, dtype: int, chunk: int, out: int, workspace: int, ws_bytes: int,
                         stream: int) -> None:
    """Device pointers as ints; lens: host ints (one per row)."""
    ln = np.ascontiguousarray(lens, dtype=np.int32)
    _check("spd_decode_attention",
           lib().spd_decode_attention(q, kv, page_table, int(num_pages), ln.ctypes.data_as(ct.POINTER(ct.c_int32)),
                                      len(ln), int(n_q_heads), int(n_kv_heads), int(head_dim), int(dtype), int(chunk),
                                      out, workspace, int(ws_bytes), stream), None)


def spd_decode_attention_noalloc(q: int, kv: int, page_table: int, num_pages: int, lens, n_q_heads: int,
                                 n_kv_heads: int, head_dim: int, dtype: int, chunk: int, out: int, stream: int) -> None:
    """spd_decode_attention with the library's static scratch (no workspace, no allocation)."""
    ln = np.ascontiguousarray(lens, dtype=np.int32)
    _check("spd_decode_attention_noalloc",
           lib().spd_decode_attention_noalloc(q, kv, page_table, int(num_pages),
                                              ln.ctypes.data_as(ct.POINTER(ct.c_int32)), len(ln), int(n_q_heads),
                                              int(n_kv_heads), int(head_dim), int(dtype), int(chunk), out, stream),
           None)


def spd_destroy(h: int) -> None:
    lib().spd_destroy(h)
