"""The C-ABI library loads, exports every entry point include/spd.h declares, and its host-only
calls (sizes, stage bounds, argument checks) behave without a GPU."""
import os
import re

import pytest

import synth
from paper_2605_30852_amd import binding as B
from paper_2605_30852_amd.engine import make_config

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    src = open(os.path.join(ROOT, "include", "spd.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(spd_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = B.lib()
    names = declared_symbols()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), f"{n} is declared in include/spd.h but not exported"
    assert set(names) == set(B.EXPORTS)


def test_status_strings():
    assert B.status_str(B.SPD_OK) == "SPD_OK"
    for s in (B.SPD_E_INVAL, B.SPD_E_STATE, B.SPD_E_CAPACITY, B.SPD_E_HIP):
        assert B.status_str(s).startswith("SPD_E_")


@pytest.mark.parametrize("L,n", [(36, 4), (36, 8), (36, 6), (4, 3), (4, 1), (5, 5)])
def test_stage_bounds_match_uniform_split(L, n):
    cfg = make_config(synth.TINY.with_(n_layers=L), 128, n=n)
    assert B.spd_stage_bounds(cfg) == [s * L // n for s in range(n + 1)]


def test_workspace_size_accounts_for_the_kv_pools():
    cfg = make_config(synth.B4, 2304)
    ws = B.spd_workspace_size(cfg)
    kv = 36 * (2304 // 16) * 2 * 8 * 16 * 128 * 2
    assert kv < ws < kv + 200 * 2**20
    # the long-context workload: 32k positions of bf16 KV for 36 layers + 2 PDM layers
    cfg5 = make_config(synth.B9_LONG, 32768 + 520)
    assert B.spd_workspace_size(cfg5) > 38 * 33288 * 4096


@pytest.mark.parametrize("field,value", [
    ("head_dim", 96), ("n_kv_heads", 3), ("n_stages", 0), ("n_stages", 9), ("pdm_layers", 0),
    ("page_size", 32), ("dtype", 7), ("d_model", 260), ("ffn_dim", 1001), ("max_tokens", 2),
    ("attn_chunk", 20), ("rms_eps", 0.0),
])
def test_invalid_configs_are_rejected(field, value):
    cfg = make_config(synth.TINY, 128)
    setattr(cfg, field, value)
    with pytest.raises(B.SPDError) as e:
        B.spd_workspace_size(cfg)
    assert e.value.status == B.SPD_E_INVAL


def test_attention_split_count_is_bounded():
    cfg = make_config(synth.TINY, 128, attn_chunk=16)  # 8 splits
    assert B.spd_workspace_size(cfg) > 0
    cfg = make_config(synth.TINY, 2048, attn_chunk=16)  # 128 splits > 64
    with pytest.raises(B.SPDError) as e:
        B.spd_workspace_size(cfg)
    assert e.value.status == B.SPD_E_INVAL
    # the default split size keeps the count at about 40 for any capacity
    assert B.spd_workspace_size(make_config(synth.B4, 1 << 20)) > 0


def test_n_larger_than_layers_rejected():
    cfg = make_config(synth.TINY, 128, n=5)  # tiny has 4 layers
    with pytest.raises(B.SPDError):
        B.spd_stage_bounds(cfg)


def test_init_rejects_null_arguments_before_touching_the_gpu():
    import ctypes as ct
    cfg = make_config(synth.TINY, 128)
    w = B.spd_weights()  # all NULL
    h = ct.c_void_p(0)
    st = B.lib().spd_init(ct.byref(cfg), ct.byref(w), ct.c_void_p(0), 0, ct.c_void_p(1), ct.c_void_p(2),
                          ct.byref(h))
    assert st == B.SPD_E_INVAL and h.value is None
    assert "NULL" in B.lib().spd_last_error(None).decode()
    # every call checks its handle
    assert B.lib().spd_step(None, None, None) == B.SPD_E_INVAL
    assert B.lib().spd_rollback(None, 0, 0) == B.SPD_E_INVAL
    assert B.lib().spd_prefill(None, None, 0, None) == B.SPD_E_INVAL


def test_pdm_vocab_config_rules():
    """The PDM's own head: pdm_vocab in [0, vocab], and an own head needs fused_head = 0 (the exit
    row and the PDM's row then stream different weights)."""
    sh = synth.TINY.with_(pdm_vocab=300)
    assert B.spd_workspace_size(make_config(sh, 128, fused_head=False)) > 0
    for cfg in (make_config(sh, 128, fused_head=True),
                make_config(synth.TINY.with_(pdm_vocab=synth.TINY.vocab + 1), 128, fused_head=False),
                make_config(synth.TINY.with_(pdm_vocab=-1), 128, fused_head=False)):
        with pytest.raises(B.SPDError) as e:
            B.spd_workspace_size(cfg)
        assert e.value.status == B.SPD_E_INVAL


def test_init_needs_the_own_head_pointers_before_touching_the_gpu():
    import ctypes as ct
    sh = synth.TINY.with_(pdm_vocab=300)
    cfg = make_config(sh, 128, fused_head=False)
    fake = 4096  # never dereferenced: the call fails on its argument checks first
    lw = B.spd_layer_weights(*([fake] * 9))
    layers = (B.spd_layer_weights * sh.n_layers)(*([lw] * sh.n_layers))
    pdm = (B.spd_layer_weights * sh.pdm_layers)(*([lw] * sh.pdm_layers))
    w = B.spd_weights()
    for f in ("embed", "final_norm", "lm_head", "pdm_in", "pdm_norm"):
        setattr(w, f, fake)
    w.layers = ct.cast(layers, ct.POINTER(B.spd_layer_weights))
    w.pdm_layers = ct.cast(pdm, ct.POINTER(B.spd_layer_weights))
    h = ct.c_void_p(0)
    st = B.lib().spd_init(ct.byref(cfg), ct.byref(w), ct.c_void_p(0), 0, ct.c_void_p(1), ct.c_void_p(2),
                          ct.byref(h))
    assert st == B.SPD_E_INVAL and h.value is None
    assert "pdm_lm_head" in B.lib().spd_last_error(None).decode()


def test_new_setters_check_their_handle():
    assert B.lib().spd_set_sampling(None, 8, 1.0, None, 0) == B.SPD_E_INVAL
    assert B.lib().spd_set_pdm_schedule(None, 1) == B.SPD_E_INVAL


def _attn_args(**kw):
    a = dict(q=256, kv=512, page_table=768, num_pages=8, lens=[20, 19], n_q_heads=8, n_kv_heads=2, head_dim=128,
             dtype=B.SPD_BF16, chunk=32, out=1024, workspace=4096, ws_bytes=1 << 20, stream=0)
    a.update(kw)
    return a


@pytest.mark.parametrize("field,value", [
    ("head_dim", 96), ("n_q_heads", 6), ("chunk", 24), ("chunk", 0), ("lens", [0]), ("lens", [129]),
    ("lens", [1] * 9), ("dtype", 5), ("workspace", 4100), ("q", 0), ("num_pages", 0),
])
def test_decode_attention_argument_checks(field, value):
    """spd_decode_attention checks its arguments on the host before it launches anything (the pointers
    here are never dereferenced): SPD_E_INVAL for bad shapes, lengths beyond the pages, a misaligned
    workspace or a NULL pointer."""
    with pytest.raises(B.SPDError) as e:
        B.spd_decode_attention(**_attn_args(**{field: value}))
    assert e.value.status == B.SPD_E_INVAL


def test_decode_attention_workspace_capacity():
    need = B.decode_attention_workspace_bytes(2, 2, 128, [20, 19], 32)
    with pytest.raises(B.SPDError) as e:
        B.spd_decode_attention(**_attn_args(ws_bytes=need - 1))
    assert e.value.status == B.SPD_E_CAPACITY
    assert str(need) in str(e.value)
    with pytest.raises(B.SPDError) as e:  # 69 splits of 16 keys: more than 64
        B.spd_decode_attention(**_attn_args(lens=[1100], chunk=16, num_pages=80, ws_bytes=1 << 30))
    assert e.value.status == B.SPD_E_INVAL
