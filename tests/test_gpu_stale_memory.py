"""GPU parity when the memory the library has not written holds NaN: keys and values of a paged cache
past its length, and the whole workspace of an SPD handle before spd_init (every byte 0xFF, a NaN in
fp32 and bf16). Past the end of the last key split, round 0 of a split reads the page its lane's key
would fall in before the cache's length is known; those keys get zero probability, and their V rows
must enter the sums as zeros, not as the stale bytes, or a NaN there would turn a row's output into
NaN. Any other read of stale memory in a step shows up the same way."""
import sys

import numpy as np
import pytest

import synth
from oracle import model as om
from tests.lockstep import forced_table, run_lockstep

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

SEED = 53


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.mark.parametrize("hq,hkv,dh,bf16,T,chunk,nrows", [
    (32, 8, 128, True, 2051, 128, 4), (8, 8, 64, True, 700, 48, 2), (4, 2, 64, False, 300, 32, 3)])
def test_decode_attention_with_nan_past_the_length(hq, hkv, dh, bf16, T, chunk, nrows):
    from paper_2605_30852_amd import binding as B
    _say(f"[decode attention, NaN past the length: {hq}/{hkv}x{dh} T={T} chunk={chunk} rows={nrows}]")
    rng = np.random.default_rng(T + chunk)
    num_pages = (T + 15) // 16 + 3
    K = rng.standard_normal((T, hkv, dh)).astype(np.float32)
    V = rng.standard_normal((T, hkv, dh)).astype(np.float32)
    if bf16:
        K = synth.bf16_bits_to_f32(synth.bf16_bits(K)).reshape(K.shape)
        V = synth.bf16_bits_to_f32(synth.bf16_bits(V)).reshape(V.shape)
    pt = rng.permutation(num_pages).astype(np.int32)
    pool = np.full((num_pages, 2, hkv, 16, dh), np.nan, dtype=np.float32)
    for p in range(T):
        pool[pt[p // 16], 0, :, p % 16] = K[p]
        pool[pt[p // 16], 1, :, p % 16] = V[p]
    q = rng.standard_normal((nrows, hq, dh)).astype(np.float32)
    lens = np.array([T - 7 * i for i in range(nrows)], dtype=np.int32)
    if bf16:
        kv_d = torch.from_numpy(synth.bf16_bits(pool).reshape(pool.shape).view(np.int16)).cuda().view(torch.bfloat16)
    else:
        kv_d = torch.from_numpy(pool).cuda()
    pt_d, q_d = torch.from_numpy(pt).cuda(), torch.from_numpy(q).cuda()
    out_d = torch.empty((nrows, hq, dh), dtype=torch.float32, device="cuda")
    wsb = B.decode_attention_workspace_bytes(nrows, hkv, dh, lens, chunk)
    ws = torch.empty(wsb + 256, dtype=torch.uint8, device="cuda")
    base = (ws.data_ptr() + 255) // 256 * 256
    B.spd_decode_attention(q_d.data_ptr(), kv_d.data_ptr(), pt_d.data_ptr(), num_pages, lens, hq, hkv, dh,
                           B.SPD_BF16 if bf16 else B.SPD_F32, chunk, out_d.data_ptr(), base, wsb,
                           torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    out = out_d.cpu().numpy()
    cache = om.LayerCache(hkv, dh, T)
    cache.k[:T], cache.v[:T], cache.n = K, V, T
    for i in range(nrows):
        assert np.all(np.isfinite(out[i])), f"row {i} (len {lens[i]}): non-finite output"
        ref = om.attend(q[i].astype(np.float64), cache, int(lens[i]) - 1).reshape(hq, dh)
        err = float(np.linalg.norm(out[i] - ref) / np.linalg.norm(ref))
        assert err <= 1e-4, f"row {i} (len {lens[i]}): rel L2 {err:.3e}"


@pytest.mark.parametrize("shape,n,p,P", [(synth.TINY, 3, 0.6, 37), (synth.MID, 3, None, 29),
                                         (synth.MID, 2, 0.7, 21)])
def test_lockstep_from_a_nan_filled_workspace(shape, n, p, P):
    from paper_2605_30852_amd.engine import DeviceWeights, Engine
    _say(f"[NaN-filled workspace {shape.name} n={n} p={p} P={P}]")
    sh = shape.with_(n_stages=n)
    model = om.Model(sh, SEED)
    w = DeviceWeights(sh, SEED)
    prompt = synth.prompt(sh, SEED + n, P)
    draft_for = None
    if p is not None:
        ref = om.ar_greedy(model, prompt, 30)
        draft_for = forced_table(ref, synth.accept_mask(p, SEED + n, 400), len(prompt), sh.vocab).get
    eng = Engine(w, max_tokens=120, n=n, page_seed=17, ws_fill=0xFF)
    res = run_lockstep(eng, model, prompt, 20, draft_for=draft_for)
    eng.close()
    _say(f"  compared {res['steps']} steps, worst {res}")
    assert res["steps"] == 20, res
