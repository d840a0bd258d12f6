"""GPU parity of the ragged paged decode attention (spd_decode_attention: the step's attention split
code as a call of its own) against the oracle's attention, row by row, at the full-size head shapes.

Every row attends over its own number of keys (ragged, as the stages of a step do: t+1, t, t-1, ...)
through a shuffled page table. The cases reach what the step's own tests reach only in part: 4B/9B
heads (32 query / 8 KV heads of 128) at a 2048-token context in 128-key splits (17 splits), at 32776
tokens in 896-key splits (37 splits of 14 rounds, the benchmark's 32K split size) and in 528-key splits
(63 splits: the merge runs two batches), eight query heads per KV head, one query head per KV head,
fp32 KV at head_dim 64, and a single split. Keys, values and queries are N(0, 1) (bf16-rounded where
the cache is bf16), so the softmax is far from uniform. Tolerance: relative L2 1e-4 per row; the kernel
accumulates in fp32 over at most 32776 keys, whose rounding stays near 1e-6."""
import sys

import numpy as np
import pytest

import synth
from oracle import model as om

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

REL = 1e-4


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _case(hq, hkv, dh, bf16, T, nrows, seed):
    rng = np.random.default_rng(seed)
    num_pages = (T + 15) // 16 + 3
    K = rng.standard_normal((T, hkv, dh)).astype(np.float32)
    V = rng.standard_normal((T, hkv, dh)).astype(np.float32)
    if bf16:
        K = synth.bf16_bits_to_f32(synth.bf16_bits(K)).reshape(K.shape)
        V = synth.bf16_bits_to_f32(synth.bf16_bits(V)).reshape(V.shape)
    pt = rng.permutation(num_pages).astype(np.int32)
    pool = np.zeros((num_pages, 2, hkv, 16, dh), dtype=np.float32)
    for p in range(T):
        pool[pt[p // 16], 0, :, p % 16] = K[p]
        pool[pt[p // 16], 1, :, p % 16] = V[p]
    q = rng.standard_normal((nrows, hq, dh)).astype(np.float32)
    lens = np.array([T - i for i in range(nrows)], dtype=np.int32)
    return K, V, pt, pool, q, lens, num_pages


def _device(pool, bf16):
    if bf16:
        bits = synth.bf16_bits(pool).reshape(pool.shape)
        return torch.from_numpy(bits.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(pool).cuda()


@pytest.mark.parametrize("hq,hkv,dh,bf16,T,chunk,nrows", [
    (32, 8, 128, True, 2051, 128, 4),      # 4B/9B heads, 2048-token context, 17 splits
    (32, 8, 128, True, 32776, 896, 8),     # 32K context, the benchmark's split size: 37 splits of 14 rounds
    (32, 8, 128, True, 32776, 528, 8),     # 63 splits: two merge batches
    (16, 2, 128, True, 1000, 64, 3),       # eight query heads per KV head
    (8, 8, 64, True, 700, 48, 2),          # one query head per KV head, splits of 48 keys
    (4, 2, 64, False, 300, 32, 2),         # fp32 KV
    (32, 8, 128, True, 100, 128, 4),       # a single split
])
def test_decode_attention_matches_oracle(hq, hkv, dh, bf16, T, chunk, nrows):
    from paper_2605_30852_amd import binding as B
    _say(f"[decode attention {hq}/{hkv}x{dh} {'bf16' if bf16 else 'f32'} T={T} chunk={chunk} rows={nrows}]")
    K, V, pt, pool, q, lens, num_pages = _case(hq, hkv, dh, bf16, T, nrows, seed=T + chunk)
    kv_d = _device(pool, bf16)
    pt_d = torch.from_numpy(pt).cuda()
    q_d = torch.from_numpy(q).cuda()
    out_d = torch.full((nrows, hq, dh), float("nan"), dtype=torch.float32, device="cuda")
    wsb = B.decode_attention_workspace_bytes(nrows, hkv, dh, lens, chunk)
    ws = torch.empty(wsb + 256, dtype=torch.uint8, device="cuda")
    base = (ws.data_ptr() + 255) // 256 * 256
    stream = torch.cuda.current_stream().cuda_stream
    B.spd_decode_attention(q_d.data_ptr(), kv_d.data_ptr(), pt_d.data_ptr(), num_pages, lens, hq, hkv, dh,
                           B.SPD_BF16 if bf16 else B.SPD_F32, chunk, out_d.data_ptr(), base, wsb, stream)
    torch.cuda.synchronize()
    out = out_d.cpu().numpy()
    cache = om.LayerCache(hkv, dh, T)
    cache.k[:T] = K
    cache.v[:T] = V
    cache.n = T
    worst = 0.0
    for i in range(nrows):
        ref = om.attend(q[i].astype(np.float64), cache, int(lens[i]) - 1).reshape(hq, dh)
        err = float(np.linalg.norm(out[i] - ref) / np.linalg.norm(ref))
        worst = max(worst, err)
        assert err <= REL, f"row {i} (len {lens[i]}): rel L2 {err:.3e}"
    _say(f"  splits {(int(lens.max()) + chunk - 1) // chunk}, worst rel L2 {worst:.2e}")


def test_decode_attention_reuses_its_workspace(capfd):
    """Two calls in a row on one workspace (the second with fewer rows and keys) both match the oracle:
    the tickets are cleared at the start of every call."""
    from paper_2605_30852_amd import binding as B
    hq, hkv, dh = 32, 8, 128
    wsb = B.decode_attention_workspace_bytes(4, hkv, dh, [2051], 128)
    ws = torch.empty(wsb + 256, dtype=torch.uint8, device="cuda")
    ws.fill_(0xAB)  # the workspace holds whatever was there before
    base = (ws.data_ptr() + 255) // 256 * 256
    for T, nrows in ((2051, 4), (777, 2)):
        K, V, pt, pool, q, lens, num_pages = _case(hq, hkv, dh, True, T, nrows, seed=5 * T)
        kv_d, pt_d, q_d = _device(pool, True), torch.from_numpy(pt).cuda(), torch.from_numpy(q).cuda()
        out_d = torch.empty((nrows, hq, dh), dtype=torch.float32, device="cuda")
        B.spd_decode_attention(q_d.data_ptr(), kv_d.data_ptr(), pt_d.data_ptr(), num_pages, lens, hq, hkv, dh,
                               B.SPD_BF16, 128, out_d.data_ptr(), base, wsb, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        cache = om.LayerCache(hkv, dh, T)
        cache.k[:T], cache.v[:T], cache.n = K, V, T
        for i in range(nrows):
            ref = om.attend(q[i].astype(np.float64), cache, int(lens[i]) - 1).reshape(hq, dh)
            assert np.linalg.norm(out_d[i].cpu().numpy() - ref) <= REL * np.linalg.norm(ref)
