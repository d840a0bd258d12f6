"""spd_decode_attention_noalloc, the decode attention for callers that cannot allocate, against
spd_decode_attention (the same kernel with a caller workspace): bit-identical outputs on two calls in a
row on one GPU, the second with fewer rows, fewer KV heads and fewer keys (the static scratch keeps the
first call's contents), and a clear capacity error beyond the scratch's 2048 split records."""
import sys

import numpy as np
import pytest

import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _inputs(hq, hkv, dh, T, nrows, seed):
    rng = np.random.default_rng(seed)
    num_pages = (T + 15) // 16 + 2
    pool = synth.bf16_bits(rng.standard_normal((num_pages, 2, hkv, 16, dh)).astype(np.float32))
    pt = rng.permutation(num_pages).astype(np.int32)
    q = rng.standard_normal((nrows, hq, dh)).astype(np.float32)
    lens = np.array([T - 3 * i for i in range(nrows)], dtype=np.int32)
    return (torch.from_numpy(pool.reshape(num_pages, 2, hkv, 16, dh).view(np.int16)).cuda(),
            torch.from_numpy(pt).cuda(), torch.from_numpy(q).cuda(), lens, num_pages)


def test_noalloc_matches_the_workspace_entry_point_on_two_calls():
    from paper_2605_30852_amd import binding as B
    stream = torch.cuda.current_stream().cuda_stream
    for call, (hq, hkv, dh, T, nrows, chunk) in enumerate([(32, 8, 128, 3000, 8, 128), (16, 4, 128, 900, 3, 64)]):
        _say(f"[no-alloc decode attention, call {call}: {hq}/{hkv}x{dh} T={T} rows={nrows} chunk={chunk}]")
        kv, pt, q, lens, num_pages = _inputs(hq, hkv, dh, T, nrows, seed=call)
        args = (q.data_ptr(), kv.data_ptr(), pt.data_ptr(), num_pages, lens, hq, hkv, dh, B.SPD_BF16, chunk)
        ref = torch.full((nrows, hq, dh), float("nan"), dtype=torch.float32, device="cuda")
        wsb = B.decode_attention_workspace_bytes(nrows, hkv, dh, lens, chunk)
        ws = torch.empty(wsb + 256, dtype=torch.uint8, device="cuda")
        B.spd_decode_attention(*args, ref.data_ptr(), (ws.data_ptr() + 255) // 256 * 256, wsb, stream)
        out = torch.full((nrows, hq, dh), float("nan"), dtype=torch.float32, device="cuda")
        B.spd_decode_attention_noalloc(*args, out.data_ptr(), stream)
        torch.cuda.synchronize()
        a, b = ref.cpu().numpy(), out.cpu().numpy()
        assert np.isfinite(a).all()
        assert np.array_equal(a, b), f"call {call}: outputs differ (max abs {np.nanmax(np.abs(a - b)):.3e})"


def test_noalloc_refuses_more_than_its_scratch_holds():
    from paper_2605_30852_amd import binding as B
    # 8 rows x 8 KV heads x 33 splits = 2112 split records > 2048; refused before anything runs
    lens = np.full(8, 33 * 64, dtype=np.int32)
    with pytest.raises(B.SPDError) as e:
        B.spd_decode_attention_noalloc(256, 512, 768, 33 * 4, lens, 32, 8, 128, B.SPD_BF16, 64, 1024, 0)
    assert e.value.status == B.SPD_E_CAPACITY
    assert "2048" in str(e.value)
