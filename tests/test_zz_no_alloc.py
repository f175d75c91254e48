"""The allocation-free prefill scores (wnw_prefill_scores_static) against the allocating entry
point (wnw_prefill_scores), through the C ABI: the same kernels on the same inputs, so the
scores must agree bit for bit.  Two calls in a row, the second on a smaller input (fewer text
tokens, so the static statistics buffer still holds the first call's rows past the second's),
then a size beyond the buffer, which must be refused before any work is enqueued."""
import numpy as np
import pytest

from synth import gen
from synth.configs import Workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _scores_both_ways(w, seed_b=0):
    import torch
    from paper_2608_22704_amd import wnw as W
    from tests.wnw_harness import log, to_dev
    log(f"[case] static prefill scores: B={w.batch} L={w.layers} Hq={w.q_heads} Hkv={w.kv_heads} Ta={w.audio_len} "
        f"Tt={w.text_len}")
    B, L, H, D, Ta, Tt = w.batch, w.layers, w.kv_heads, w.head_dim, w.audio_len, w.text_len
    kd = torch.empty((B, L, H, w.total_len, D), dtype=torch.int16, device="cuda")
    qt = torch.empty((B, L, w.q_heads, Tt, D), dtype=torch.int16, device="cuda")
    for b in range(B):
        seq = gen.sequence(w, b)
        kd[b].copy_(to_dev(seq["k"]))
        q = np.stack([gen.text_queries(w, b, l, kv, seq["k"][l, kv]) for l in range(L) for kv in range(H)])
        qt[b].copy_(to_dev(q.reshape(L, w.q_heads, Tt, D)))
    cfg = W.make_config(B, L, w.q_heads, H, Ta, Tt, w.chunk_len, w.budget_bp)
    ref = torch.full((B, L, H, Ta), -1.0, dtype=torch.float32, device="cuda")
    got = torch.full((B, L, H, Ta), -2.0, dtype=torch.float32, device="cuda")
    ctx = W.wnw_init_cache(cfg, kd, kd)
    try:
        W.wnw_prefill_scores(ctx, qt, ref)
        stream = torch.cuda.Stream()
        W.wnw_prefill_scores_static(ctx, qt, got, stream)
        stream.synchronize()
    finally:
        W.wnw_destroy(ctx)
    return ref.cpu().numpy(), got.cpu().numpy()


def _w(name, seed, B, L, Hq, Hkv, Ta, Tt):
    n = L * Hkv
    return Workload(name, seed, B, L, Hq, Hkv, 128, Ta, Tt, 32, 2000, 1, 1, max(0, n // 2), n - 1 - max(0, n // 2))


def test_static_prefill_scores_match_the_allocating_entry_point():
    first = _w("static_prefill_a", 201, 2, 2, 8, 2, 777, 300)
    second = _w("static_prefill_b", 202, 1, 3, 12, 4, 250, 17)
    for w in (first, second):
        ref, got = _scores_both_ways(w)
        assert np.isfinite(ref).all() and (ref > 0).any()
        assert np.array_equal(ref.view(np.uint32), got.view(np.uint32)), f"{w.name}: scores differ"


def test_static_prefill_scores_refuse_sizes_beyond_the_buffer():
    import torch
    from paper_2608_22704_amd import wnw as W
    from tests.wnw_harness import log
    log("[case] static prefill scores: size beyond the static buffer")
    # 1 * 2 * 32 * 131 073 statistics rows > 8 388 608: refused before anything is read or launched
    cfg = W.make_config(1, 2, 32, 8, 16, 131073, 16, 2000)
    dummy = torch.zeros(16, dtype=torch.int16, device="cuda")
    ctx = W.lib.wnw_init_cache  # the binding's size checks would refuse the dummy first: call the C ABI
    import ctypes as C
    h = C.c_void_p()
    assert ctx(C.byref(cfg), dummy.data_ptr(), dummy.data_ptr(), None, C.byref(h)) == W.WNW_OK
    try:
        out = torch.zeros(16, dtype=torch.float32, device="cuda")
        st = W.lib.wnw_prefill_scores_static(h, dummy.data_ptr(), out.data_ptr(), None)
        assert st == W.WNW_ERR_UNSUPPORTED
        assert "static buffer" in W.wnw_last_error(h)
        torch.cuda.synchronize()
        assert not out.cpu().numpy().any()
    finally:
        W.lib.wnw_destroy(h)
