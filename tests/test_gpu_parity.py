"""GPU parity of the HIP decode step against the CPU oracle, through the C ABI.

Every test prints the case it runs before touching the GPU.
"""
import numpy as np
import pytest

from synth import configs, gen
from synth.configs import Workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from oracle import oracle as O
    O.build()


def _run(w, steps=None, head_mask_fn=None, **kw):
    from tests.wnw_harness import Lockstep, log
    log(f"[case] {w.name} B={w.batch} L={w.layers} Hq={w.q_heads} Hkv={w.kv_heads} Ta={w.audio_len} "
        f"Tt={w.text_len} chunk={w.chunk_len} budget={kw.get('budget_bp', w.budget_bp)} {kw}")
    h = Lockstep(w, **kw)
    try:
        n = w.steps if steps is None else steps
        for s in range(n):
            h.step(s, None if head_mask_fn is None else head_mask_fn(s, h))
            if s % 32 == 31:
                log(f"[step] {w.name}: {s + 1}/{n}, max out err {h.max_err:.3g}")
        log(f"[done] {w.name}: {n} steps, max out err {h.max_err:.3g}, max score rel {h.max_score_rel:.3g}, "
            f"excused flips {h.flips}")
        return h
    finally:
        h.close()


def test_tiny_single_layer():
    _run(configs.TINY)


def test_tiny_memcpy_recall_path():
    from paper_2608_22704_amd import wnw as W
    _run(configs.TINY.with_(steps=4), flags=W.WNW_F_RECALL_MEMCPY)


def test_qwen_shaped_all_steps():
    _run(configs.QWEN_10MIN)


def _sampled(n_heads):
    def fn(s, h):
        L, H = h.w.layers, h.w.kv_heads
        if s < 4:
            return np.ones((L, H), dtype=np.uint8)
        rng = np.random.default_rng(1000 + s)
        m = np.zeros(L * H, dtype=np.uint8)
        m[rng.choice(L * H, size=n_heads, replace=False)] = 1
        return m.reshape(L, H)
    return fn


def test_voxtral_shaped_all_steps_sampled_heads():
    _run(configs.VOXTRAL_10MIN, head_mask_fn=_sampled(16))


def _small(name, seed_id, L=2, Hq=8, Hkv=4, Ta=300, Tt=9, cl=32, budget=2000, steps=6, roles=None, B=2):
    n = L * Hkv
    a, t, f = roles if roles is not None else (max(1, n // 4), max(1, n // 2), n - max(1, n // 4) - max(1, n // 2))
    return Workload(name, seed_id, B, L, Hq, Hkv, 128, Ta, Tt, cl, budget, steps, a, t, f)


EDGE = [
    _small("g1_chunk7", 101, Hq=4, Hkv=4, cl=7),
    _small("g2_chunk50_ragged", 102, Hq=8, cl=50, Ta=517),
    _small("g6_chunk100", 103, Hq=12, Hkv=2, cl=100, Ta=1111, Tt=3),
    _small("g8_chunk256_long_tail", 104, Hq=16, Hkv=2, cl=256, Ta=1300, Tt=300),
    _small("g4_chunk1", 105, Hq=8, Hkv=2, cl=1, Ta=97, budget=2500),
    _small("no_text", 106, Tt=0),
    _small("budget_zero", 107, budget=0),
    _small("budget_full", 108, budget=10000),
    _small("audio_shorter_than_chunk", 109, Ta=20, cl=64, budget=5000),
    _small("text_only", 110, Ta=0, Tt=40),
    _small("all_tidal_but_one_anchor", 111, L=1, Hkv=4, Hq=12, roles=(1, 3, 0)),
    _small("anchors_only", 112, L=1, Hkv=4, Hq=8, roles=(4, 0, 0)),
    _small("batch3_tile_ragged", 113, B=3, Ta=777, Tt=1, cl=37, budget=3000, steps=9),
]


@pytest.mark.parametrize("w", EDGE, ids=[w.name for w in EDGE])
def test_edge_shapes(w):
    _run(w)


def test_budget_full_is_full_attention():
    """At 100 % budget every head must equal plain attention over its whole cache."""
    import torch
    from tests.wnw_harness import Lockstep, log
    w = _small("full_budget_sdpa", 120, budget=10000, steps=2)
    log("[case] full budget vs SDPA")
    h = Lockstep(w)
    try:
        out, _, _, _ = h.gpu_step(0)
        k = torch.from_numpy(gen.bf16_to_f32(h.ok_).astype(np.float64))
        v = torch.from_numpy(gen.bf16_to_f32(h.ov_).astype(np.float64))
        q = torch.from_numpy(gen.bf16_to_f32(h.q[0]).astype(np.float64))
        g = w.group
        ref = torch.nn.functional.scaled_dot_product_attention(
            q.unsqueeze(-2), k.repeat_interleave(g, dim=2), v.repeat_interleave(g, dim=2)).squeeze(-2)
        assert np.abs(out - ref.numpy()).max() <= 2e-2
    finally:
        h.close()


def test_recall_bytes_identical_to_host_copy_and_cache():
    from tests.wnw_harness import Lockstep, log
    w = configs.TINY.with_(steps=1)
    log("[case] recall byte identity, tiny workload")
    h = Lockstep(w)
    try:
        _, _, sel, _ = h.gpu_step(0)
        W = h.W
        nbytes = h.geo["chunk_bytes"]
        kd, vd = h.ok_[0], h.ov_[0]                       # [L][H][T][D] of sequence 0
        tidal = [(l, kv) for l in range(w.layers) for kv in range(w.kv_heads) if h.roles[l, kv] == 1]
        assert sel.shape[1] == h.k and h.k > 0
        for c in sel[0]:
            dev = np.empty(nbytes // 2, dtype=np.uint16)
            hst = np.empty(nbytes // 2, dtype=np.uint16)
            W.wnw_debug_read_slot(h.ctx, 0, int(c), dev, nbytes)
            W.wnw_debug_read_host_chunk(h.ctx, 0, int(c), hst, nbytes)
            assert np.array_equal(dev, hst)
            comp_max = nbytes // 2 // (len(tidal) * 2 * 128)
            blk = dev.reshape(len(tidal), 2, comp_max, 128)
            for ti, (l, kv) in enumerate(tidal):
                keep = h.oracle.keep_mask(0, l, kv)
                c0, c1 = int(c) * w.chunk_len, min((int(c) + 1) * w.chunk_len, w.audio_len)
                rows = [t for t in range(c0, c1) if not keep[t]]
                assert np.array_equal(blk[ti, 0, : len(rows)], kd[l, kv, rows])
                assert np.array_equal(blk[ti, 1, : len(rows)], vd[l, kv, rows])
                assert not blk[ti, :, len(rows):].any()
        with pytest.raises(W.WnwError):
            notres = [c for c in range(h.nc) if c not in set(sel[0].tolist())][0]
            W.wnw_debug_read_slot(h.ctx, 0, notres, np.empty(nbytes // 2, dtype=np.uint16), nbytes)
    finally:
        h.close()


def test_two_runs_bit_identical():
    from tests.wnw_harness import Lockstep, log
    w = _small("determinism", 130, steps=5)
    log("[case] determinism")
    outs = []
    for _ in range(2):
        h = Lockstep(w)
        try:
            outs.append([h.gpu_step(s) for s in range(w.steps)])
        finally:
            h.close()
    for a, b in zip(*outs):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)


def test_selection_override_and_call_order():
    import torch
    from tests.wnw_harness import Lockstep, log, to_dev
    w = _small("override", 140, steps=5, cl=16, Ta=160)
    log("[case] override and call order")
    h = Lockstep(w)
    W = h.W
    try:
        k = h.k
        forced = np.full((w.batch, k), -1, dtype=np.int32)
        forced[:, 0] = 3
        if k > 1:
            forced[:, 1] = 7
        fd = torch.from_numpy(forced).cuda()
        W.wnw_set_selection_override(h.ctx, fd)
        for s in range(3):
            out, sc, sel, res = h.gpu_step(s)
            r = h.oracle.step(h.q[s], forced=forced)
            assert (res == r["resident"]).all()
            assert np.abs(out - r["out"]).max() <= 2e-2
            assert sorted(x for x in sel[0] if x >= 0) == sorted(x for x in forced[0] if x >= 0)
        W.wnw_set_selection_override(h.ctx, None)
        with pytest.raises(W.WnwError) as e:
            W.wnw_set_roles(h.ctx, h.roles, h.prefill)
        assert e.value.status == W.WNW_ERR_STATE
        with pytest.raises(W.WnwError) as e:
            W.wnw_decode_step(h.ctx, None, h.out)
        assert e.value.status == W.WNW_ERR_INVALID
    finally:
        h.close()
    kd = torch.zeros((1, 1, 2, 40, 128), dtype=torch.int16, device="cuda")
    cfg = W.make_config(1, 1, 2, 2, 32, 8, 8, 2000)
    ctx = W.wnw_init_cache(cfg, kd, kd)
    try:
        with pytest.raises(W.WnwError) as e:
            W.wnw_decode_step(ctx, kd, torch.zeros(256, device="cuda"))
        assert e.value.status == W.WNW_ERR_STATE
    finally:
        W.wnw_destroy(ctx)


def test_timing_stats():
    from paper_2608_22704_amd import wnw as W
    from tests.wnw_harness import Lockstep, log
    w = _small("timing", 150, steps=4)
    log("[case] timing statistics")
    h = Lockstep(w, flags=W.WNW_F_TIMING)
    try:
        for s in range(w.steps):
            h.gpu_step(s)
        st = W.wnw_get_stats(h.ctx)
        assert st["steps"] == w.steps and st["timed_steps"] == w.steps
        assert st["t_anchor_ms"] > 0 and st["t_tidal_fixed_ms"] > 0 and st["t_step_ms"] > 0
        assert 0 < st["r_gpu"] <= st["r_gpu_cpu"] <= 1.0 + 1e-9
        assert st["anchor_bytes"] == w.batch * w.n_anchor * w.total_len * 512
    finally:
        h.close()


def test_resident_slots_match_host_copies_over_steps():
    """After every step, every resident chunk's device slot (copied or revived) is byte-identical
    to its host complement; revivals happen on this workload."""
    from tests.wnw_harness import Lockstep, log
    w = _small("slots_over_steps", 160, L=2, Hq=8, Hkv=4, Ta=480, Tt=5, cl=16, budget=2000, steps=24)
    log("[case] resident slots vs host copies over 24 steps")
    h = Lockstep(w)
    W = h.W
    try:
        nbytes = h.geo["chunk_bytes"]
        for s in range(w.steps):
            _, _, _, res = h.step(s)
            for b in range(w.batch):
                for c in np.nonzero(res[b])[0]:
                    dev = np.empty(nbytes // 2, dtype=np.uint16)
                    hst = np.empty(nbytes // 2, dtype=np.uint16)
                    W.wnw_debug_read_slot(h.ctx, b, int(c), dev, nbytes)
                    W.wnw_debug_read_host_chunk(h.ctx, b, int(c), hst, nbytes)
                    assert np.array_equal(dev, hst), f"step {s} seq {b} chunk {c}"
        st = W.wnw_get_stats(h.ctx)
        log(f"[done] recalled {st['recalled_chunks']} revived {st['revived_chunks']} dropped {st['dropped_chunks']}")
        assert st["revived_chunks"] > 0
    finally:
        h.close()


# ---- full-size batched and long-form workloads: every sequence runs on the GPU; the oracle
# checks the sequences, heads and steps it can afford (sampled outputs at full size).

def test_voxtral_b16_full_size_sampled():
    """Batch 16 of the 15k-audio cache, 256 steps: per-sequence selection, residency, scores
    and outputs of sequences 0 and 9 against the oracle at every step, sampled heads."""
    _run(configs.VOXTRAL_10MIN_B16, head_mask_fn=_sampled(8), seqs=[0, 9])


@pytest.mark.parametrize("w", [configs.VOXTRAL_60MIN_B4_20, configs.VOXTRAL_60MIN_B4_10],
                         ids=["budget20", "budget10"])
def test_voxtral_60min_b4_full_size_sampled(w):
    """Batch 4 of 90k audio + 1k text positions, chunk 128: the first 64 of 512 steps, sequence 2
    against the oracle with sampled heads (the oracle's anchor pass alone is ~2 G multiply-adds
    per step per sequence); the slot pool (3 k slots) is reused many times over."""
    h = _run(w, steps=64, head_mask_fn=_sampled(6), seqs=[2])
    assert h.recalled_total > h.geo["n_slots"], "the slot pool was not wrapped"


@pytest.mark.parametrize("w", [configs.VOXTRAL_60MIN_B4_20, configs.VOXTRAL_60MIN_B4_10],
                         ids=["budget20", "budget10"])
def test_voxtral_60min_b4_benchmark_mode_full_size_sampled(w):
    """The 60-minute batch-4 caches in the benchmark's launch configuration (the paper's
    next-step timing, copy-engine recall from the pinned complement): 64 of 512 steps, sequence
    1 against the oracle at every step (scores, selection, residency, anchor outputs, sampled
    non-anchor heads), no slot ever exhausted, and more complements copied than there are slots
    (4 k per sequence), so freed slots are refilled many times."""
    from paper_2608_22704_amd import wnw as W
    h = _run(w, steps=64, head_mask_fn=_sampled(6), seqs=[1], flags=W.WNW_F_SELECT_NEXT_STEP | W.WNW_F_RECALL_MEMCPY)
    assert h.recalled_total > h.geo["n_slots"] * w.batch, "the slot pool was not wrapped"


@pytest.mark.parametrize("nxt", [0, 1], ids=["same_step", "next_step"])
def test_selection_state_above_64k_of_shared_memory(nxt):
    """1 250 segments of 16 positions and k = 250 (up to 1 000 slots): the select kernel's
    state needs ~103-109 KB of shared memory, above the 64 KB of a default launch."""
    from paper_2608_22704_amd import wnw as W
    w = _small("select_lds_109k", 170, L=1, Hq=8, Hkv=4, Ta=20000, Tt=16, cl=16, budget=2000, steps=6, roles=(1, 2, 1),
               B=1)
    _run(w, flags=W.WNW_F_SELECT_NEXT_STEP | W.WNW_F_RECALL_MEMCPY if nxt else 0)


def test_pinned_allocation_failure_is_reported():
    """Set-up with pinned memory refused (WNW_TEST_PINNED_LIMIT): wnw_set_roles returns
    WNW_ERR_OOM, the context is failed (later steps return WNW_ERR_STATE) and destroys cleanly;
    a context made afterwards works."""
    import os
    import torch
    from paper_2608_22704_amd import wnw as W
    from tests.wnw_harness import log, to_dev
    w = configs.TINY
    log("[case] pinned allocation failure")
    seq = gen.sequence(w, 0)
    kd, vd = to_dev(seq["k"][None]), to_dev(seq["v"][None])
    cfg = W.make_config(1, w.layers, w.q_heads, w.kv_heads, w.audio_len, w.text_len, w.chunk_len, w.budget_bp)
    ctx = W.wnw_init_cache(cfg, kd, vd)
    os.environ["WNW_TEST_PINNED_LIMIT"] = "4096"
    try:
        with pytest.raises(W.WnwError) as e:
            W.wnw_set_roles(ctx, gen.roles(w), seq["prefill"][None])
        assert e.value.status == W.WNW_ERR_OOM and "WNW_TEST_PINNED_LIMIT" in str(e.value)
    finally:
        del os.environ["WNW_TEST_PINNED_LIMIT"]
    try:
        out = torch.empty((1, w.layers, w.q_heads, w.head_dim), dtype=torch.float32, device="cuda")
        with pytest.raises(W.WnwError) as e:
            W.wnw_decode_step(ctx, to_dev(seq["q"][0][None]), out)
        assert e.value.status == W.WNW_ERR_STATE
    finally:
        W.wnw_destroy(ctx)
    ctx = W.wnw_init_cache(cfg, kd, vd)
    try:
        W.wnw_set_roles(ctx, gen.roles(w), seq["prefill"][None])
        W.wnw_decode_step(ctx, to_dev(seq["q"][0][None]), out)
        torch.cuda.synchronize()
        assert np.isfinite(out.cpu().numpy()).all()
    finally:
        W.wnw_destroy(ctx)


def test_headline_config_full_size_sampled():
    """The benchmark's launch configuration at full size: the 15k-audio cache with the paper's
    next-step timing and copy-engine recall, all 256 steps; selection, residency, scores and
    anchor outputs at every step, sampled non-anchor heads."""
    from paper_2608_22704_amd import wnw as W
    _run(configs.VOXTRAL_10MIN, head_mask_fn=_sampled(8),
         flags=W.WNW_F_SELECT_NEXT_STEP | W.WNW_F_RECALL_MEMCPY)


def test_b16_next_step_copy_engines_full_size_sampled():
    """Batch 16 of the 15k-audio cache with next-step timing and copy-engine recall (every
    sequence's new complements in one step's transfers): sequences 3 and 12 against the oracle
    for 48 steps, sampled heads."""
    from paper_2608_22704_amd import wnw as W
    _run(configs.VOXTRAL_10MIN_B16, steps=48, head_mask_fn=_sampled(6), seqs=[3, 12],
         flags=W.WNW_F_SELECT_NEXT_STEP | W.WNW_F_RECALL_MEMCPY)


# ---- next-step selection timing: the tidal heads of step s attend over the resident set left
# by step s-1; the oracle runs the same timing (its next_step mode).

def _next(extra=0):
    from paper_2608_22704_amd import wnw as W
    return W.WNW_F_SELECT_NEXT_STEP | extra


def test_next_step_tiny():
    _run(configs.TINY.with_(steps=6), flags=_next())


@pytest.mark.parametrize("w", EDGE, ids=[w.name for w in EDGE])
def test_next_step_edge_shapes(w):
    _run(w, flags=_next())


def test_next_step_memcpy_recall_path():
    from paper_2608_22704_amd import wnw as W
    _run(_small("next_memcpy", 170, L=2, Hq=8, Hkv=4, Ta=480, Tt=5, cl=16, steps=12),
         flags=_next(W.WNW_F_RECALL_MEMCPY))


def test_wnw_log_trace(capfd, monkeypatch):
    """WNW_LOG=1 at context creation: one trace line per step on stderr, naming the timing, the
    recall path and where the selection ran (small recalls: inside the tidal launch)."""
    from paper_2608_22704_amd import wnw as W
    monkeypatch.setenv("WNW_LOG", "1")
    _run(_small("log_trace", 117, steps=3), flags=_next(W.WNW_F_RECALL_MEMCPY))
    err = capfd.readouterr().err
    lines = [l for l in err.splitlines() if l.startswith("[wnw] step ")]
    assert len(lines) == 3, err[-2000:]
    assert all("next-step timing, copy-engine recall" in l and "selection inside the tidal launch" in l for l in lines), lines


@pytest.mark.parametrize("timed", [0, 1], ids=["plain", "timing_events"])
@pytest.mark.parametrize("nxt", [0, 1], ids=["same_step", "next_step"])
def test_copy_engine_paths_without_audio(nxt, timed):
    """No audio, so no chunk to select: with copy-engine recall no selection runs and no tag is
    published, and neither the step nor the library's recall thread may wait for one (both
    timings, with and without timing events, whose recall interval is then empty)."""
    from paper_2608_22704_amd import wnw as W
    flags = W.WNW_F_RECALL_MEMCPY | (W.WNW_F_SELECT_NEXT_STEP if nxt else 0) | (W.WNW_F_TIMING if timed else 0)
    h = _run(_small("memcpy_text_only", 116, Ta=0, Tt=40), flags=flags)
    assert h.final_stats["recalled_chunks"] == 0 and h.final_stats["selections_in_tidal"] == 0


@pytest.mark.parametrize("w", EDGE, ids=[w.name for w in EDGE])
def test_next_step_memcpy_edge_shapes(w):
    """Copy-engine recall with next-step timing on the edge shapes: their recalls are small, so
    every step's chunk-mass merge and selection run inside the tidal launch (group sizes 1 to 8,
    ragged tiles, no text, no audio, anchors only), against the oracle step by step."""
    from paper_2608_22704_amd import wnw as W
    h = _run(w, flags=_next(W.WNW_F_RECALL_MEMCPY))
    if w.audio_len > 0:   # chunks to select
        assert h.final_stats["selections_in_tidal"] == w.steps, h.final_stats["selections_in_tidal"]


@pytest.mark.parametrize("timing", ["same", "next"])
def test_slot_rows_pointer_path(timing):
    """Slot groups read through per-row pointers (forced by a zero slot offset limit; the default
    takes buffer offsets below 4 GB of slots) match the oracle and, bit for bit, the offset path
    on the same steps."""
    from paper_2608_22704_amd import wnw as W
    from tests.wnw_harness import Lockstep, log
    w = _small(f"slot_ptr_{timing}", 190 if timing == "same" else 191, L=2, Hq=8, Hkv=4, Ta=480, Tt=5, cl=16,
               steps=10)
    flags = _next() if timing == "next" else 0
    log(f"[case] slot rows through pointers vs buffer offsets, {timing}-step timing")
    h, h2 = Lockstep(w, flags=flags), Lockstep(w, flags=flags)
    try:
        with pytest.raises(W.WnwError) as e:
            W.wnw_debug_set_slot_offset_limit(h.ctx, -1)
        assert e.value.status == W.WNW_ERR_INVALID
        W.wnw_debug_set_slot_offset_limit(h.ctx, 0)
        for s in range(w.steps):
            h.step(s)
            ref = h2.gpu_step(s)[0]
            assert np.array_equal(h.out.cpu().numpy(), ref), f"step {s}: pointer and offset paths differ"
    finally:
        h.close()
        h2.close()


@pytest.mark.parametrize("timing", ["same", "next"])
def test_out_bf16(timing):
    """WNW_F_OUT_BF16: every step's bf16 output is, bit for bit, the fp32 output of a context
    without the flag rounded to nearest (ties to even), and the fp32 run matches the oracle."""
    import torch
    from paper_2608_22704_amd import wnw as W
    from tests.wnw_harness import Lockstep, log
    w = _small(f"out_bf16_{timing}", 192 if timing == "same" else 193, L=2, Hq=8, Hkv=4, Ta=480, Tt=5, cl=16,
               steps=8)
    flags = _next(W.WNW_F_RECALL_MEMCPY) if timing == "next" else 0
    log(f"[case] bf16 output, {timing}-step timing")
    h, h2 = Lockstep(w, flags=flags), Lockstep(w, flags=flags | W.WNW_F_OUT_BF16)
    try:
        h2.out = torch.empty(h.out.shape, dtype=torch.int16, device="cuda")
        for s in range(w.steps):
            h.step(s)
            got = h2.gpu_step(s)[0].view(np.uint16)
            want = gen.f32_to_bf16(h.out.cpu().numpy())
            assert np.array_equal(got, want), f"step {s}: bf16 output is not the rounded fp32 output"
    finally:
        h.close()
        h2.close()


def test_next_step_qwen_shaped_all_steps():
    _run(configs.QWEN_10MIN, flags=_next())


def test_next_step_voxtral_shaped_sampled_heads():
    _run(configs.VOXTRAL_10MIN.with_(steps=64), head_mask_fn=_sampled(16), flags=_next())


@pytest.mark.parametrize("memcpy", [False, True], ids=["zero_copy", "memcpy"])
def test_next_step_slots_over_steps(memcpy):
    """Next-step timing: after every step the chunks holding a slot are the resident set that the
    following step attends to, and each slot (recalled during the step, or revived) is
    byte-identical to the chunk's host complement."""
    from paper_2608_22704_amd import wnw as W
    from tests.wnw_harness import Lockstep, log
    w = _small("next_slots_over_steps", 161, L=2, Hq=8, Hkv=4, Ta=480, Tt=5, cl=16, budget=2000, steps=24)
    log(f"[case] next-step slots vs host copies over 24 steps, memcpy={memcpy}")
    h = Lockstep(w, flags=_next(W.WNW_F_RECALL_MEMCPY if memcpy else 0))
    try:
        nbytes = h.geo["chunk_bytes"]
        assert h.geo["n_slots"] == 4 * h.k
        held_before = None
        for s in range(w.steps):
            _, _, _, res = h.step(s)
            if held_before is not None:
                assert np.array_equal(res, held_before), f"step {s}: attended set is not the previous resident set"
            held = np.zeros_like(res)
            for b in range(w.batch):
                for c in range(h.nc):
                    dev = np.empty(nbytes // 2, dtype=np.uint16)
                    try:
                        W.wnw_debug_read_slot(h.ctx, b, c, dev, nbytes)
                    except W.WnwError:
                        continue
                    held[b, c] = 1
                    hst = np.empty(nbytes // 2, dtype=np.uint16)
                    W.wnw_debug_read_host_chunk(h.ctx, b, c, hst, nbytes)
                    assert np.array_equal(dev, hst), f"step {s} seq {b} chunk {c}"
            held_before = held
        st = W.wnw_get_stats(h.ctx)
        log(f"[done] recalled {st['recalled_chunks']} revived {st['revived_chunks']} dropped {st['dropped_chunks']}")
        assert st["revived_chunks"] > 0
    finally:
        h.close()


def test_next_step_two_runs_bit_identical():
    from tests.wnw_harness import Lockstep, log
    w = _small("determinism_next", 131, steps=5)
    log("[case] determinism, next-step timing")
    outs = []
    for _ in range(2):
        h = Lockstep(w, flags=_next())
        try:
            outs.append([h.gpu_step(s) for s in range(w.steps)])
        finally:
            h.close()
    for a, b in zip(*outs):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)


# ---- overlapping chunks: a chunk is two consecutive half-length segments and a chunk starts at
# every segment; selection per chunk, residency and recall per segment (the oracle's chunk_span 2).

def _ovl(extra=0):
    from paper_2608_22704_amd import wnw as W
    return W.WNW_F_OVERLAP_CHUNKS | extra


EDGE_OVL = [
    _small("ovl_g1_chunk8", 201, Hq=4, Hkv=4, cl=8),
    _small("ovl_g2_chunk50_ragged", 202, Hq=8, cl=50, Ta=517),
    _small("ovl_g6_chunk100", 203, Hq=12, Hkv=2, cl=100, Ta=1111, Tt=3),
    _small("ovl_g8_chunk512_long_tail", 204, Hq=16, Hkv=2, cl=512, Ta=1300, Tt=300, budget=5000),
    _small("ovl_g4_chunk2", 205, Hq=8, Hkv=2, cl=2, Ta=97, budget=2500),
    _small("ovl_no_text", 206, Tt=0),
    _small("ovl_budget_zero", 207, budget=0),
    _small("ovl_budget_full", 208, budget=10000),
    _small("ovl_audio_shorter_than_segment", 209, Ta=20, cl=64, budget=5000),
    _small("ovl_text_only", 210, Ta=0, Tt=40),
    _small("ovl_all_tidal_but_one_anchor", 211, L=1, Hkv=4, Hq=12, roles=(1, 3, 0)),
    _small("ovl_batch3_tile_ragged", 213, B=3, Ta=777, Tt=1, cl=38, budget=3000, steps=9),
]


@pytest.mark.parametrize("w", EDGE_OVL, ids=[w.name for w in EDGE_OVL])
def test_overlap_edge_shapes(w):
    _run(w, flags=_ovl())


@pytest.mark.parametrize("w", EDGE_OVL, ids=[w.name for w in EDGE_OVL])
def test_overlap_next_step_edge_shapes(w):
    _run(w, flags=_ovl(_next()))


@pytest.mark.parametrize("w", EDGE_OVL, ids=[w.name for w in EDGE_OVL])
def test_overlap_next_step_memcpy_edge_shapes(w):
    """Overlapping chunks (two segments each) with copy-engine recall and next-step timing: the
    selection inside the tidal launch scores segment pairs, against the oracle step by step."""
    from paper_2608_22704_amd import wnw as W
    h = _run(w, flags=_ovl(_next(W.WNW_F_RECALL_MEMCPY)))
    if w.audio_len > 0:
        assert h.final_stats["selections_in_tidal"] == w.steps, h.final_stats["selections_in_tidal"]


def test_overlap_two_segments_one_chunk():
    """Two segments make one chunk, which top-k 1 selects at every step."""
    _run(_small("ovl_two_segments", 214, Ta=60, cl=64, budget=2000), flags=_ovl(), top_k=1)


def test_overlap_memcpy_recall_paths():
    from paper_2608_22704_amd import wnw as W
    w = _small("ovl_memcpy", 215, L=2, Hq=8, Hkv=4, Ta=480, Tt=5, cl=32, steps=10)
    _run(w, flags=_ovl(W.WNW_F_RECALL_MEMCPY))
    _run(w, flags=_ovl(_next(W.WNW_F_RECALL_MEMCPY)))


def test_overlap_qwen_shaped_all_steps():
    _run(configs.QWEN_10MIN, flags=_ovl(_next()))


def test_overlap_voxtral_shaped_sampled_heads():
    _run(configs.VOXTRAL_10MIN.with_(steps=64), head_mask_fn=_sampled(16), flags=_ovl(_next()))


@pytest.mark.parametrize("nxt", [False, True], ids=["same_step", "next_step"])
def test_overlap_slots_over_steps(nxt):
    """Every segment that holds a slot after a step is byte-identical to its host complement, the
    segments held are those the following step attends to (next-step timing), and segments are
    revived."""
    from paper_2608_22704_amd import wnw as W
    from tests.wnw_harness import Lockstep, log
    w = _small("ovl_slots_over_steps", 216, L=2, Hq=8, Hkv=4, Ta=480, Tt=5, cl=32, budget=2000, steps=24)
    log(f"[case] overlapping chunks, slots vs host copies over 24 steps, next_step={nxt}")
    h = Lockstep(w, flags=_ovl(_next() if nxt else 0))
    try:
        nbytes = h.geo["chunk_bytes"]
        assert h.nseg == h.nc + 1
        assert h.geo["n_slots"] == min(h.nseg, 4 * 2 * h.k)
        held_before = None
        for s in range(w.steps):
            _, _, _, res = h.step(s)
            if nxt and held_before is not None:
                assert np.array_equal(res, held_before), f"step {s}: attended set is not the previous resident set"
            held = np.zeros_like(res)
            for b in range(w.batch):
                for c in range(h.nseg):
                    dev = np.empty(nbytes // 2, dtype=np.uint16)
                    try:
                        W.wnw_debug_read_slot(h.ctx, b, c, dev, nbytes)
                    except W.WnwError:
                        continue
                    held[b, c] = 1
                    hst = np.empty(nbytes // 2, dtype=np.uint16)
                    W.wnw_debug_read_host_chunk(h.ctx, b, c, hst, nbytes)
                    assert np.array_equal(dev, hst), f"step {s} seq {b} segment {c}"
            if not nxt:
                assert np.array_equal(held, res), f"step {s}: held slots are not the resident segments"
            held_before = held
        st = W.wnw_get_stats(h.ctx)
        log(f"[done] recalled {st['recalled_chunks']} revived {st['revived_chunks']} dropped {st['dropped_chunks']}")
        assert st["revived_chunks"] > 0
    finally:
        h.close()


# ---- per-head retention (Eq. 1): retention = min(importance * lambda, 1) per tidal/fixed head;
# static tiers, complements and slots are ragged by head.

def _imp(w, seed, zeros=(), ones=()):
    rng = np.random.default_rng(seed)
    imp = rng.random((w.layers, w.kv_heads), dtype=np.float32)
    for lh in zeros:
        imp[lh] = 0.0
    for lh in ones:
        imp[lh] = 1.0
    return imp


RET = [
    (_small("ret_mixed", 301, L=2, Hq=8, Hkv=4, Ta=300, cl=32), 1.0, ((0, 1),), ((1, 2),)),
    (_small("ret_g8_chunk256", 302, Hq=16, Hkv=2, L=3, cl=256, Ta=1300, Tt=300), 1.0, ((1, 0),), ()),
    (_small("ret_g1_chunk7", 303, Hq=4, Hkv=4, cl=7), 0.6, (), ((0, 3),)),
    (_small("ret_chunk1", 304, Hq=8, Hkv=2, L=3, cl=1, Ta=97), 1.0, (), ()),
    (_small("ret_scale_up", 305, L=2, Hq=12, Hkv=4, Ta=517, cl=50, Tt=3), 2.5, (), ()),
    (_small("ret_batch3", 306, B=3, Ta=777, Tt=1, cl=37, steps=9), 0.4, ((0, 0), (1, 1)), ()),
]


def _ret_run(w, lam, zeros, ones, seed, **kw):
    return _run(w, importance=_imp(w, seed, zeros, ones), lam=lam, **kw)


@pytest.mark.parametrize("case", RET, ids=[c[0].name for c in RET])
def test_retention_edge_shapes(case):
    w, lam, zeros, ones = case
    _ret_run(w, lam, zeros, ones, w.seed_id)


@pytest.mark.parametrize("case", RET, ids=[c[0].name for c in RET])
def test_retention_next_step_edge_shapes(case):
    w, lam, zeros, ones = case
    _ret_run(w, lam, zeros, ones, w.seed_id, flags=_next())


def test_retention_overlap_and_memcpy():
    from paper_2608_22704_amd import wnw as W
    w = _small("ret_ovl", 307, L=2, Hq=8, Hkv=4, Ta=480, Tt=5, cl=32, steps=10)
    _ret_run(w, 0.7, ((0, 1),), ((1, 1),), 307, flags=_ovl(_next()))
    _ret_run(w, 0.7, ((0, 1),), ((1, 1),), 307, flags=_ovl(W.WNW_F_RECALL_MEMCPY))
    _ret_run(w, 0.7, ((0, 1),), ((1, 1),), 307, flags=_next(W.WNW_F_RECALL_MEMCPY))


def test_retention_all_heads_full_and_all_empty():
    """Retention 1 everywhere: no complement, nothing recalled, every head is plain attention.
    Retention 0 everywhere: tidal heads see text + resident chunks, fixed heads text only."""
    w = _small("ret_extremes", 308, L=2, Hq=8, Hkv=4, Ta=300, cl=32, steps=4)
    h = _run(w, importance=np.ones((2, 4), np.float32), lam=1.0)
    assert h.geo["keep_total"] == -1 and (h.head_keep == w.audio_len).all()
    _run(w, importance=np.ones((2, 4), np.float32), lam=0.0, flags=_next())


def test_retention_qwen_shaped_all_steps():
    _run(configs.QWEN_10MIN, importance=gen.importance(configs.QWEN_10MIN), lam=0.4, flags=_next())


def test_retention_voxtral_shaped_sampled_heads():
    w = configs.VOXTRAL_10MIN.with_(steps=48)
    _run(w, head_mask_fn=_sampled(16), importance=gen.importance(w), lam=0.4, flags=_next())


def test_retention_recall_bytes_ragged_layout():
    """Per segment block: every tidal head in role order, its complement K rows then V rows with
    that head's own row count (padding zero); device slot = host block = the cache's rows."""
    from tests.wnw_harness import Lockstep, log
    w = _small("ret_bytes", 309, L=2, Hq=8, Hkv=4, Ta=300, Tt=5, cl=32, steps=2)
    log("[case] ragged recall bytes")
    h = Lockstep(w, importance=_imp(w, 309, ((0, 1),), ((1, 2),)), lam=1.0)
    try:
        _, _, sel, res = h.gpu_step(0)
        W = h.W
        nbytes = h.geo["chunk_bytes"]
        kd, vd = h.ok_[0], h.ov_[0]
        tidal = [(l, kv) for l in range(w.layers) for kv in range(w.kv_heads) if h.roles[l, kv] == 1]
        segs = [(c0, min(c0 + w.chunk_len, w.audio_len)) for c0 in range(0, w.audio_len, w.chunk_len)]
        comps = []
        for l, kv in tidal:
            keep = h.oracle.keep_mask(0, l, kv)
            comps.append(max(sum(1 for t in range(a, e) if not keep[t]) for a, e in segs))
        assert nbytes == 2 * 128 * 2 * sum(comps)
        for c in np.nonzero(res[0])[0]:
            dev = np.empty(nbytes // 2, dtype=np.uint16)
            hst = np.empty(nbytes // 2, dtype=np.uint16)
            W.wnw_debug_read_slot(h.ctx, 0, int(c), dev, nbytes)
            W.wnw_debug_read_host_chunk(h.ctx, 0, int(c), hst, nbytes)
            assert np.array_equal(dev, hst)
            off = 0
            for (l, kv), cm in zip(tidal, comps):
                blk = dev[off * 128:(off + 2 * cm) * 128].reshape(2, cm, 128)
                off += 2 * cm
                keep = h.oracle.keep_mask(0, l, kv)
                a, e = segs[int(c)]
                rows = [t for t in range(a, e) if not keep[t]]
                assert np.array_equal(blk[0, : len(rows)], kd[l, kv, rows])
                assert np.array_equal(blk[1, : len(rows)], vd[l, kv, rows])
                assert not blk[:, len(rows):].any()
            assert off * 128 * 2 == nbytes
    finally:
        h.close()


# ---- prefill compression on the device: text-to-audio attention sums (wnw_prefill_scores) and
# the per-segment ranking (wnw_set_roles_device); the scores are checked against the oracle's,
# then the oracle takes the device's fp32 scores and the decode steps run in lock step.

PRE = [
    _small("pre_g2", 401, Tt=9),
    _small("pre_g1_text_ragged", 402, Hq=4, Hkv=4, Tt=77, Ta=333, cl=40),
    _small("pre_g4_long_text", 403, Hq=8, Hkv=2, Tt=300, Ta=517, cl=50),
    _small("pre_g8_chunk256", 404, Hq=16, Hkv=2, Tt=130, Ta=1300, cl=256),
    _small("pre_g6", 405, Hq=12, Hkv=2, Tt=3, Ta=1111, cl=100),
    _small("pre_no_text", 406, Tt=0),
    _small("pre_batch3", 407, B=3, Ta=777, Tt=65, cl=37, steps=4),
    _small("pre_short_audio", 419, Ta=40, Tt=70, cl=16),   # fewer audio keys than one wavefront's
]


@pytest.mark.parametrize("w", PRE, ids=[w.name for w in PRE])
def test_prefill_device_lockstep(w):
    h = _run(w, prefill_device=True)
    from tests.wnw_harness import log
    log(f"[prefill] {w.name}: max prefill score rel err {h.prefill_err:.3g}")


def test_prefill_device_with_overlap_and_retention():
    w = _small("pre_ovl_ret", 408, L=2, Hq=8, Hkv=4, Ta=480, Tt=33, cl=32, steps=6)
    _run(w, prefill_device=True, flags=_ovl(_next()))
    _run(w, prefill_device=True, importance=_imp(w, 408, ((0, 1),), ((1, 2),)), lam=1.0, flags=_next())


@pytest.mark.parametrize("glob", [False, True], ids=["per_segment", "global"])
def test_prefill_device_ranking_equals_host_ranking(glob):
    """The same fp32 scores through wnw_set_roles_device and wnw_set_roles give byte-identical
    host complements and bitwise identical steps (ties, -0 and +0 included)."""
    import torch
    from paper_2608_22704_amd import wnw as W
    from tests.wnw_harness import log, to_dev
    w = _small("pre_dev_vs_host", 409, L=2, Hq=8, Hkv=4, Ta=517, Tt=20, cl=50, steps=5)
    log("[case] device ranking vs host ranking")
    B, L, H, T, D = w.batch, w.layers, w.kv_heads, w.total_len, w.head_dim
    kd = torch.empty((B, L, H, T, D), dtype=torch.int16, device="cuda")
    vd = torch.empty_like(kd)
    qs = []
    for b in range(B):
        seq = gen.sequence(w, b)
        kd[b].copy_(to_dev(seq["k"]))
        vd[b].copy_(to_dev(seq["v"]))
        qs.append(seq["q"])
    rng = np.random.default_rng(7)
    sc = (rng.integers(-25, 25, size=(B, L, H, w.audio_len)) / 50.0).astype(np.float32)   # many ties
    sc[rng.random(sc.shape) < 0.05] = -0.0
    roles = gen.roles(w)
    cfg = W.make_config(B, L, w.q_heads, H, w.audio_len, w.text_len, w.chunk_len, w.budget_bp,
                        flags=W.WNW_F_PREFILL_GLOBAL if glob else 0)
    ctxs = [W.wnw_init_cache(cfg, kd, vd), W.wnw_init_cache(cfg, kd, vd)]
    try:
        W.wnw_set_roles(ctxs[0], roles, sc)
        W.wnw_set_roles_device(ctxs[1], roles, torch.from_numpy(sc).cuda())
        geo = W.wnw_query_geometry(ctxs[0])
        nb = geo["chunk_bytes"]
        for b in range(B):
            for c in range(geo["n_segments"]):
                a0, a1 = np.empty(nb // 2, np.uint16), np.empty(nb // 2, np.uint16)
                W.wnw_debug_read_host_chunk(ctxs[0], b, c, a0, nb)
                W.wnw_debug_read_host_chunk(ctxs[1], b, c, a1, nb)
                assert np.array_equal(a0, a1), f"seq {b} segment {c}"
        outs = [torch.empty((B, L, w.q_heads, D), dtype=torch.float32, device="cuda") for _ in ctxs]
        for s in range(w.steps):
            q = to_dev(np.stack([qs[b][s] for b in range(B)]))
            for c, o in zip(ctxs, outs):
                W.wnw_decode_step(c, q, o)
            torch.cuda.synchronize()
            assert torch.equal(outs[0], outs[1]), f"step {s}"
    finally:
        for c in ctxs:
            W.wnw_destroy(c)


def test_prefill_scores_voxtral_full_size_sampled():
    """Full-size 15k-audio cache with 512 text tokens: device scores of sampled heads against the
    oracle (every head is computed on the device)."""
    import torch
    from paper_2608_22704_amd import wnw as W
    from tests.wnw_harness import PREFILL_RTOL, log, to_dev
    from oracle import oracle as O
    w = configs.VOXTRAL_10MIN
    log("[case] prefill scores, 15k audio + 512 text, sampled heads")
    B, L, H, T, D = w.batch, w.layers, w.kv_heads, w.total_len, w.head_dim
    seq = gen.sequence(w, 0)
    kd = to_dev(seq["k"])[None].contiguous()
    qt = np.stack([gen.text_queries(w, 0, l, kv, seq["k"][l, kv]) for l in range(L) for kv in range(H)])
    qt = qt.reshape(L, w.q_heads, w.text_len, D)
    cfg = W.make_config(B, L, w.q_heads, H, w.audio_len, w.text_len, w.chunk_len, w.budget_bp)
    ctx = W.wnw_init_cache(cfg, kd, kd)
    try:
        sc = torch.empty((B, L, H, w.audio_len), dtype=torch.float32, device="cuda")
        W.wnw_prefill_scores(ctx, to_dev(qt)[None].contiguous(), sc)
        torch.cuda.synchronize()
        got = sc.cpu().numpy()[0]
    finally:
        W.wnw_destroy(ctx)
    rng = np.random.default_rng(11)
    heads = [(int(x) // H, int(x) % H) for x in rng.choice(L * H, size=3, replace=False)]
    for l, kv in heads:
        c1 = O.make_cfg(1, 1, w.group, 1, D, w.audio_len, w.text_len, w.chunk_len, w.budget_bp)
        ref = O.prefill_scores(c1, seq["k"][l, kv][None, None, None], qt[l, kv * w.group:(kv + 1) * w.group][None, None])[0, 0, 0]
        rel = np.abs(got[l, kv] - ref) / np.maximum(ref, 1e-300)
        log(f"[prefill] head ({l},{kv}): max rel err {rel.max():.3g}")
        assert (rel <= PREFILL_RTOL).all()


# ---- global prefill variant: the per-segment total kept over the whole audio of a head (ablation
# of per-segment selection); complements then differ in size from segment to segment.

def _glob(extra=0):
    from paper_2608_22704_amd import wnw as W
    return W.WNW_F_PREFILL_GLOBAL | extra


GLOB = [
    _small("glob_g2", 501, Tt=9),
    _small("glob_g1_chunk7", 502, Hq=4, Hkv=4, cl=7),
    _small("glob_g8_chunk256", 503, Hq=16, Hkv=2, cl=256, Ta=1300, Tt=300),
    _small("glob_batch3", 504, B=3, Ta=777, Tt=1, cl=37, budget=3000, steps=9),
    _small("glob_low_budget", 505, Ta=600, cl=16, budget=500, steps=8),
]


@pytest.mark.parametrize("w", GLOB, ids=[w.name for w in GLOB])
def test_prefill_global_lockstep(w):
    _run(w, flags=_glob())
    _run(w, flags=_glob(_next()))


def test_prefill_global_device_scores_and_variants():
    w = _small("glob_dev", 506, L=2, Hq=8, Hkv=4, Ta=480, Tt=33, cl=32, steps=6)
    _run(w, prefill_device=True, flags=_glob(_next()))
    _run(w, prefill_device=True, flags=_glob(_ovl()))
    _run(w, flags=_glob(_next()), importance=_imp(w, 506, ((0, 1),), ((1, 2),)), lam=1.0)


# ---- decode-time append: the generated token's K/V rows join every head's key set before each
# step (room reserved for w.steps tokens); the oracle appends the same rows.

APP = [
    _small("app_g2", 601, Tt=9),
    _small("app_anchor_tile_boundary", 602, Ta=250, Tt=4, cl=32, steps=8),
    _small("app_static_tile_boundary", 603, Ta=250, Tt=4, cl=32, budget=10000, steps=6),
    _small("app_no_text", 604, Tt=0),
    _small("app_budget_zero", 605, budget=0),
    _small("app_g8_chunk256", 606, Hq=16, Hkv=2, cl=256, Ta=1300, Tt=300),
    _small("app_text_only", 607, Ta=0, Tt=40),
]


@pytest.mark.parametrize("w", APP, ids=[w.name for w in APP])
def test_append_lockstep(w):
    _run(w, append=True)
    _run(w, append=True, flags=_next())


def test_append_with_variants():
    w = _small("app_variants", 608, L=2, Hq=8, Hkv=4, Ta=480, Tt=5, cl=32, steps=8)
    _run(w, append=True, flags=_ovl(_next()))
    _run(w, append=True, flags=_next(), importance=_imp(w, 608, ((0, 1),), ((1, 2),)), lam=1.0)
    _run(w, append=True, flags=_glob(_next()))
    from paper_2608_22704_amd import wnw as W
    _run(w, append=True, flags=_next(W.WNW_F_RECALL_MEMCPY))


def test_append_qwen_shaped_all_steps():
    _run(configs.QWEN_10MIN, append=True, flags=_next())


def test_append_beyond_reserved_rows_is_refused():
    from paper_2608_22704_amd import wnw as W
    from tests.wnw_harness import Lockstep, log, to_dev
    w = _small("app_full", 609, steps=2)
    log("[case] append beyond the reserved rows")
    h = Lockstep(w, append=True)
    try:
        h.step(0)
        h.step(1)
        kn, vn = h.new_token(2)
        with pytest.raises(W.WnwError):
            W.wnw_append_kv(h.ctx, to_dev(kn), to_dev(vn))
    finally:
        h.close()


# ---- head triage arithmetic on the device: voice-score hits (exact against the oracle) and key
# sensitivity (fp32 squares, double sums; 1e-5 relative), then the roles.

VH = [  # (L, H_q, H_kv, T_a, T_t, n_tok, K)
    (1, 8, 2, 300, 5, 7, 4),
    (2, 8, 8, 97, 0, 64, 8),
    (2, 12, 4, 517, 9, 22, 1),
    (1, 24, 3, 1000, 3, 17, 4),
    (1, 16, 2, 64, 1, 9, 8),
    (1, 8, 2, 5, 2, 3, 4),        # fewer audio keys than one 16-key block
    (1, 4, 1, 16, 0, 16, 8),      # exactly one key tile and one 64-row work-group
    (1, 8, 1, 33, 2, 40, 4),      # five work-groups, a ragged key tail
]


@pytest.mark.parametrize("shape", VH, ids=[f"L{s[0]}_q{s[1]}_kv{s[2]}_Ta{s[3]}_tok{s[5]}_K{s[6]}" for s in VH])
def test_voice_hits_match_oracle(shape):
    import torch
    from oracle import oracle as O
    from paper_2608_22704_amd import wnw as W
    from tests.wnw_harness import log, to_dev
    L, Hq, Hkv, Ta, Tt, n_tok, K = shape
    log(f"[case] voice hits {shape}")
    rng = np.random.default_rng(sum(shape))
    k = gen.f32_to_bf16(rng.standard_normal((L, Hkv, Ta + Tt, 128), dtype=np.float32))
    k[:, :, 5] = k[:, :, 2]                      # duplicate keys: ties go to the lower position
    q = gen.f32_to_bf16(rng.standard_normal((n_tok, L, Hq, 128), dtype=np.float32))
    a = rng.integers(0, Ta, size=n_tok)
    span = np.stack([a, np.minimum(a + rng.integers(1, 12, size=n_tok), Ta)], axis=1).astype(np.int32)
    span[0] = (2, 3)
    hits = torch.empty((n_tok, L, Hq), dtype=torch.int32, device="cuda")
    W.wnw_voice_hits(to_dev(k), to_dev(q), torch.from_numpy(span).cuda(), K, Ta, hits)
    torch.cuda.synchronize()
    want = O.voice_hits(k, q, span, K, Ta)
    assert np.array_equal(hits.cpu().numpy(), want)


def test_key_sensitivity_and_roles_match_oracle():
    import torch
    from oracle import oracle as O
    from paper_2608_22704_amd import wnw as W
    from tests.wnw_harness import log
    log("[case] key sensitivity and roles")
    rng = np.random.default_rng(3)
    n_tok, L, Hkv, Ta = 5, 3, 4, 333
    grad = (rng.standard_normal((n_tok, L, Hkv, Ta, 128), dtype=np.float32)
            * rng.random((n_tok, L, Hkv, 1, 1), dtype=np.float32))
    sens = torch.empty((n_tok, L, Hkv), dtype=torch.float32, device="cuda")
    W.wnw_key_sensitivity(torch.from_numpy(grad).cuda(), sens)
    torch.cuda.synchronize()
    got = sens.cpu().numpy()
    want = O.key_sensitivity(grad)
    rel = np.abs(got - want) / want
    log(f"[triage] key sensitivity max rel err {rel.max():.3g}")
    assert (rel <= 1e-5).all()
    hits = rng.integers(0, 5, size=(n_tok, L, Hkv * 2)).astype(np.int32)
    sample = np.array([0, 0, 1, 1, 1], dtype=np.int32)
    r1, i1, _, _ = W.wnw_triage(hits, 4, got, sample, 6, 2)
    r2, _, _, i2 = O.triage(hits, 4, got.astype(np.float64), sample, 6, 2)
    assert np.array_equal(r1, r2)
    np.testing.assert_allclose(i1, i2, rtol=1e-6)


# ---- feature combinations: every option of the step together, batch 3

COMBOS = [
    dict(flags=("ovl", "next"), importance=True, append=True, prefill_device=True),
    dict(flags=("ovl", "glob"), importance=True, append=True),
    dict(flags=("next", "glob", "memcpy"), append=True, prefill_device=True),
    dict(flags=("ovl", "next", "memcpy"), importance=True),
]


@pytest.mark.parametrize("combo", COMBOS, ids=["+".join(c["flags"]) + ("+imp" if c.get("importance") else "") +
                                                ("+app" if c.get("append") else "") +
                                                ("+dev" if c.get("prefill_device") else "") for c in COMBOS])
def test_feature_combinations(combo):
    from paper_2608_22704_amd import wnw as W
    bits = {"ovl": W.WNW_F_OVERLAP_CHUNKS, "next": W.WNW_F_SELECT_NEXT_STEP, "glob": W.WNW_F_PREFILL_GLOBAL,
            "memcpy": W.WNW_F_RECALL_MEMCPY}
    w = _small("combo", 701, B=3, L=2, Hq=12, Hkv=4, Ta=611, Tt=17, cl=34, budget=2500, steps=7)
    kw = dict(flags=sum(bits[f] for f in combo["flags"]), append=combo.get("append", False),
              prefill_device=combo.get("prefill_device", False))
    if combo.get("importance"):
        kw.update(importance=_imp(w, 701, ((0, 1),), ((1, 3),)), lam=0.9)
    _run(w, **kw)


# ---- stream ordering of the recall: every reader of a recalled slot waits for the recall ------

@pytest.mark.parametrize("mode", ["next_memcpy", "next_kernel", "same_memcpy"])
def test_delayed_recall_gives_identical_results(mode):
    """Each recall delayed by 3 ms (the host waits before issuing the copies and a host function
    sleeps ahead of them on every copy stream; ahead of the copy kernel without copy engines):
    twelve steps enqueued back to back with no host synchronisation between them (outputs, scores
    and selections copied on the caller's stream after each step) are bit-identical to an
    undelayed run.  With next-step timing and copy engines the copies are issued by the library's
    recall thread while the caller keeps enqueueing steps."""
    import torch
    from paper_2608_22704_amd import wnw as W
    from tests.wnw_harness import log, to_dev
    flags = {"next_memcpy": W.WNW_F_SELECT_NEXT_STEP | W.WNW_F_RECALL_MEMCPY,
             "next_kernel": W.WNW_F_SELECT_NEXT_STEP, "same_memcpy": W.WNW_F_RECALL_MEMCPY}[mode]
    w = _small("recall_delay", 180, L=2, Hq=8, Hkv=4, Ta=480, Tt=5, cl=16, budget=2000, steps=12)
    log(f"[case] delayed recall, {mode}")
    B, L, H, T, D = w.batch, w.layers, w.kv_heads, w.total_len, w.head_dim
    seqs = [gen.sequence(w, b) for b in range(B)]
    kd = torch.stack([to_dev(sq["k"]) for sq in seqs])
    vd = torch.stack([to_dev(sq["v"]) for sq in seqs])
    qd = torch.stack([to_dev(np.stack([sq["q"][s] for sq in seqs])) for s in range(w.steps)])
    prefill = np.stack([sq["prefill"] for sq in seqs])
    runs = []
    for delay in (0, 3000):
        cfg = W.make_config(B, L, w.q_heads, H, w.audio_len, w.text_len, w.chunk_len, w.budget_bp, flags=flags)
        ctx = W.wnw_init_cache(cfg, kd, vd)
        try:
            W.wnw_set_roles(ctx, gen.roles(w), prefill)
            W.wnw_debug_set_recall_delay(ctx, delay)
            geo = W.wnw_query_geometry(ctx)
            out = torch.empty((B, L, w.q_heads, D), dtype=torch.float32, device="cuda")
            sc = torch.empty((B, geo["n_chunks"]), dtype=torch.float32, device="cuda")
            sel = torch.empty((B, geo["k"]), dtype=torch.int32, device="cuda")
            kept = []
            for s in range(w.steps):
                W.wnw_decode_step(ctx, qd[s], out, sc, sel)
                kept.append((out.clone(), sc.clone(), sel.clone()))
            torch.cuda.synchronize()
            st = W.wnw_get_stats(ctx)
            assert st["recalled_chunks"] > 0
            runs.append([[x.cpu().numpy() for x in step] for step in kept])
        finally:
            W.wnw_destroy(ctx)
    for s, (a, b) in enumerate(zip(*runs)):
        for x, y in zip(a, b):
            assert np.array_equal(x.view(np.uint32) if x.dtype == np.float32 else x,
                                  y.view(np.uint32) if y.dtype == np.float32 else y), f"step {s} differs"


def test_selection_inside_and_before_the_tidal_launch_bit_identical():
    """With next-step timing and copy-engine recall a step runs the chunk-mass merge and the
    selection inside the tidal launch after a previous-step recall of at most 4 MiB, else as two
    kernels before it; the copy-kernel path always runs the two kernels.  A forced schedule whose
    selected set moves to a disjoint one every second step alternates recalls of tens of MB with
    steps that recall nothing, so the copy-engine run takes both routes, switching back and forth;
    outputs, scores and selections match the other path bit for bit at every step."""
    import torch
    from paper_2608_22704_amd import wnw as W
    from tests.wnw_harness import log, to_dev
    w = _small("selection_place", 191, B=4, L=4, Hq=16, Hkv=8, Ta=8000, Tt=40, cl=32, budget=2000, steps=24)
    log("[case] selection inside / before the tidal launch, bit for bit")
    B, L, H, D = w.batch, w.layers, w.kv_heads, w.head_dim
    seqs = [gen.sequence(w, b) for b in range(B)]
    kd = torch.stack([to_dev(sq["k"]) for sq in seqs])
    vd = torch.stack([to_dev(sq["v"]) for sq in seqs])
    qd = torch.stack([to_dev(np.stack([sq["q"][s] for sq in seqs])) for s in range(w.steps)])
    prefill = np.stack([sq["prefill"] for sq in seqs])
    runs, placed = [], []
    for flags in (W.WNW_F_SELECT_NEXT_STEP | W.WNW_F_RECALL_MEMCPY, W.WNW_F_SELECT_NEXT_STEP):
        cfg = W.make_config(B, L, w.q_heads, H, w.audio_len, w.text_len, w.chunk_len, w.budget_bp, flags=flags)
        ctx = W.wnw_init_cache(cfg, kd, vd)
        try:
            W.wnw_set_roles(ctx, gen.roles(w), prefill)
            geo = W.wnw_query_geometry(ctx)
            k, nch = geo["k"], geo["n_chunks"]
            # disjoint sets of k chunks, a new one every second step (sequences offset)
            sched = np.empty((w.steps, B, k), dtype=np.int32)
            for s in range(w.steps):
                for b in range(B):
                    sched[s, b] = np.sort((np.arange(k) + (s // 2 + b) * k) % nch)
            sd = torch.from_numpy(sched).cuda()
            out = torch.empty((B, L, w.q_heads, D), dtype=torch.float32, device="cuda")
            sc = torch.empty((B, nch), dtype=torch.float32, device="cuda")
            sel = torch.empty((B, k), dtype=torch.int32, device="cuda")
            kept = []
            for s in range(w.steps):
                W.wnw_set_selection_override(ctx, sd[s])
                W.wnw_decode_step(ctx, qd[s], out, sc, sel)
                kept.append((out.clone(), sc.clone(), sel.clone()))
            torch.cuda.synchronize()
            W.wnw_set_selection_override(ctx, None)
            st = W.wnw_get_stats(ctx)
            assert st["recalled_bytes"] > 2 * (4 << 20) * (w.steps // 4), st["recalled_bytes"]
            placed.append(st["selections_in_tidal"])
            runs.append([[x.cpu().numpy() for x in step] for step in kept])
        finally:
            W.wnw_destroy(ctx)
    # the copy-engine run switched between the two routes; the copy-kernel run never used the first
    assert 0 < placed[0] < w.steps and placed[1] == 0, placed
    for s, (a, b) in enumerate(zip(*runs)):
        for x, y in zip(a, b):
            assert np.array_equal(x.view(np.uint32) if x.dtype == np.float32 else x,
                                  y.view(np.uint32) if y.dtype == np.float32 else y), f"step {s} differs"


def test_next_step_recall_paths_bit_identical():
    """With next-step timing the copy engines (the host knows each step's list length from the
    mirror and launches one work-group per slot item) and the copy kernel (the item count comes
    from the select kernel, and resident work-groups loop over the items, here more than a full
    round of them) attend to the same slot items into the same partials: outputs, scores and
    selections are bit-identical step by step, four sequences with lists of their own lengths."""
    import torch
    from paper_2608_22704_amd import wnw as W
    from tests.wnw_harness import log, to_dev
    w = _small("recall_paths", 190, B=4, L=4, Hq=16, Hkv=8, Ta=8000, Tt=40, cl=32, budget=2000, steps=16)
    log("[case] next-step recall paths, bit for bit")
    B, L, H, D = w.batch, w.layers, w.kv_heads, w.head_dim
    seqs = [gen.sequence(w, b) for b in range(B)]
    kd = torch.stack([to_dev(sq["k"]) for sq in seqs])
    vd = torch.stack([to_dev(sq["v"]) for sq in seqs])
    qd = torch.stack([to_dev(np.stack([sq["q"][s] for sq in seqs])) for s in range(w.steps)])
    prefill = np.stack([sq["prefill"] for sq in seqs])
    runs, items = [], []
    for flags in (W.WNW_F_SELECT_NEXT_STEP | W.WNW_F_RECALL_MEMCPY, W.WNW_F_SELECT_NEXT_STEP):
        cfg = W.make_config(B, L, w.q_heads, H, w.audio_len, w.text_len, w.chunk_len, w.budget_bp, flags=flags)
        ctx = W.wnw_init_cache(cfg, kd, vd)
        try:
            W.wnw_set_roles(ctx, gen.roles(w), prefill)
            geo = W.wnw_query_geometry(ctx)
            out = torch.empty((B, L, w.q_heads, D), dtype=torch.float32, device="cuda")
            sc = torch.empty((B, geo["n_chunks"]), dtype=torch.float32, device="cuda")
            sel = torch.empty((B, geo["k"]), dtype=torch.int32, device="cuda")
            kept = []
            for s in range(w.steps):
                W.wnw_decode_step(ctx, qd[s], out, sc, sel)
                kept.append((out.clone(), sc.clone(), sel.clone()))
            torch.cuda.synchronize()
            st = W.wnw_get_stats(ctx)
            assert st["recalled_chunks"] > geo["n_slots"], "the slot pool was not wrapped"
            # complement rows attended per step and tidal head, in 128-row items
            items.append(st["slot_rows"] / w.steps / B / w.n_tidal / 128.0)
            runs.append([[x.cpu().numpy() for x in step] for step in kept])
        finally:
            W.wnw_destroy(ctx)
    # more slot items per step than 1 024 resident work-groups take in one round
    assert items[0] * w.n_tidal * B > 1024, items
    for s, (a, b) in enumerate(zip(*runs)):
        for x, y in zip(a, b):
            assert np.array_equal(x.view(np.uint32) if x.dtype == np.float32 else x,
                                  y.view(np.uint32) if y.dtype == np.float32 else y), f"step {s} differs"
