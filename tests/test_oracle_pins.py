"""Pins of the CPU oracle against things other than itself.

Each test ties one part of the oracle to an independent fact: a library routine computing the
same definition (torch's scaled_dot_product_attention in double), a closed form, a brute-force
enumeration, a hand-worked trace, or a value printed in the paper.  A plausible mistake in the
oracle (a dropped text term, a sum instead of a mean, a reversed tie rule, an off-by-one in the
eviction lag, a wrong keep count) fails at least one of them.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

from synth.gen import f32_to_bf16, bf16_to_f32

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _rand_cache(rng, B, L, H, T, D, scale=1.0):
    k = f32_to_bf16(rng.standard_normal((B, L, H, T, D)).astype(np.float32) * scale)
    v = f32_to_bf16(rng.standard_normal((B, L, H, T, D)).astype(np.float32))
    return k, v


def _sdpa(q, k, v, mask=None):
    """One query q [d] over rows k [T][d], v [T][e] (bf16 bit patterns or float), double."""
    f = lambda a: torch.from_numpy(bf16_to_f32(a).astype(np.float64)) if a.dtype == np.uint16 else torch.from_numpy(a.astype(np.float64))
    qq, kk, vv = f(q)[None, None], f(k)[None], f(v)[None]
    m = None if mask is None else torch.from_numpy(mask.astype(bool))[None, None]
    return torch.nn.functional.scaled_dot_product_attention(qq, kk, vv, attn_mask=m)[0, 0].numpy()


def _small(oracle_mod, seed=0, B=2, L=2, H=3, g=2, D=16, Ta=37, Tt=5, cl=8, budget=2500, **kw):
    rng = np.random.default_rng(seed)
    k, v = _rand_cache(rng, B, L, H, Ta + Tt, D)
    roles = np.array([[0, 1, 2], [1, 2, 0]], dtype=np.uint8)[:L, :H]
    pf = rng.random((B, L, H, Ta), dtype=np.float32)
    cfg = oracle_mod.make_cfg(B, L, H * g, H, D, Ta, Tt, cl, budget, **kw)
    o = oracle_mod.Oracle(cfg, k, v, roles, pf)
    q = f32_to_bf16(rng.standard_normal((B, L, H * g, D)).astype(np.float32))
    return o, k, v, roles, pf, q


def test_full_budget_equals_full_attention(oracle_mod):
    """At 100 % budget every head holds every row, so WnW is plain attention (Full Cache)."""
    o, k, v, roles, pf, q = _small(oracle_mod, budget=10000)
    r = o.step(q)
    B, L, Hq, D = q.shape
    g = Hq // k.shape[2]
    for b, l, hq in itertools.product(range(B), range(L), range(Hq)):
        ref = _sdpa(q[b, l, hq], k[b, l, hq // g], v[b, l, hq // g])
        np.testing.assert_allclose(r["out"][b, l, hq], ref, rtol=0, atol=1e-12)


def test_keep_masks_are_per_segment_top_by_prefill_score(oracle_mod):
    """Prefill compression: in every segment exactly floor(retention * len) positions are kept
    and each kept position outranks each dropped one (score, then lower position)."""
    rng = np.random.default_rng(3)
    B, L, H, D, Ta, Tt, cl, budget = 2, 1, 3, 8, 70, 2, 16, 3000
    k, v = _rand_cache(rng, B, L, H, Ta + Tt, D)
    pf = (rng.integers(0, 4, size=(B, L, H, Ta)) / 4.0).astype(np.float32)   # heavy ties
    roles = np.array([[0, 1, 2]], dtype=np.uint8)
    o = oracle_mod.Oracle(oracle_mod.make_cfg(B, L, H, H, D, Ta, Tt, cl, budget), k, v, roles, pf)
    for b, h in itertools.product(range(B), range(H)):
        m = o.keep_mask(b, 0, h)
        if roles[0, h] == 0:
            assert m.all()
            continue
        for c0 in range(0, Ta, cl):
            seg = range(c0, min(c0 + cl, Ta))
            kept = [t for t in seg if m[t]]
            drop = [t for t in seg if not m[t]]
            assert len(kept) == (budget * len(seg)) // 10000
            for a in kept:
                for d in drop:
                    assert (pf[b, 0, h, a], -a) > (pf[b, 0, h, d], -d)


def test_chunk_mass_is_softmax_mass_of_the_chunk(oracle_mod):
    """Eq. 2 per anchor q-head: the mass of chunk c is the attention output for V = the
    indicator of c (library attention), and the chunk masses add up to the audio mass."""
    o, k, v, roles, pf, q = _small(oracle_mod, seed=5, Ta=45, Tt=6, cl=8)
    r = o.step(q)
    B, L, Hq, D = q.shape
    H = k.shape[2]
    g = Hq // H
    Ta, T, nc = 45, 51, o.n_chunks
    ind = np.zeros((T, nc + 2))
    for t in range(Ta):
        ind[t, t // 8] = 1.0
    ind[:Ta, nc] = 1.0            # audio indicator
    ind[Ta:, nc + 1] = 1.0        # text indicator
    a = 0
    for l, h in itertools.product(range(L), range(H)):
        if roles[l, h] != 0:
            continue
        for j in range(g):
            for b in range(B):
                ref = _sdpa(q[b, l, h * g + j], k[b, l, h], ind)
                np.testing.assert_allclose(r["mass"][b, a * g + j], ref[:nc], rtol=1e-12, atol=1e-15)
                assert abs(r["mass"][b, a * g + j].sum() - ref[nc]) < 1e-12
                assert abs(ref[nc] + ref[nc + 1] - 1.0) < 1e-12
        a += 1


def test_equal_logits_closed_form(oracle_mod):
    """q = 0 makes every logit equal: p = 1 / T on every row, so every chunk (the short last
    one included) scores n_anchor_q / T -- a mean, not a sum -- and the tie rule selects the
    lowest ids 0..k-1."""
    o, k, v, roles, pf, q = _small(oracle_mod, seed=7, Ta=37, Tt=5, cl=8, budget=4000)
    q[:] = 0
    r = o.step(q)
    T = 42
    assert o.k == (4000 * 37) // (10000 * 8)
    np.testing.assert_allclose(r["scores"], o.n_anchor_q / T, rtol=1e-13)
    assert (r["selected"] == np.arange(o.k)).all()
    # equal logits over the whole key set also make every output the mean of V over that set
    B, L, Hq, D = q.shape
    g = Hq // k.shape[2]
    for b, l, hq in itertools.product(range(B), range(L), range(Hq)):
        h = hq // g
        vv = bf16_to_f32(v[b, l, h]).astype(np.float64)
        if roles[l, h] == 0:
            rows = np.arange(T)
        elif roles[l, h] == 2:
            rows = np.concatenate([np.nonzero(o.keep_mask(b, l, h))[0], np.arange(37, T)])
        else:
            continue
        np.testing.assert_allclose(r["out"][b, l, hq], vv[rows].mean(axis=0), rtol=1e-12, atol=1e-14)


def _brute_topk(s, k):
    """The unique k-subset whose members all beat all non-members under (score desc, id asc)."""
    n = len(s)
    found = []
    for sub in itertools.combinations(range(n), k):
        ins = set(sub)
        if all((s[i], -i) > (s[j], -j) for i in ins for j in range(n) if j not in ins):
            found.append(sub)
    assert len(found) == 1
    return list(found[0])


@pytest.mark.parametrize("seed", range(12))
def test_topk_matches_brute_force(oracle_mod, seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 13))
    k = int(rng.integers(0, n + 1))
    s = (rng.integers(0, 5, size=n) / 7.0).astype(np.float32)   # planted ties
    assert list(oracle_mod.topk(s, k)) == _brute_topk(list(s), k)


def test_residency_trace_matches_hand_worked_lag(oracle_mod):
    gold = json.load(open(os.path.join(GOLD, "residency_trace.json")))
    rng = np.random.default_rng(11)
    B, L, H, D, Ta, Tt, cl = 1, 1, 2, 8, 160, 3, 16           # 10 chunks
    k, v = _rand_cache(rng, B, L, H, Ta + Tt, D)
    roles = np.array([[0, 1]], dtype=np.uint8)
    pf = rng.random((B, L, H, Ta), dtype=np.float32)
    for mode, key in ((0, "resident_same_step"), (1, "resident_next_step")):
        cfg = oracle_mod.make_cfg(B, L, H, H, D, Ta, Tt, cl, 2000, top_k=1, evict_lag=gold["delta"], next_step=mode)
        o = oracle_mod.Oracle(cfg, k, v, roles, pf)
        q = f32_to_bf16(rng.standard_normal((B, L, H, D)).astype(np.float32))
        for s, want in zip(gold["selections"], gold[key]):
            r = o.step(q, forced=np.array([[s]]))
            assert list(np.nonzero(r["resident"][0])[0]) == want


def test_tidal_and_fixed_attend_over_their_key_sets(oracle_mod):
    """Tidal heads: kept rows + resident chunks + text; fixed heads: kept rows + text
    (library attention with a boolean mask built from the keep flags and the resident set)."""
    o, k, v, roles, pf, q = _small(oracle_mod, seed=13, Ta=64, Tt=4, cl=8, budget=2500)
    B, L, Hq, D = q.shape
    H = k.shape[2]
    g = Hq // H
    for step in range(4):
        qs = f32_to_bf16((np.random.default_rng(100 + step).standard_normal(q.shape)).astype(np.float32))
        r = o.step(qs)
        for b, l, hq in itertools.product(range(B), range(L), range(Hq)):
            h = hq // g
            mask = np.ones(68, dtype=bool)
            if roles[l, h] != 0:
                keep = o.keep_mask(b, l, h).astype(bool)
                if roles[l, h] == 1:
                    keep |= np.repeat(r["resident"][b].astype(bool), 8)[:64]
                mask[:64] = keep
            ref = _sdpa(qs[b, l, hq], k[b, l, h], v[b, l, h], mask)
            np.testing.assert_allclose(r["out"][b, l, hq], ref, rtol=0, atol=1e-12)


def test_next_step_equals_same_step_with_previous_selection(oracle_mod):
    """With next-step timing, step s uses the resident set of step s-1: the same as running the
    same-step oracle on the selections shifted by one step (nothing selected at step 0)."""
    rng = np.random.default_rng(17)
    B, L, H, g, D, Ta, Tt, cl = 2, 2, 3, 2, 8, 96, 4, 8
    k, v = _rand_cache(rng, B, L, H, Ta + Tt, D)
    roles = np.array([[0, 1, 2], [1, 1, 0]], dtype=np.uint8)
    pf = rng.random((B, L, H, Ta), dtype=np.float32)
    nxt = oracle_mod.Oracle(oracle_mod.make_cfg(B, L, H * g, H, D, Ta, Tt, cl, 2500, next_step=1), k, v, roles, pf)
    same = oracle_mod.Oracle(oracle_mod.make_cfg(B, L, H * g, H, D, Ta, Tt, cl, 2500), k, v, roles, pf)
    prev_sel = np.full((B, nxt.k), -1, dtype=np.int32)
    for s in range(6):
        q = f32_to_bf16(rng.standard_normal((B, L, H * g, D)).astype(np.float32))
        a = nxt.step(q)
        b_ = same.step(q, forced=prev_sel)
        np.testing.assert_array_equal(a["out"], b_["out"])
        np.testing.assert_array_equal(a["resident"], b_["resident"])
        prev_sel = a["selected"].copy()


def test_single_text_row_and_dominant_logit(oracle_mod):
    """Budget 0 leaves a fixed head one text row: its output is that V row.  A key with a huge
    logit takes all the mass: the anchor output is that key's V row."""
    rng = np.random.default_rng(19)
    B, L, H, D, Ta, Tt, cl = 1, 1, 2, 8, 24, 1, 8
    k, v = _rand_cache(rng, B, L, H, Ta + Tt, D)
    q = f32_to_bf16(rng.standard_normal((B, L, H, D)).astype(np.float32))
    k[0, 0, 0, 5] = f32_to_bf16(bf16_to_f32(q[0, 0, 0]) * 64.0)    # logit ~ 64 |q|^2 / sqrt(d)
    roles = np.array([[0, 2]], dtype=np.uint8)
    pf = rng.random((B, L, H, Ta), dtype=np.float32)
    o = oracle_mod.Oracle(oracle_mod.make_cfg(B, L, H, H, D, Ta, Tt, cl, 0), k, v, roles, pf)
    assert o.k == 0 and o.keep_total == 0
    r = o.step(q)
    np.testing.assert_array_equal(r["out"][0, 0, 1], bf16_to_f32(v[0, 0, 1, Ta]).astype(np.float64))
    np.testing.assert_allclose(r["out"][0, 0, 0], bf16_to_f32(v[0, 0, 0, 5]), rtol=0, atol=1e-9)
    assert r["mass"][0, 0].argmax() == 0 and abs(r["mass"][0, 0, 0] - 1.0) < 1e-9


def test_chunk_structure_worked_values(oracle_mod):
    gold = json.load(open(os.path.join(GOLD, "chunk_structure.json")))
    for c in gold["cases"]:
        assert oracle_mod.tokens_for_window(gold["window_seconds"]["chunk"], c["rate"]) == c["chunk_tokens"]
        assert oracle_mod.tokens_for_window(gold["window_seconds"]["segment"], c["rate"]) == c["segment_tokens"]


def test_workload_geometry(oracle_mod):
    gold = json.load(open(os.path.join(GOLD, "workload_geometry.json")))
    for c in gold["cases"]:
        cfg = oracle_mod.make_cfg(1, 1, 4, 1, 128, c["audio_len"], 16, c["chunk_len"], c["budget_bp"])
        assert oracle_mod.geometry(cfg) == (c["n_chunks"], c["k"], c["keep_total"])


def test_selection_is_topk_of_fp32_scores(oracle_mod):
    """The oracle's selection is the brute-force top-k of its own scores rounded to fp32."""
    o, k, v, roles, pf, q = _small(oracle_mod, seed=23, Ta=96, Tt=4, cl=8, budget=2500)
    for s in range(3):
        qs = f32_to_bf16(np.random.default_rng(200 + s).standard_normal(q.shape).astype(np.float32))
        r = o.step(qs)
        for b in range(q.shape[0]):
            assert list(r["selected"][b]) == _brute_topk(list(r["scores"][b].astype(np.float32)), o.k)


def test_invalid_configurations_rejected(oracle_mod):
    bad = [dict(chunk_len=0), dict(budget_bp=10001), dict(top_k=99), dict(q_heads=5)]
    for b in bad:
        kw = dict(batch=1, layers=1, q_heads=4, kv_heads=2, head_dim=8, audio_len=64, text_len=2,
                  chunk_len=8, budget_bp=2000)
        kw.update(b)
        with pytest.raises(ValueError):
            oracle_mod.geometry(oracle_mod.make_cfg(**kw))


# ---- the paper's overlapping chunks (Method, "Chunk Structure"): a chunk is two consecutive
# segments of chunk_len / 2 positions and one chunk starts at every segment.

def test_span2_geometry(oracle_mod):
    """Segments of chunk_len / 2; one chunk per segment start except the last; keep counts per
    segment; odd chunk lengths rejected."""
    cfg = oracle_mod.make_cfg(1, 1, 4, 1, 8, 100, 4, 16, 2500, chunk_span=2)
    n, k, kt = oracle_mod.geometry(cfg)
    assert oracle_mod.segments(cfg) == 13                  # ceil(100 / 8)
    assert n == 12                                         # chunks start at segments 0..11
    assert k == (2500 * 100) // (10000 * 16)               # floor(budget * T_a / chunk_len) = 1
    assert kt == 12 * 2 + (4 * 2500) // 10000              # 12 full segments keep 2, the 4-long one 1
    with pytest.raises(ValueError):
        oracle_mod.geometry(oracle_mod.make_cfg(1, 1, 4, 1, 8, 100, 4, 15, 2500, chunk_span=2))


def test_span2_residency_trace_matches_hand_worked_segments(oracle_mod):
    gold = json.load(open(os.path.join(GOLD, "residency_trace_span2.json")))
    rng = np.random.default_rng(29)
    B, L, H, D, Ta, Tt, cl = 1, 1, 2, 8, 96, 3, 16           # 12 segments of 8, 11 chunks
    k, v = _rand_cache(rng, B, L, H, Ta + Tt, D)
    roles = np.array([[0, 1]], dtype=np.uint8)
    pf = rng.random((B, L, H, Ta), dtype=np.float32)
    for mode, key in ((0, "resident_segments_same_step"), (1, "resident_segments_next_step")):
        cfg = oracle_mod.make_cfg(B, L, H, H, D, Ta, Tt, cl, 2000, top_k=1, evict_lag=gold["delta"],
                                  next_step=mode, chunk_span=2)
        o = oracle_mod.Oracle(cfg, k, v, roles, pf)
        q = f32_to_bf16(rng.standard_normal((B, L, H, D)).astype(np.float32))
        for s, want in zip(gold["selections"], gold[key]):
            r = o.step(q, forced=np.array([[s]]))
            assert list(np.nonzero(r["resident"][0])[0]) == want


def test_span2_even_chunks_are_the_disjoint_chunks_of_twice_the_segment(oracle_mod):
    """Chunk 2j of the overlapping layout covers the same positions as chunk j of the disjoint
    layout with chunks of two segments: same scores.  Segment masses equal the disjoint layout's
    chunk masses at one segment per chunk (pinned against SDPA elsewhere)."""
    rng = np.random.default_rng(31)
    B, L, H, g, D, Ta, Tt, seg = 2, 2, 3, 2, 8, 96, 4, 6     # 16 full segments, chunks of 12
    k, v = _rand_cache(rng, B, L, H, Ta + Tt, D)
    roles = np.array([[0, 1, 2], [1, 0, 0]], dtype=np.uint8)
    pf = rng.random((B, L, H, Ta), dtype=np.float32)
    span2 = oracle_mod.Oracle(oracle_mod.make_cfg(B, L, H * g, H, D, Ta, Tt, 2 * seg, 2500, chunk_span=2), k, v, roles, pf)
    disj = oracle_mod.Oracle(oracle_mod.make_cfg(B, L, H * g, H, D, Ta, Tt, 2 * seg, 2500), k, v, roles, pf)
    unit = oracle_mod.Oracle(oracle_mod.make_cfg(B, L, H * g, H, D, Ta, Tt, seg, 2500), k, v, roles, pf)
    assert span2.n_chunks == Ta // seg - 1 and disj.n_chunks == Ta // (2 * seg)
    for s in range(3):
        q = f32_to_bf16(rng.standard_normal((B, L, H * g, D)).astype(np.float32))
        a, b_, u = span2.step(q), disj.step(q), unit.step(q)
        np.testing.assert_allclose(a["scores"][:, 0::2], b_["scores"], rtol=1e-13, atol=0)
        np.testing.assert_allclose(a["mass"], u["mass"], rtol=1e-13, atol=1e-300)


def test_span2_tidal_heads_attend_over_resident_segments(oracle_mod):
    """Tidal heads: kept rows + the resident segments (both segments of every resident chunk) +
    text, against SDPA with that mask; fixed heads: kept rows + text."""
    rng = np.random.default_rng(37)
    B, L, H, g, D, Ta, Tt, cl = 2, 2, 3, 2, 8, 64, 4, 16
    k, v = _rand_cache(rng, B, L, H, Ta + Tt, D)
    roles = np.array([[0, 1, 2], [1, 2, 0]], dtype=np.uint8)
    pf = rng.random((B, L, H, Ta), dtype=np.float32)
    o = oracle_mod.Oracle(oracle_mod.make_cfg(B, L, H * g, H, D, Ta, Tt, cl, 2500, chunk_span=2), k, v, roles, pf)
    for step in range(4):
        q = f32_to_bf16(rng.standard_normal((B, L, H * g, D)).astype(np.float32))
        r = o.step(q)
        for b in range(B):
            segs = set()
            for c in r["selected"][b]:
                segs |= {int(c), int(c) + 1}
            assert segs <= set(np.nonzero(r["resident"][b])[0].tolist())
        for b, l, hq in itertools.product(range(B), range(L), range(H * g)):
            h = hq // g
            mask = np.ones(Ta + Tt, dtype=bool)
            if roles[l, h] != 0:
                keep = o.keep_mask(b, l, h).astype(bool)
                if roles[l, h] == 1:
                    keep |= np.repeat(r["resident"][b].astype(bool), cl // 2)[:Ta]
                mask[:Ta] = keep
            ref = _sdpa(q[b, l, hq], k[b, l, h], v[b, l, h], mask)
            np.testing.assert_allclose(r["out"][b, l, hq], ref, rtol=0, atol=1e-12)


def test_span2_selection_is_topk_of_fp32_scores(oracle_mod):
    o, k, v, roles, pf, q = _small(oracle_mod, seed=41, Ta=96, Tt=4, cl=8, budget=2500, chunk_span=2)
    for s in range(3):
        qs = f32_to_bf16(np.random.default_rng(300 + s).standard_normal(q.shape).astype(np.float32))
        r = o.step(qs)
        for b in range(q.shape[0]):
            assert list(r["selected"][b]) == _brute_topk(list(r["scores"][b].astype(np.float32)), o.k)


# ---- per-head retention (Eq. 1): retention = min(importance * lambda, 1) per tidal/fixed head

def _retention_case(oracle_mod, seed, imp, lam, B=2, D=8, Ta=70, Tt=3, cl=16, g=2, pf=None, **kw):
    rng = np.random.default_rng(seed)
    L, H = imp.shape
    k, v = _rand_cache(rng, B, L, H, Ta + Tt, D)
    roles = (np.arange(L * H).reshape(L, H) % 3).astype(np.uint8)   # anchor, tidal, fixed in turn
    if pf is None:
        pf = rng.random((B, L, H, Ta), dtype=np.float32)
    cfg = oracle_mod.make_cfg(B, L, H * g, H, D, Ta, Tt, cl, 2000, **kw)
    o = oracle_mod.Oracle(cfg, k, v, roles, pf, importance=imp, lam=lam)
    return o, k, v, roles, pf


def test_retention_keep_counts_follow_eq1(oracle_mod):
    """Per segment, floor(min(importance * lambda, 1) * len) positions are kept (exact rational
    arithmetic; the case has no product within 1e-9 of an integer), each outranking every
    dropped one; importance 0 keeps nothing, importance * lambda >= 1 keeps every position,
    anchors keep everything."""
    from fractions import Fraction
    rng = np.random.default_rng(41)
    L, H, Ta, cl = 3, 4, 70, 16
    imp = rng.random((L, H), dtype=np.float32)
    imp[0, 1], imp[1, 1], imp[2, 2] = 0.0, 1.0, 0.0
    lam = np.float32(0.7310585)
    pf = (rng.integers(0, 4, size=(2, L, H, Ta)) / 4.0).astype(np.float32)   # heavy ties
    o, k, v, roles, pf = _retention_case(oracle_mod, 5, imp, lam, Ta=Ta, cl=cl, pf=pf)
    lam2 = np.float32(3.0)
    o2, *_ = _retention_case(oracle_mod, 5, imp, lam2, Ta=Ta, cl=cl, pf=pf)
    for oo, lm in ((o, lam), (o2, lam2)):
        for b, l, h in itertools.product(range(2), range(L), range(H)):
            m = oo.keep_mask(b, l, h)
            if roles[l, h] == 0:
                assert m.all()
                continue
            r = min(Fraction(float(imp[l, h])) * Fraction(float(lm)), Fraction(1))
            for c0 in range(0, Ta, cl):
                seg = range(c0, min(c0 + cl, Ta))
                x = r * len(seg)
                assert x.denominator == 1 or abs(float(x - round(x))) > 1e-9
                kept = [t for t in seg if m[t]]
                drop = [t for t in seg if not m[t]]
                assert len(kept) == math.floor(x), (l, h, c0)
                for a in kept:
                    for d in drop:
                        assert (pf[b, l, h, a], -a) > (pf[b, l, h, d], -d)
    assert not o.keep_mask(0, 0, 1).any() and o.keep_mask(0, 1, 1).sum() == math.floor(float(lam) * 16) * 4 + math.floor(float(lam) * 6)
    assert o2.keep_mask(0, 1, 1).all()


def test_retention_uniform_importance_is_the_uniform_budget(oracle_mod):
    """importance 0.25 with lambda 1, and 0.5 with lambda 0.5, give retention 1/4 exactly: the
    keep sets and every output equal those of the uniform 25 % budget."""
    rng = np.random.default_rng(43)
    B, L, H, g, D, Ta, Tt, cl = 2, 2, 3, 2, 8, 64, 4, 8
    k, v = _rand_cache(rng, B, L, H, Ta + Tt, D)
    roles = np.array([[0, 1, 2], [1, 2, 0]], dtype=np.uint8)
    pf = rng.random((B, L, H, Ta), dtype=np.float32)
    cfg = oracle_mod.make_cfg(B, L, H * g, H, D, Ta, Tt, cl, 2500)
    ref = oracle_mod.Oracle(cfg, k, v, roles, pf)
    alts = [oracle_mod.Oracle(cfg, k, v, roles, pf, importance=np.full((L, H), s, np.float32), lam=lm)
            for s, lm in ((0.25, 1.0), (0.5, 0.5))]
    for b, l, h in itertools.product(range(B), range(L), range(H)):
        for a in alts:
            assert np.array_equal(a.keep_mask(b, l, h), ref.keep_mask(b, l, h))
    for step in range(3):
        q = f32_to_bf16(rng.standard_normal((B, L, H * g, D)).astype(np.float32))
        r0 = ref.step(q)
        for a in alts:
            r = a.step(q)
            assert np.array_equal(r["out"], r0["out"]) and np.array_equal(r["resident"], r0["resident"])


def test_retention_heads_attend_over_their_own_key_sets(oracle_mod):
    """Heterogeneous retention (including 0 and 1): every tidal head attends over its own kept
    rows + the resident chunks + text and every fixed head over its own kept rows + text (SDPA
    with that mask); a tidal or fixed head at retention 1 is plain attention."""
    rng = np.random.default_rng(47)
    L, H, Ta, Tt, cl, g = 2, 6, 64, 4, 8, 2
    imp = rng.random((L, H), dtype=np.float32)
    imp[0, 1], imp[0, 2], imp[1, 4] = 0.0, 1.0, 1.0       # tidal at 0, fixed at 1, tidal at 1
    o, k, v, roles, pf = _retention_case(oracle_mod, 9, imp, np.float32(1.0), Ta=Ta, Tt=Tt, cl=cl, g=g)
    assert roles[0, 1] == 1 and roles[0, 2] == 2 and roles[1, 4] == 1
    B = 2
    for step in range(4):
        q = f32_to_bf16(rng.standard_normal((B, L, H * g, 8)).astype(np.float32))
        r = o.step(q)
        for b, l, hq in itertools.product(range(B), range(L), range(H * g)):
            h = hq // g
            mask = np.ones(Ta + Tt, dtype=bool)
            if roles[l, h] != 0:
                keep = o.keep_mask(b, l, h).astype(bool)
                if roles[l, h] == 1:
                    keep |= np.repeat(r["resident"][b].astype(bool), cl)[:Ta]
                mask[:Ta] = keep
            ref = _sdpa(q[b, l, hq], k[b, l, h], v[b, l, h], mask)
            np.testing.assert_allclose(r["out"][b, l, hq], ref, rtol=0, atol=1e-12)
            if (l, h) in ((0, 2), (1, 4)):
                full = _sdpa(q[b, l, hq], k[b, l, h], v[b, l, h])
                np.testing.assert_allclose(r["out"][b, l, hq], full, rtol=0, atol=1e-12)


def test_retention_invalid_inputs_rejected(oracle_mod):
    rng = np.random.default_rng(1)
    k, v = _rand_cache(rng, 1, 1, 3, 20, 8)
    roles = np.array([[0, 1, 2]], dtype=np.uint8)
    pf = rng.random((1, 1, 3, 16), dtype=np.float32)
    cfg = oracle_mod.make_cfg(1, 1, 3, 3, 8, 16, 4, 8, 2000)
    for imp, lam in ((np.array([[0.5, 1.5, 0.5]]), 1.0), (np.array([[0.5, -0.1, 0.5]]), 1.0),
                     (np.array([[0.5, np.nan, 0.5]]), 1.0), (np.full((1, 3), 0.5), -1.0),
                     (np.full((1, 3), 0.5), np.inf), (np.full((1, 3), 0.5), np.nan)):
        with pytest.raises(ValueError):
            oracle_mod.Oracle(cfg, k, v, roles, pf, importance=imp.astype(np.float32), lam=lam)


# ---- prefill compression: text-to-audio attention sums and the global top-k variant

def _prefill_case(oracle_mod, seed, B=2, L=2, H=2, g=2, D=16, Ta=29, Tt=6, scale=1.0):
    rng = np.random.default_rng(seed)
    k, _ = _rand_cache(rng, B, L, H, Ta + Tt, D, scale=scale)
    q = f32_to_bf16(rng.standard_normal((B, L, H * g, Tt, D)).astype(np.float32) * scale)
    cfg = oracle_mod.make_cfg(B, L, H * g, H, D, Ta, Tt, 8, 2000)
    return cfg, k, q


def test_prefill_scores_equal_library_causal_attention(oracle_mod):
    """p equals causal SDPA (double) of the text queries over all rows with V = one-hot audio
    indicators, summed over the text tokens and the q-heads of each KV-head."""
    cfg, k, q = _prefill_case(oracle_mod, 51, scale=2.0)
    p = oracle_mod.prefill_scores(cfg, k, q)
    B, L, H, Ta, Tt, g = cfg.batch, cfg.layers, cfg.kv_heads, cfg.audio_len, cfg.text_len, cfg.q_heads // cfg.kv_heads
    T = Ta + Tt
    onehot = np.zeros((T, Ta))
    onehot[np.arange(Ta), np.arange(Ta)] = 1.0
    mask = np.zeros((Tt, T), dtype=bool)
    for t in range(Tt):
        mask[t, : Ta + t + 1] = True
    f = lambda a: torch.from_numpy(bf16_to_f32(a).astype(np.float64))
    for b, l, kv in itertools.product(range(B), range(L), range(H)):
        ref = np.zeros(Ta)
        for j in range(g):
            o = torch.nn.functional.scaled_dot_product_attention(
                f(q[b, l, kv * g + j])[None], f(k[b, l, kv])[None], torch.from_numpy(onehot)[None],
                attn_mask=torch.from_numpy(mask)[None])[0].numpy()
            ref += o.sum(axis=0)
        np.testing.assert_allclose(p[b, l, kv], ref, rtol=0, atol=1e-12)


def test_prefill_scores_zero_queries_closed_form(oracle_mod):
    """q = 0: text token t spreads its weight evenly over its T_a + t + 1 keys, so every audio
    position gets g * sum_t 1 / (T_a + t + 1); no text gives p = 0."""
    cfg, k, q = _prefill_case(oracle_mod, 53)
    q[:] = 0
    p = oracle_mod.prefill_scores(cfg, k, q)
    g, Ta, Tt = cfg.q_heads // cfg.kv_heads, cfg.audio_len, cfg.text_len
    np.testing.assert_allclose(p, g * sum(1.0 / (Ta + t + 1) for t in range(Tt)), rtol=1e-14, atol=0)
    cfg0 = oracle_mod.make_cfg(1, 1, 2, 1, 16, 10, 0, 4, 2000)
    k0 = f32_to_bf16(np.random.default_rng(1).standard_normal((1, 1, 1, 10, 16)).astype(np.float32))
    assert not oracle_mod.prefill_scores(cfg0, k0, np.zeros((1, 1, 2, 0, 16), np.uint16)).any()


def test_prefill_global_keep_is_brute_force_top(oracle_mod):
    """Global variant: the per-segment total of floor(retention * len) positions, the best over
    the whole audio by (score desc, position asc); with one segment it equals per-segment
    selection."""
    rng = np.random.default_rng(55)
    B, L, H, D, Ta, Tt, cl, budget = 2, 1, 3, 8, 70, 2, 16, 3000
    k, v = _rand_cache(rng, B, L, H, Ta + Tt, D)
    pf = (rng.integers(0, 6, size=(B, L, H, Ta)) / 6.0).astype(np.float32)   # ties
    roles = np.array([[0, 1, 2]], dtype=np.uint8)
    o = oracle_mod.Oracle(oracle_mod.make_cfg(B, L, H, H, D, Ta, Tt, cl, budget, prefill_global=1), k, v, roles, pf)
    total = sum((budget * (min(c0 + cl, Ta) - c0)) // 10000 for c0 in range(0, Ta, cl))
    for b, h in itertools.product(range(B), range(1, H)):
        order = sorted(range(Ta), key=lambda t: (-float(pf[b, 0, h, t]), t))
        want = np.zeros(Ta, dtype=np.uint8)
        want[order[:total]] = 1
        assert np.array_equal(o.keep_mask(b, 0, h), want)
    one = dict(B=1, L=1, H=3, D=8, Ta=14, Tt=2, cl=16)
    k1, v1 = _rand_cache(rng, 1, 1, 3, 16, 8)
    pf1 = rng.random((1, 1, 3, 14), dtype=np.float32)
    a = oracle_mod.Oracle(oracle_mod.make_cfg(1, 1, 3, 3, 8, 14, 2, 16, 4000, prefill_global=1), k1, v1, roles, pf1)
    s = oracle_mod.Oracle(oracle_mod.make_cfg(1, 1, 3, 3, 8, 14, 2, 16, 4000), k1, v1, roles, pf1)
    for h in range(3):
        assert np.array_equal(a.keep_mask(0, 0, h), s.keep_mask(0, 0, h))


# ---- decode-time append: generated tokens join every head's key set, kept in full like text

def test_append_equals_extra_text_rows(oracle_mod):
    """Appending a token's K/V rows is the same as having them as trailing text rows: after one
    append the step equals a fresh oracle with one more text row; after a second append (and
    the same selection history) it equals one with two more, bit for bit."""
    rng = np.random.default_rng(61)
    B, L, H, g, D, Ta, Tt, cl = 2, 2, 3, 2, 8, 64, 4, 8
    roles = np.array([[0, 1, 2], [1, 2, 0]], dtype=np.uint8)
    k, v = _rand_cache(rng, B, L, H, Ta + Tt + 2, D)
    pf = rng.random((B, L, H, Ta), dtype=np.float32)
    q1, q2 = (f32_to_bf16(rng.standard_normal((B, L, H * g, D)).astype(np.float32)) for _ in range(2))
    mk = lambda tt, mx: oracle_mod.make_cfg(B, L, H * g, H, D, Ta, tt, cl, 2500, max_new=mx)
    a = oracle_mod.Oracle(mk(Tt, 2), k[:, :, :, : Ta + Tt], v[:, :, :, : Ta + Tt], roles, pf)
    a.append(k[:, :, :, Ta + Tt], v[:, :, :, Ta + Tt])
    ra1 = a.step(q1)
    b1 = oracle_mod.Oracle(mk(Tt + 1, 0), k[:, :, :, : Ta + Tt + 1], v[:, :, :, : Ta + Tt + 1], roles, pf)
    rb1 = b1.step(q1)
    for key in ("out", "scores", "selected", "resident"):
        assert np.array_equal(ra1[key], rb1[key]), key
    a.append(k[:, :, :, Ta + Tt + 1], v[:, :, :, Ta + Tt + 1])
    ra2 = a.step(q2)
    b2 = oracle_mod.Oracle(mk(Tt + 2, 0), k, v, roles, pf)
    b2.step(q1, forced=ra1["selected"])
    rb2 = b2.step(q2)
    for key in ("out", "scores", "selected", "resident"):
        assert np.array_equal(ra2[key], rb2[key]), key
    with pytest.raises(ValueError):
        a.append(k[:, :, :, 0], v[:, :, :, 0])


def test_appended_rows_in_every_key_set(oracle_mod):
    """After appends every head attends over its key set plus the appended rows (SDPA with the
    mask), and a dominant appended key takes a head's whole weight."""
    rng = np.random.default_rng(63)
    B, L, H, g, D, Ta, Tt, cl = 2, 2, 3, 2, 16, 64, 4, 8
    roles = np.array([[0, 1, 2], [1, 2, 0]], dtype=np.uint8)
    k, v = _rand_cache(rng, B, L, H, Ta + Tt, D)
    pf = rng.random((B, L, H, Ta), dtype=np.float32)
    o = oracle_mod.Oracle(oracle_mod.make_cfg(B, L, H * g, H, D, Ta, Tt, cl, 2500, max_new=3), k, v, roles, pf)
    kn, vn = [], []
    for step in range(3):
        q = f32_to_bf16(rng.standard_normal((B, L, H * g, D)).astype(np.float32))
        kk = f32_to_bf16(rng.standard_normal((B, L, H, D)).astype(np.float32))
        if step == 2:
            kk = f32_to_bf16(bf16_to_f32(q[:, :, ::g]) * 40.0)   # aligned with q-head 0 of each KV-head
        vv = f32_to_bf16(rng.standard_normal((B, L, H, D)).astype(np.float32))
        kn.append(kk)
        vn.append(vv)
        o.append(kk, vv)
        r = o.step(q)
        K = np.concatenate([k, np.stack(kn, axis=3)], axis=3)
        V = np.concatenate([v, np.stack(vn, axis=3)], axis=3)
        T = Ta + Tt + step + 1
        for b, l, hq in itertools.product(range(B), range(L), range(H * g)):
            h = hq // g
            mask = np.ones(T, dtype=bool)
            if roles[l, h] != 0:
                keep = o.keep_mask(b, l, h).astype(bool)
                if roles[l, h] == 1:
                    keep |= np.repeat(r["resident"][b].astype(bool), cl)[:Ta]
                mask[:Ta] = keep
            ref = _sdpa(q[b, l, hq], K[b, l, h], V[b, l, h], mask)
            np.testing.assert_allclose(r["out"][b, l, hq], ref, rtol=0, atol=1e-12)
            if step == 2 and hq % g == 0:
                np.testing.assert_allclose(r["out"][b, l, hq], bf16_to_f32(vv[b, l, h]), rtol=0, atol=1e-6)


# ---- head triage arithmetic: voice-score hits, key sensitivity, VS x HS roles

def _basis_keys(L, H, T, d, mags):
    """Key tau = mags[tau] * e_(tau mod d) (exact in bf16 for the magnitudes used)."""
    k = np.zeros((L, H, T, d), dtype=np.float32)
    for tau in range(T):
        k[:, :, tau, tau % d] = mags[tau]
    return f32_to_bf16(k)


def test_voice_hits_planted_top_positions(oracle_mod):
    """Keys are scaled basis vectors, so a query's logits are known in closed form: the query
    e_j weights position tau by mags[tau] when tau = j (mod d) and 0 otherwise.  The top-K are then
    the K largest magnitudes on residue j (ties to the lower position), and hits count those inside
    the span; K = T_a ranks every position, a span over all audio gives K hits."""
    L, H, g, d, Ta, Tt = 1, 2, 2, 8, 40, 3
    mags = np.array([1 + (tau * 7) % 11 for tau in range(Ta + Tt)], dtype=np.float32)
    mags[[3, 11]] = 12.0                       # a tie on residue 3: position 3 ranks before 11
    k = _basis_keys(L, H, Ta + Tt, d, mags)
    q = np.zeros((4, L, H * g, d), dtype=np.float32)
    resid = [3, 5, 0, 7]
    for t, j in enumerate(resid):
        q[t, :, :, j] = 1.0
    q = f32_to_bf16(q)
    span = np.array([[0, 10], [20, 40], [0, 40], [39, 40]], dtype=np.int32)
    for K in (1, 3, 5):
        hits = oracle_mod.voice_hits(k, q, span, K, Ta)
        for t, j in enumerate(resid):
            cand = sorted([tau for tau in range(Ta) if tau % d == j], key=lambda tau: (-mags[tau], tau))
            top = cand[:K] + [tau for tau in range(Ta) if tau % d != j][: max(0, K - len(cand))]
            want = sum(span[t, 0] <= tau < span[t, 1] for tau in top)
            assert (hits[t] == want).all(), (K, t)
    assert (oracle_mod.voice_hits(k, q, np.array([[0, Ta]] * 4, np.int32), 5, Ta) == 5).all()
    full = oracle_mod.voice_hits(k, q, span, Ta, Ta)
    assert (full[:, 0, 0] == np.minimum(span[:, 1], Ta) - span[:, 0]).all()
    one = oracle_mod.voice_hits(k, q[:1], np.array([[11, 12]], np.int32), 1, Ta)
    assert (one == 0).all()                    # the tie went to position 3


def test_key_sensitivity_closed_forms(oracle_mod):
    """A gradient of constant entries c has norm |c| sqrt(d) at every position; the measure is
    linear in the gradient's scale and the mean over positions of per-position norms."""
    n, L, H, Ta, d = 2, 2, 3, 5, 16
    grad = np.zeros((n, L, H, Ta, d), dtype=np.float32)
    c = np.arange(1, n * L * H + 1, dtype=np.float32).reshape(n, L, H)
    grad += c[..., None, None]
    np.testing.assert_allclose(oracle_mod.key_sensitivity(grad), c * np.sqrt(d), rtol=1e-14)
    grad2 = np.zeros_like(grad)
    grad2[:, :, :, 0, 0] = 3.0
    grad2[:, :, :, 1, :2] = 4.0 / np.sqrt(2.0)                    # norm 4
    np.testing.assert_allclose(oracle_mod.key_sensitivity(grad2), (3.0 + 4.0) / Ta, rtol=1e-6)
    np.testing.assert_allclose(oracle_mod.key_sensitivity(-2.5 * grad2), 2.5 * (3.0 + 4.0) / Ta, rtol=1e-6)


def test_triage_hand_worked_example(oracle_mod):
    with open(os.path.join(GOLD, "triage_example.json")) as f:
        ex = json.load(f)
    roles, vs, hs, imp = oracle_mod.triage(np.array(ex["hits"]), ex["K"], np.array(ex["sens"]), np.array(ex["sample"]),
                                           ex["n_voice"], ex["n_anchor"])
    np.testing.assert_allclose(vs, ex["vs"], rtol=0, atol=1e-15)
    np.testing.assert_allclose(hs, ex["hs"], rtol=0, atol=1e-15)
    assert roles.tolist() == ex["roles"]
    np.testing.assert_allclose(imp, ex["importance_norm"], rtol=0, atol=1e-15)


def test_triage_ranking_counts_and_normalisation(oracle_mod):
    """Random scores: exactly n_anchor anchors and n_voice - n_anchor tidal heads, every anchor
    outranks every tidal head, which outranks every fixed head by VS * HS; the normalised
    importance peaks at 1 on the best head."""
    rng = np.random.default_rng(71)
    n, L, H, g = 6, 3, 4, 2
    hits = rng.integers(0, 5, size=(n, L, H * g)).astype(np.int32)
    sens = rng.random((n, L, H))
    sample = np.array([0, 0, 1, 1, 1, 2], dtype=np.int32)
    roles, vs, hs, imp = oracle_mod.triage(hits, 4, sens, sample, 7, 2)
    assert (roles == 0).sum() == 2 and (roles == 1).sum() == 5 and (roles == 2).sum() == L * H - 7
    prod = vs * hs
    assert prod[roles == 0].min() >= prod[roles == 1].max() >= prod[roles == 2].max() - 0.0
    assert abs(imp.max() - 1.0) < 1e-15 and np.argmax(imp) == np.argmax(prod)
