"""The seeded workload generator: determinism, bf16 rounding, structure of the inputs."""
import numpy as np

from synth import configs, gen


def test_bf16_round_to_nearest_even():
    x = np.array([1.0, 1.0 + 2**-8, 1.0 + 3 * 2**-8, 1.0 + 2**-8 + 2**-20, -2.5, 0.0], dtype=np.float32)
    want = np.array([1.0, 1.0, 1.0 + 4 * 2**-8, 1.0 + 2**-7, -2.5, 0.0], dtype=np.float32)
    np.testing.assert_array_equal(gen.bf16_to_f32(gen.f32_to_bf16(x)), want)


def test_sequences_are_deterministic_and_independent():
    w = configs.TINY.with_(steps=3)
    a, b = gen.sequence(w, 0), gen.sequence(w, 0)
    for key in a:
        np.testing.assert_array_equal(a[key], b[key])
    c = gen.sequence(w, 1)
    assert not np.array_equal(a["k"], c["k"])
    # one (layer, kv-head) slice regenerates on its own
    k1, v1 = gen.head_kv(w, 0, 0, 3, a["drift"])
    np.testing.assert_array_equal(k1, a["k"][0, 3])
    np.testing.assert_array_equal(v1, a["v"][0, 3])


def test_roles_counts_and_sharing():
    for w in configs.ALL:
        r = gen.roles(w)
        assert r.shape == (w.layers, w.kv_heads)
        assert [(r == i).sum() for i in range(3)] == [w.n_anchor, w.n_tidal, w.n_fixed]
    assert (configs.VOXTRAL_10MIN.n_anchor, configs.VOXTRAL_10MIN.n_tidal) == (24, 120)
    assert (configs.QWEN_10MIN.n_anchor, configs.QWEN_10MIN.n_tidal, configs.QWEN_10MIN.n_fixed) == (7, 36, 29)


def test_drift_advances_across_the_clip():
    w = configs.VOXTRAL_10MIN
    d = gen.drift(w, 0)
    assert len(d) == w.steps and d.min() >= 0 and d.max() < w.audio_len
    width = w.audio_len // w.steps
    assert (d >= (np.arange(w.steps) * w.audio_len) // w.steps).all()
    assert (d < (np.arange(w.steps) * w.audio_len) // w.steps + width).all()


def test_queries_pull_towards_drift_key_and_sink():
    w = configs.TINY
    s = gen.sequence(w, 0)
    k = gen.bf16_to_f32(s["k"][0]).astype(np.float64)       # [H][T][d]
    q = gen.bf16_to_f32(s["q"][0, 0]).astype(np.float64)    # [Hq][d]
    d = int(s["drift"][0])
    for hq in range(w.q_heads):
        logits = k[hq // w.group] @ q[hq]
        assert logits.argmax() == d                       # 2 |K|^2 dominates the noise
    # sink keys carry + 3 u: their mean projection on u is ~3 above the other audio keys
    kr = k[0]
    u = kr[:16].mean(0) - kr[16:1000].mean(0)
    assert np.linalg.norm(u) > 2.5
