"""Workload shapes for the WnW decode step (synthetic stand-ins, no method arithmetic).

Each workload is the shape of a speech-LLM KV cache at decode time: a number of decoder
layers, query/KV heads with a grouped-query ratio, a head dimension, an audio region of
T_a positions followed by T_t text positions, a chunk length, an on-GPU audio budget and a
number of decode steps.  The backbone shapes are those the paper lists in its notation
paragraph (Voxtral-mini-3b: 30 layers, 32 query / 8 KV heads; Qwen2.5-Omni-3B: 36 layers,
16 query / 2 KV heads); the audio lengths correspond to 10 and 60 minutes of audio at the
frame rates the paper quotes in its introduction (12.5-25 tokens per second).  The paper does
not state the head dimension; 128 is used throughout.

Roles are given as counts over the layers x KV-heads grid (anchor / tidal / fixed).  Which
(layer, KV-head) gets which role is drawn by ``synth.gen.roles``.
"""
from __future__ import annotations

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class Workload:
    name: str
    seed_id: int          # selects the seed base, see synth.gen.seed_base
    batch: int
    layers: int
    q_heads: int
    kv_heads: int
    head_dim: int
    audio_len: int        # T_a
    text_len: int         # T_t
    chunk_len: int        # tokens per chunk (disjoint chunks)
    budget_bp: int        # on-GPU audio budget in basis points (2000 = 20 %)
    steps: int            # decode steps in the workload
    n_anchor: int
    n_tidal: int
    n_fixed: int
    sink_len: int = 16    # first audio keys pushed along the mean query direction
    sink_gain: float = 3.0
    drift_gain: float = 2.0

    @property
    def group(self) -> int:
        return self.q_heads // self.kv_heads

    @property
    def total_len(self) -> int:
        return self.audio_len + self.text_len

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


def _split(n: int) -> tuple[int, int, int]:
    """10 % anchor / 50 % tidal / rest fixed over n KV-heads (round half to even)."""
    a = round(0.1 * n)
    t = round(0.5 * n)
    return a, t, n - a - t


def _mk(name, seed_id, batch, layers, hq, hkv, ta, tt, chunk, budget, steps, roles=None):
    a, t, f = roles if roles is not None else _split(layers * hkv)
    return Workload(name, seed_id, batch, layers, hq, hkv, 128, ta, tt, chunk, budget, steps, a, t, f)


# Single layer, 8 KV heads (GQA 3), 1000 audio + 64 text, chunk 32, 20 %, one step.
TINY = _mk("tiny_1L_8kv_1k", 1, 1, 1, 24, 8, 1000, 64, 32, 2000, 1, roles=(2, 4, 2))
# Qwen2.5-Omni-3B-shaped cache, 10 min of audio at 12.5 tok/s.
QWEN_10MIN = _mk("qwen3b_36L_2kv_7.5k", 2, 1, 36, 16, 2, 7500, 256, 32, 2000, 128)
# Voxtral-mini-3B-shaped cache, 10 min of audio at 25 tok/s (the headline workload).
VOXTRAL_10MIN = _mk("voxtral3b_30L_8kv_15k", 3, 1, 30, 32, 8, 15000, 512, 64, 2000, 256)
# Same cache at batch 16, independent sequences.
VOXTRAL_10MIN_B16 = _mk("voxtral3b_30L_8kv_15k_b16", 4, 16, 30, 32, 8, 15000, 512, 64, 2000, 256)
# Long-form stress: 60 min at 25 tok/s, batch 4, chunk 128, budgets 20 % and 10 %.
VOXTRAL_60MIN_B4_20 = _mk("voxtral3b_30L_8kv_90k_b4_20pct", 5, 4, 30, 32, 8, 90000, 1024, 128, 2000, 512)
VOXTRAL_60MIN_B4_10 = VOXTRAL_60MIN_B4_20.with_(name="voxtral3b_30L_8kv_90k_b4_10pct", budget_bp=1000)

ALL = [TINY, QWEN_10MIN, VOXTRAL_10MIN, VOXTRAL_10MIN_B16, VOXTRAL_60MIN_B4_20, VOXTRAL_60MIN_B4_10]
BY_NAME = {w.name: w for w in ALL}
HEADLINE = VOXTRAL_10MIN
