"""Seeded synthetic inputs for the WnW decode step.

This module only draws inputs: KV caches, decode-step queries, head roles and prefill
scores.  It holds none of the method's arithmetic (no attention, no chunking, no
selection), so both the CPU oracle and the HIP path can consume what it produces.

Recipe (one sequence b of workload w; every stream is an independent Philox generator keyed
by (seed, tag, indices), so any (layer, KV-head) slice regenerates on its own):

* seed = 260822704 + 1000 * w.seed_id + b.
* K_raw, V ~ N(0, 1) in fp32, shape [T_a + T_t][d] per (layer, KV-head), audio rows first.
* drift(s): the audio position the queries are pulled towards at step s.  With one step it is
  uniform over the audio; otherwise it advances uniformly across the clip,
  floor(s * T_a / S) + U{0 .. floor(T_a / S) - 1}, clipped to T_a - 1.
* u(l, kv): the mean query direction of the KV-head's group.  The query noise has zero mean,
  so the mean query is drift_gain times the mean of K_raw over the drift positions; u is that
  mean, normalised.
* sink: the first ``sink_len`` audio keys get + sink_gain * u.
* K and V are rounded to bf16 (round to nearest even); the rounded values are the cache.
* q(s, l, hq) = bf16(z + drift_gain * K[l, kv(hq), drift(s)]), z ~ N(0, 1) fresh each step.
* roles: a seeded permutation of the L * H_kv KV-heads; the first n_anchor are anchor (0),
  the next n_tidal tidal (1), the rest fixed (2).  Shared by every sequence of the batch.
* prefill scores: U(0, 1) fp32 per (layer, KV-head, audio position); they stand in for the
  summed text-to-audio prefill attention that ranks positions at prefill.

bf16 values are carried as uint16 bit patterns.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .configs import Workload

TAG_K, TAG_V, TAG_Z, TAG_DRIFT, TAG_ROLES, TAG_PREFILL, TAG_IMPORTANCE = 1, 2, 3, 4, 5, 6, 7
TAG_QTEXT, TAG_QTEXT_POS = 8, 9
ANCHOR, TIDAL, FIXED = 0, 1, 2


def default_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def seed_base(w: Workload) -> int:
    return 260822704 + 1000 * w.seed_id


def seq_seed(w: Workload, b: int) -> int:
    return seed_base(w) + b


def _rng(seed: int, tag: int, *idx: int) -> np.random.Generator:
    return np.random.Generator(np.random.Philox(np.random.SeedSequence([seed, tag, *idx])))


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_to_f32(h: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def roles(w: Workload) -> np.ndarray:
    """uint8 [L][H_kv] role table (0 anchor, 1 tidal, 2 fixed)."""
    n = w.layers * w.kv_heads
    assert w.n_anchor + w.n_tidal + w.n_fixed == n
    perm = _rng(seed_base(w), TAG_ROLES).permutation(n)
    r = np.empty(n, dtype=np.uint8)
    r[perm[: w.n_anchor]] = ANCHOR
    r[perm[w.n_anchor: w.n_anchor + w.n_tidal]] = TIDAL
    r[perm[w.n_anchor + w.n_tidal:]] = FIXED
    return r.reshape(w.layers, w.kv_heads)


def drift(w: Workload, b: int) -> np.ndarray:
    """int64 [S] drift positions of sequence b."""
    g = _rng(seq_seed(w, b), TAG_DRIFT)
    s_n, ta = w.steps, w.audio_len
    if s_n == 1:
        return g.integers(0, ta, size=1).astype(np.int64)
    width = max(ta // s_n, 1)
    base = (np.arange(s_n, dtype=np.int64) * ta) // s_n
    return np.minimum(base + g.integers(0, width, size=s_n), ta - 1).astype(np.int64)


def head_kv(w: Workload, b: int, l: int, kv: int, drift_pos: np.ndarray):
    """(K, V) uint16 [T][d] of one (layer, KV-head), sink included, bf16-rounded."""
    seed = seq_seed(w, b)
    shape = (w.total_len, w.head_dim)
    k = _rng(seed, TAG_K, l, kv).standard_normal(shape, dtype=np.float32)
    v = _rng(seed, TAG_V, l, kv).standard_normal(shape, dtype=np.float32)
    ns = min(w.sink_len, w.audio_len)
    if ns > 0 and w.sink_gain != 0.0:
        u = k[drift_pos].astype(np.float64).mean(axis=0)
        nrm = float(np.linalg.norm(u))
        if nrm > 0.0:
            k[:ns] += np.float32(w.sink_gain) * (u / nrm).astype(np.float32)
    return f32_to_bf16(k), f32_to_bf16(v)


def head_queries(w: Workload, b: int, l: int, kv: int, k_bf16: np.ndarray, drift_pos: np.ndarray):
    """uint16 [S][g][d] queries of the q-heads of one KV-head."""
    seed = seq_seed(w, b)
    kd = bf16_to_f32(k_bf16[drift_pos])                 # [S][d]
    out = np.empty((len(drift_pos), w.group, w.head_dim), dtype=np.uint16)
    for j in range(w.group):
        hq = kv * w.group + j
        z = _rng(seed, TAG_Z, l, hq).standard_normal((len(drift_pos), w.head_dim), dtype=np.float32)
        out[:, j, :] = f32_to_bf16(z + np.float32(w.drift_gain) * kd)
    return out


def prefill_scores(w: Workload, b: int, l: int, kv: int) -> np.ndarray:
    return _rng(seq_seed(w, b), TAG_PREFILL, l, kv).random(w.audio_len, dtype=np.float32)


def text_queries(w: Workload, b: int, l: int, kv: int, k_bf16: np.ndarray) -> np.ndarray:
    """uint16 [g][T_t][d]: the text tokens' queries at prefill for the q-heads of one KV-head,
    built like the decode queries: N(0,1) noise plus drift_gain times the key of one audio
    position drawn uniformly per (q-head, token)."""
    seed = seq_seed(w, b)
    out = np.empty((w.group, w.text_len, w.head_dim), dtype=np.uint16)
    for j in range(w.group):
        hq = kv * w.group + j
        z = _rng(seed, TAG_QTEXT, l, hq).standard_normal((w.text_len, w.head_dim), dtype=np.float32)
        if w.audio_len > 0:
            pos = _rng(seed, TAG_QTEXT_POS, l, hq).integers(0, w.audio_len, size=w.text_len)
            z += np.float32(w.drift_gain) * bf16_to_f32(k_bf16[pos])
        out[j] = f32_to_bf16(z)
    return out


def importance(w: Workload) -> np.ndarray:
    """Normalised per-head importance [L][H_kv] fp32, U(0, 1), shared by the batch (the input of
    the per-head retention schedule; calibration, which would produce it, is not modelled)."""
    return _rng(seed_base(w), TAG_IMPORTANCE).random((w.layers, w.kv_heads), dtype=np.float32)


def _head_job(w, b, l, kv, dpos):
    k, v = head_kv(w, b, l, kv, dpos)
    return k, v, head_queries(w, b, l, kv, k, dpos), prefill_scores(w, b, l, kv)


def iter_layers(w: Workload, b: int, threads: int | None = None, layers_per_batch: int = 2):
    """Yield (l, K [H_kv][T][d], V, q [S][g*H_kv][d], prefill [H_kv][T_a]) layer by layer.

    Memory stays bounded to ``layers_per_batch`` layers; generation runs on a thread pool
    (numpy releases the GIL while drawing)."""
    dpos = drift(w, b)
    threads = threads or default_threads()
    with ThreadPoolExecutor(threads) as ex:
        for l0 in range(0, w.layers, layers_per_batch):
            ls = range(l0, min(w.layers, l0 + layers_per_batch))
            futs = {(l, kv): ex.submit(_head_job, w, b, l, kv, dpos) for l in ls for kv in range(w.kv_heads)}
            for l in ls:
                res = [futs[(l, kv)].result() for kv in range(w.kv_heads)]
                k = np.stack([r[0] for r in res])
                v = np.stack([r[1] for r in res])
                q = np.concatenate([r[2] for r in res], axis=1)     # [S][H_q][d]
                pf = np.stack([r[3] for r in res])
                yield l, k, v, q, pf


def sequence(w: Workload, b: int, threads: int | None = None) -> dict:
    """Whole sequence b: k, v uint16 [L][H_kv][T][d]; q uint16 [S][L][H_q][d];
    prefill fp32 [L][H_kv][T_a]; drift int64 [S]."""
    L, H, T, D, S = w.layers, w.kv_heads, w.total_len, w.head_dim, w.steps
    k = np.empty((L, H, T, D), dtype=np.uint16)
    v = np.empty_like(k)
    q = np.empty((S, L, w.q_heads, D), dtype=np.uint16)
    pf = np.empty((L, H, w.audio_len), dtype=np.float32)
    for l, kl, vl, ql, pl in iter_layers(w, b, threads):
        k[l], v[l], q[:, l], pf[l] = kl, vl, ql, pl
    return {"k": k, "v": v, "q": q, "prefill": pf, "drift": drift(w, b)}
