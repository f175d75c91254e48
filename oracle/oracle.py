"""ctypes wrapper of the WnW CPU oracle (plain C, double precision), TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use
this module.  It neither imports nor links anything of the HIP library.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "wnw_oracle.c")
LIB = os.path.join(HERE, "libwnw_oracle.so")


def build(verbose: bool = False) -> str:
    """Compile the oracle with gcc (C99, OpenMP)."""
    tmp = f"{LIB}.tmp{os.getpid()}"
    cmd = ["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra", "-o", tmp, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


class _Cfg(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "batch", "layers", "q_heads", "kv_heads", "head_dim", "audio_len", "text_len",
        "chunk_len", "budget_bp", "top_k", "evict_lag", "next_step", "chunk_span", "prefill_global", "max_new")]


_lib = None


def lib():
    global _lib
    if _lib is None:
        # WNW_ORACLE_LIB lets the mutation tests load a deliberately broken copy of the oracle.
        path = os.environ.get("WNW_ORACLE_LIB") or LIB
        if path == LIB and not os.path.exists(LIB):
            build()
        L = C.CDLL(path)
        P = C.c_void_p
        L.wnwo_geometry.argtypes = [C.POINTER(_Cfg), C.POINTER(C.c_int32), C.POINTER(C.c_int32), C.POINTER(C.c_int32)]
        L.wnwo_create.argtypes = [C.POINTER(_Cfg), P, P, P, P]
        L.wnwo_create.restype = P
        L.wnwo_create_retention.argtypes = [C.POINTER(_Cfg), P, P, P, P, P, C.c_float]
        L.wnwo_create_retention.restype = P
        L.wnwo_destroy.argtypes = [P]
        L.wnwo_keep_mask.argtypes = [P, C.c_int32, C.c_int32, C.c_int32, P]
        L.wnwo_step.argtypes = [P, P, P, P, P, P, P, P, P]
        L.wnwo_topk.argtypes = [P, C.c_int32, C.c_int32, P]
        L.wnwo_tokens_for_window.argtypes = [C.c_double, C.c_double]
        L.wnwo_tokens_for_window.restype = C.c_int32
        L.wnwo_segments.argtypes = [C.POINTER(_Cfg), C.POINTER(C.c_int32)]
        L.wnwo_prefill_scores.argtypes = [C.POINTER(_Cfg), P, P, P]
        L.wnwo_append.argtypes = [P, P, P]
        I = C.c_int32
        L.wnwo_voice_hits.argtypes = [I, I, I, I, I, I, I, P, P, P, I, P]
        L.wnwo_key_sensitivity.argtypes = [I, I, I, I, I, P, P]
        L.wnwo_triage.argtypes = [I, I, I, I, P, P, I, P, I, I, P, P, P, P]
        L.wnwo_set_threads.argtypes = [C.c_int]
        L.wnwo_set_threads.restype = C.c_int
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def make_cfg(batch, layers, q_heads, kv_heads, head_dim, audio_len, text_len, chunk_len,
             budget_bp, top_k=0, evict_lag=0, next_step=0, chunk_span=1, prefill_global=0, max_new=0) -> _Cfg:
    return _Cfg(batch, layers, q_heads, kv_heads, head_dim, audio_len, text_len, chunk_len,
                budget_bp, top_k, evict_lag, next_step, chunk_span, prefill_global, max_new)


def cfg_from_workload(w, batch=None, **over) -> _Cfg:
    kw = dict(batch=batch or w.batch, layers=w.layers, q_heads=w.q_heads, kv_heads=w.kv_heads,
              head_dim=w.head_dim, audio_len=w.audio_len, text_len=w.text_len,
              chunk_len=w.chunk_len, budget_bp=w.budget_bp)
    kw.update(over)
    return make_cfg(**kw)


def geometry(cfg: _Cfg):
    n, k, kt = C.c_int32(), C.c_int32(), C.c_int32()
    if lib().wnwo_geometry(C.byref(cfg), C.byref(n), C.byref(k), C.byref(kt)):
        raise ValueError("invalid oracle configuration")
    return n.value, k.value, kt.value


def segments(cfg: _Cfg) -> int:
    n = C.c_int32()
    if lib().wnwo_segments(C.byref(cfg), C.byref(n)):
        raise ValueError("invalid oracle configuration")
    return n.value


def topk(scores: np.ndarray, k: int) -> np.ndarray:
    s = np.ascontiguousarray(scores, dtype=np.float32)
    out = np.empty(max(k, 1), dtype=np.int32)
    if lib().wnwo_topk(_ptr(s), len(s), k, _ptr(out)):
        raise ValueError("bad top-k arguments")
    return out[:k]


def tokens_for_window(seconds: float, rate: float) -> int:
    return lib().wnwo_tokens_for_window(seconds, rate)


def prefill_scores(cfg: _Cfg, k, q_text) -> np.ndarray:
    """Text-to-audio attention sums [B][L][H_kv][T_a] (double) of Prefill Compression."""
    k = np.ascontiguousarray(k, dtype=np.uint16)
    q = np.ascontiguousarray(q_text, dtype=np.uint16)
    B, L, H, Hq, Ta, Tt, D = cfg.batch, cfg.layers, cfg.kv_heads, cfg.q_heads, cfg.audio_len, cfg.text_len, cfg.head_dim
    assert k.shape == (B, L, H, Ta + Tt, D) and q.shape == (B, L, Hq, Tt, D)
    p = np.empty((B, L, H, Ta), dtype=np.float64)
    if lib().wnwo_prefill_scores(C.byref(cfg), _ptr(k), _ptr(q), _ptr(p)):
        raise ValueError("wnwo_prefill_scores failed")
    return p


def voice_hits(k, q, span, K, audio_len) -> np.ndarray:
    """k uint16 [L][H_kv][T][d], q uint16 [n_tok][L][H_q][d], span int32 [n_tok][2] ->
    hits int32 [n_tok][L][H_q]."""
    k = np.ascontiguousarray(k, dtype=np.uint16)
    q = np.ascontiguousarray(q, dtype=np.uint16)
    span = np.ascontiguousarray(span, dtype=np.int32)
    L, Hkv, T, d = k.shape
    n_tok, _, Hq, _ = q.shape
    out = np.empty((n_tok, L, Hq), dtype=np.int32)
    if lib().wnwo_voice_hits(L, Hq, Hkv, d, T, audio_len, n_tok, _ptr(k), _ptr(q), _ptr(span), K, _ptr(out)):
        raise ValueError("wnwo_voice_hits failed")
    return out


def key_sensitivity(grad) -> np.ndarray:
    """grad fp32 [n_tok][L][H_kv][T_a][d] -> sens double [n_tok][L][H_kv]."""
    g = np.ascontiguousarray(grad, dtype=np.float32)
    n_tok, L, Hkv, Ta, d = g.shape
    out = np.empty((n_tok, L, Hkv), dtype=np.float64)
    if lib().wnwo_key_sensitivity(L, Hkv, d, Ta, n_tok, _ptr(g), _ptr(out)):
        raise ValueError("wnwo_key_sensitivity failed")
    return out


def triage(hits, K, sens, sample, n_voice, n_anchor):
    """hits int32 [n][L][H_q], sens [n][L][H_kv], sample int32 [n] -> (roles uint8, vs, hs,
    importance_norm), each [L][H_kv]."""
    hits = np.ascontiguousarray(hits, dtype=np.int32)
    sens = np.ascontiguousarray(sens, dtype=np.float64)
    sample = np.ascontiguousarray(sample, dtype=np.int32)
    n, L, Hq = hits.shape
    Hkv = sens.shape[2]
    roles = np.empty((L, Hkv), dtype=np.uint8)
    vs, hs, imp = (np.empty((L, Hkv), dtype=np.float64) for _ in range(3))
    if lib().wnwo_triage(L, Hkv, Hq // Hkv, n, _ptr(sample), _ptr(hits), K, _ptr(sens), n_voice, n_anchor,
                         _ptr(roles), _ptr(vs), _ptr(hs), _ptr(imp)):
        raise ValueError("wnwo_triage failed")
    return roles, vs, hs, imp


def set_threads(n: int) -> int:
    """Threads of the oracle's parallel loops from now on (n <= 0: unchanged); returns the count."""
    return lib().wnwo_set_threads(n)


class Oracle:
    """Stateful oracle over one batch of sequences.  k, v: uint16 [B][L][H_kv][T][d];
    roles uint8 [L][H_kv]; prefill fp32 [B][L][H_kv][T_a].  The arrays are referenced, not
    copied, so they are kept alive here."""

    def __init__(self, cfg: _Cfg, k, v, roles, prefill, importance=None, lam=None):
        """importance [L][H_kv] fp32 and lam (fp32): per-head retention min(importance * lam, 1)
        of Eq. 1 instead of the uniform budget."""
        self.cfg = cfg
        self.n_chunks, self.k, self.keep_total = geometry(cfg)
        self.n_segments = segments(cfg)   # the unit of masses and residency (= chunks when disjoint)
        self._k = np.ascontiguousarray(k, dtype=np.uint16)
        self._v = np.ascontiguousarray(v, dtype=np.uint16)
        self._roles = np.ascontiguousarray(roles, dtype=np.uint8)
        self._pf = np.ascontiguousarray(prefill, dtype=np.float32)
        B, L, H, D = cfg.batch, cfg.layers, cfg.kv_heads, cfg.head_dim
        T = cfg.audio_len + cfg.text_len
        assert self._k.shape == (B, L, H, T, D) and self._v.shape == self._k.shape
        assert self._roles.shape == (L, H) and self._pf.shape == (B, L, H, cfg.audio_len)
        self.n_anchor_q = int((self._roles == 0).sum()) * (cfg.q_heads // cfg.kv_heads)
        self._imp = None if importance is None else np.ascontiguousarray(importance, dtype=np.float32)
        if self._imp is not None:
            assert self._imp.shape == (L, H) and lam is not None
        self._h = lib().wnwo_create_retention(C.byref(cfg), _ptr(self._k), _ptr(self._v), _ptr(self._roles),
                                              _ptr(self._pf), _ptr(self._imp),
                                              float(np.float32(lam)) if lam is not None else 0.0)
        if not self._h:
            raise ValueError("wnwo_create failed")

    def close(self):
        if getattr(self, "_h", None):
            lib().wnwo_destroy(self._h)
            self._h = None

    __del__ = close

    def keep_mask(self, b, l, kv) -> np.ndarray:
        m = np.empty(self.cfg.audio_len, dtype=np.uint8)
        if lib().wnwo_keep_mask(self._h, b, l, kv, _ptr(m)):
            raise ValueError("bad head index")
        return m

    def append(self, k_new, v_new):
        """K, V rows [B][L][H_kv][d] (uint16 bf16) of the token generated at this step."""
        c = self.cfg
        k = np.ascontiguousarray(k_new, dtype=np.uint16)
        v = np.ascontiguousarray(v_new, dtype=np.uint16)
        assert k.shape == (c.batch, c.layers, c.kv_heads, c.head_dim) and v.shape == k.shape
        if lib().wnwo_append(self._h, _ptr(k), _ptr(v)):
            raise ValueError("wnwo_append failed (more than max_new tokens?)")

    def step(self, q, forced=None, head_mask=None):
        c = self.cfg
        B, L, Hq, D = c.batch, c.layers, c.q_heads, c.head_dim
        q = np.ascontiguousarray(q, dtype=np.uint16)
        assert q.shape == (B, L, Hq, D)
        out = np.empty((B, L, Hq, D), dtype=np.float64)
        scores = np.empty((B, self.n_chunks), dtype=np.float64)
        sel = np.empty((B, max(self.k, 1)), dtype=np.int32)
        ns = self.n_segments
        mass = np.empty((B, max(self.n_anchor_q, 1), max(ns, 1)), dtype=np.float64)
        res = np.empty((B, max(ns, 1)), dtype=np.uint8)
        f = None if forced is None else np.ascontiguousarray(forced, dtype=np.int32).reshape(B, self.k)
        hm = None if head_mask is None else np.ascontiguousarray(head_mask, dtype=np.uint8).reshape(L, c.kv_heads)
        rc = lib().wnwo_step(self._h, _ptr(q), _ptr(f), _ptr(hm), _ptr(out), _ptr(scores), _ptr(sel),
                             _ptr(mass), _ptr(res))
        if rc:
            raise ValueError(f"wnwo_step failed ({rc})")
        return {"out": out, "scores": scores, "selected": sel[:, : self.k],
                "mass": mass[:, : self.n_anchor_q, : ns], "resident": res[:, : ns]}
