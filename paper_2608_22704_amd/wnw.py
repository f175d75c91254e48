"""Python binding of the WnW decode-step library (libwnw.so), argument marshalling only.

Function names match the C ABI of include/wnw.h.  Every computation runs in the HIP library;
this module only converts arguments (torch tensors -> device pointers, torch streams -> HIP
streams) and turns error codes into exceptions.  It raises at import time when the library has
not been built: there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libwnw.so")

WNW_OK, WNW_ERR_INVALID, WNW_ERR_OOM, WNW_ERR_HIP, WNW_ERR_STATE, WNW_ERR_UNSUPPORTED = 0, -1, -2, -3, -4, -5
WNW_ANCHOR, WNW_TIDAL, WNW_FIXED = 0, 1, 2
WNW_F_SELECT_NEXT_STEP, WNW_F_RECALL_MEMCPY, WNW_F_TIMING, WNW_F_OVERLAP_CHUNKS, WNW_F_PREFILL_GLOBAL = 1, 2, 4, 8, 16
WNW_F_OUT_BF16 = 32

EXPORTS = ("wnw_init_cache", "wnw_set_retention", "wnw_set_roles", "wnw_prefill_scores", "wnw_prefill_scores_static",
           "wnw_set_roles_device",
           "wnw_append_kv", "wnw_decode_step", "wnw_query_geometry",
           "wnw_query_segments", "wnw_query_head_keep", "wnw_get_stats",
           "wnw_set_selection_override", "wnw_debug_read_slot", "wnw_debug_read_host_chunk",
           "wnw_debug_set_slot_offset_limit", "wnw_debug_set_recall_delay",
           "wnw_debug_read_resident", "wnw_last_error", "wnw_destroy", "wnw_voice_hits", "wnw_key_sensitivity",
           "wnw_triage", "wnw_triage_last_error")


class wnw_config(C.Structure):
    _fields_ = [("batch", C.c_int32), ("layers", C.c_int32), ("q_heads", C.c_int32), ("kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("audio_len", C.c_int32), ("text_len", C.c_int32),
                ("chunk_len", C.c_int32), ("budget_bp", C.c_int32), ("top_k", C.c_int32),
                ("evict_lag", C.c_int32), ("flags", C.c_uint32), ("max_new_tokens", C.c_int32)]


class wnw_stats(C.Structure):
    _fields_ = [("steps", C.c_int64), ("recalled_chunks", C.c_int64), ("revived_chunks", C.c_int64),
                ("recalled_bytes", C.c_int64),
                ("dropped_chunks", C.c_int64), ("resident_chunks", C.c_int64), ("peak_resident", C.c_int32),
                ("n_slots", C.c_int32), ("r_gpu", C.c_double), ("r_gpu_cpu", C.c_double),
                ("anchor_bytes", C.c_int64), ("static_bytes", C.c_int64), ("slot_rows", C.c_int64),
                ("timed_steps", C.c_int64), ("t_anchor_ms", C.c_double), ("t_select_ms", C.c_double),
                ("t_tidal_fixed_ms", C.c_double), ("t_new_ms", C.c_double), ("t_combine_ms", C.c_double),
                ("t_step_ms", C.c_double), ("t_recall_ms", C.c_double), ("slot_exhausted", C.c_int64),
                ("t_host_wait_ms", C.c_double), ("t_recall_wait_ms", C.c_double), ("kept_rows", C.c_int64),
                ("selections_in_tidal", C.c_int64)]

    def as_dict(self) -> dict:
        return {name: getattr(self, name) for name, _ in self._fields_}


class WnwError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"wnw status {status}: {msg}")
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build the HIP library first (__graft_entry__.build())")
    lib = C.CDLL(LIB_PATH)
    P, I32, I64, SZ = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
    sig = {
        "wnw_init_cache": ([C.POINTER(wnw_config), P, P, P, C.POINTER(P)], C.c_int),
        "wnw_set_roles": ([P, P, P], C.c_int),
        "wnw_set_retention": ([P, P, C.c_float], C.c_int),
        "wnw_prefill_scores": ([P, P, P], C.c_int),
        "wnw_prefill_scores_static": ([P, P, P, P], C.c_int),
        "wnw_append_kv": ([P, P, P, P], C.c_int),
        "wnw_voice_hits": ([I32, I32, I32, I32, I32, I32, P, P, P, I32, P, P], C.c_int),
        "wnw_key_sensitivity": ([I32, I32, I32, I32, P, P, P], C.c_int),
        "wnw_triage": ([I32, I32, I32, I32, P, P, I32, P, I32, I32, P, P, P, P], C.c_int),
        "wnw_triage_last_error": ([], C.c_char_p),
        "wnw_set_roles_device": ([P, P, P], C.c_int),
        "wnw_query_head_keep": ([P, P], C.c_int),
        "wnw_decode_step": ([P, P, P, P, P, P], C.c_int),
        "wnw_query_geometry": ([P, C.POINTER(I32), C.POINTER(I32), C.POINTER(I32), C.POINTER(I32), C.POINTER(I64)], C.c_int),
        "wnw_query_segments": ([P, C.POINTER(I32)], C.c_int),
        "wnw_get_stats": ([P, C.POINTER(wnw_stats)], C.c_int),
        "wnw_set_selection_override": ([P, P], C.c_int),
        "wnw_debug_read_slot": ([P, I32, I32, P, SZ], C.c_int),
        "wnw_debug_read_host_chunk": ([P, I32, I32, P, SZ], C.c_int),
        "wnw_debug_read_resident": ([P, P], C.c_int),
        "wnw_debug_set_slot_offset_limit": ([P, I64], C.c_int),
        "wnw_debug_set_recall_delay": ([P, I32], C.c_int),
        "wnw_last_error": ([P], C.c_char_p),
        "wnw_destroy": ([P], None),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes, fn.restype = args, res
    return lib


lib = _load()


def _check(status: int, ctx=None):
    if status != WNW_OK:
        raise WnwError(status, lib.wnw_last_error(ctx).decode())


def _ptr(t):
    """Device (or host) address of a tensor / numpy array / int, or None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if hasattr(t, "data_ptr"):
        return t.data_ptr()
    return t.ctypes.data


# element sizes the library reads or writes: bf16 bit patterns (any 2-byte dtype), fp32, int32
_BF16, _F32, _I32 = "bf16", "f32", "i32"


def _dev(t, kind, numel=None, what="tensor"):
    """Address of a device tensor after checking it holds at least `numel` contiguous elements
    of the kind the library expects (no conversion: the library reads the raw buffer)."""
    if t is None or isinstance(t, int):
        return t
    if not hasattr(t, "data_ptr"):
        raise TypeError(f"{what} must be a device tensor")
    import torch
    ok = {_BF16: t.element_size() == 2 and not t.dtype.is_complex,
          _F32: t.dtype == torch.float32, _I32: t.dtype == torch.int32}[kind]
    if not ok:
        raise TypeError(f"{what}: expected {kind} elements, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{what}: needs {numel} elements, got {t.numel()}")
    return t.data_ptr()


def _host_in(a, dtype, numel=None, what="array"):
    """A contiguous host copy (or view) of `a` with the given numpy dtype, size checked."""
    a = np.ascontiguousarray(a, dtype=dtype)
    if numel is not None and a.size != numel:
        raise ValueError(f"{what}: expected {numel} elements, got {a.size}")
    return a


def _host_out(a, nbytes, what="host_dst"):
    """Address of a writable, contiguous host array of exactly nbytes."""
    if not isinstance(a, np.ndarray) or not a.flags.c_contiguous or not a.flags.writeable:
        raise TypeError(f"{what} must be a writable C-contiguous numpy array")
    if a.nbytes != nbytes:
        raise ValueError(f"{what}: expected {nbytes} bytes, got {a.nbytes}")
    return a.ctypes.data


_CFG = {}   # handle value -> wnw_config, for the size checks of later calls


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


# ---- the C ABI, one wrapper per entry point -------------------------------------------------

def _cache_numel(cfg):
    return cfg.batch * cfg.layers * cfg.kv_heads * (cfg.audio_len + cfg.text_len) * cfg.head_dim


def wnw_init_cache(cfg: wnw_config, k_dev, v_dev, stream=None):
    n = _cache_numel(cfg)
    h = C.c_void_p()
    _check(lib.wnw_init_cache(C.byref(cfg), _dev(k_dev, _BF16, n, "k_dev"), _dev(v_dev, _BF16, n, "v_dev"),
                              _stream(stream), C.byref(h)))
    _CFG[h.value] = wnw_config.from_buffer_copy(cfg)
    return h


def _cfg(ctx):
    return _CFG.get(getattr(ctx, "value", ctx))


def wnw_set_retention(ctx, importance, lam):
    """importance: host fp32 [L][H_kv] (or None for the uniform budget); lam: the scale."""
    c = _cfg(ctx)
    imp = None if importance is None else _host_in(importance, np.float32, c and c.layers * c.kv_heads, "importance")
    _check(lib.wnw_set_retention(ctx, _ptr(imp), float(lam)), ctx)


def wnw_set_roles(ctx, roles, prefill_scores):
    """roles: host uint8 [L][H_kv]; prefill_scores: host fp32 [B][L][H_kv][T_a]."""
    c = _cfg(ctx)
    r = _host_in(roles, np.uint8, c and c.layers * c.kv_heads, "roles")
    p = _host_in(prefill_scores, np.float32, c and c.batch * c.layers * c.kv_heads * c.audio_len, "prefill_scores")
    _check(lib.wnw_set_roles(ctx, _ptr(r), _ptr(p)), ctx)


def _tcheck(status):
    if status != WNW_OK:
        raise WnwError(status, lib.wnw_triage_last_error().decode())


def wnw_voice_hits(k_dev, q_dev, span_dev, top_k, audio_len, hits_dev, stream=None):
    """k_dev [L][H_kv][rows][d] bf16, q_dev [n_tok][L][H_q][d] bf16, span_dev int32 [n_tok][2] ->
    hits_dev int32 [n_tok][L][H_q] (tensors on the device)."""
    L, Hkv, rows, D = k_dev.shape
    n_tok, _, Hq, _ = q_dev.shape
    _tcheck(lib.wnw_voice_hits(L, Hq, Hkv, rows, audio_len, n_tok, _dev(k_dev, _BF16, None, "k_dev"),
                               _dev(q_dev, _BF16, n_tok * L * Hq * D, "q_dev"), _dev(span_dev, _I32, n_tok * 2, "span_dev"),
                               top_k, _dev(hits_dev, _I32, n_tok * L * Hq, "hits_dev"), _stream(stream)))


def wnw_key_sensitivity(grad_dev, sens_dev, stream=None):
    """grad_dev fp32 [n_tok][L][H_kv][T_a][d] -> sens_dev fp32 [n_tok][L][H_kv]."""
    n_tok, L, Hkv, Ta, _ = grad_dev.shape
    _tcheck(lib.wnw_key_sensitivity(L, Hkv, Ta, n_tok, _dev(grad_dev, _F32, None, "grad_dev"),
                                    _dev(sens_dev, _F32, n_tok * L * Hkv, "sens_dev"), _stream(stream)))


def wnw_triage(hits, top_k, sens, sample, n_voice, n_anchor):
    """Host arrays hits int32 [n][L][H_q], sens fp32 [n][L][H_kv], sample int32 [n] ->
    (roles uint8, importance fp32, vs, hs) each [L][H_kv]."""
    hits = np.ascontiguousarray(hits, dtype=np.int32)
    sens = np.ascontiguousarray(sens, dtype=np.float32)
    sample = np.ascontiguousarray(sample, dtype=np.int32)
    n, L, Hq = hits.shape
    Hkv = sens.shape[2]
    roles = np.empty((L, Hkv), dtype=np.uint8)
    imp = np.empty((L, Hkv), dtype=np.float32)
    vs, hs = np.empty((L, Hkv)), np.empty((L, Hkv))
    _tcheck(lib.wnw_triage(L, Hkv, Hq // Hkv, n, _ptr(sample), _ptr(hits), top_k, _ptr(sens), n_voice, n_anchor,
                           _ptr(roles), _ptr(imp), _ptr(vs), _ptr(hs)))
    return roles, imp, vs, hs


def wnw_append_kv(ctx, k_new_dev, v_new_dev, stream=None):
    c = _cfg(ctx)
    n = c and c.batch * c.layers * c.kv_heads * c.head_dim
    _check(lib.wnw_append_kv(ctx, _dev(k_new_dev, _BF16, n, "k_new_dev"), _dev(v_new_dev, _BF16, n, "v_new_dev"),
                             _stream(stream)), ctx)


def wnw_prefill_scores(ctx, q_text_dev, scores_dev):
    c = _cfg(ctx)
    nq = c and c.batch * c.layers * c.q_heads * c.text_len * c.head_dim
    ns = c and c.batch * c.layers * c.kv_heads * c.audio_len
    _check(lib.wnw_prefill_scores(ctx, _dev(q_text_dev, _BF16, nq, "q_text_dev"), _dev(scores_dev, _F32, ns, "scores_dev")),
           ctx)


def wnw_prefill_scores_static(ctx, q_text_dev, scores_dev, stream=None):
    c = _cfg(ctx)
    nq = c and c.batch * c.layers * c.q_heads * c.text_len * c.head_dim
    ns = c and c.batch * c.layers * c.kv_heads * c.audio_len
    _check(lib.wnw_prefill_scores_static(ctx, _dev(q_text_dev, _BF16, nq, "q_text_dev"),
                                         _dev(scores_dev, _F32, ns, "scores_dev"), _stream(stream)), ctx)


def wnw_set_roles_device(ctx, roles, prefill_scores_dev):
    c = _cfg(ctx)
    r = _host_in(roles, np.uint8, c and c.layers * c.kv_heads, "roles")
    ns = c and c.batch * c.layers * c.kv_heads * c.audio_len
    _check(lib.wnw_set_roles_device(ctx, _ptr(r), _dev(prefill_scores_dev, _F32, ns, "prefill_scores_dev")), ctx)


def wnw_query_head_keep(ctx, layers, kv_heads) -> np.ndarray:
    keep = np.empty((layers, kv_heads), dtype=np.int32)
    _check(lib.wnw_query_head_keep(ctx, _ptr(keep)), ctx)
    return keep


def wnw_decode_step(ctx, q_dev, out_dev, chunk_scores_dev=None, selected_dev=None, stream=None):
    c = _cfg(ctx)
    nq = c and c.batch * c.layers * c.q_heads * c.head_dim
    okind = _BF16 if c and c.flags & WNW_F_OUT_BF16 else _F32
    _check(lib.wnw_decode_step(ctx, _dev(q_dev, _BF16, nq, "q_dev"), _dev(out_dev, okind, nq, "out_dev"),
                               _dev(chunk_scores_dev, _F32, None, "chunk_scores_dev"),
                               _dev(selected_dev, _I32, None, "selected_dev"), _stream(stream)), ctx)


def wnw_query_geometry(ctx) -> dict:
    n, k, kt, ns, cb = C.c_int32(), C.c_int32(), C.c_int32(), C.c_int32(), C.c_int64(-1)
    _check(lib.wnw_query_geometry(ctx, C.byref(n), C.byref(k), C.byref(kt), C.byref(ns), None), ctx)
    out = {"n_chunks": n.value, "k": k.value, "keep_total": kt.value, "n_slots": ns.value}
    seg = C.c_int32()
    _check(lib.wnw_query_segments(ctx, C.byref(seg)), ctx)
    out["n_segments"] = seg.value
    if lib.wnw_query_geometry(ctx, None, None, None, None, C.byref(cb)) == WNW_OK:
        out["chunk_bytes"] = cb.value
    return out


def wnw_get_stats(ctx) -> dict:
    st = wnw_stats()
    _check(lib.wnw_get_stats(ctx, C.byref(st)), ctx)
    return st.as_dict()


def wnw_set_selection_override(ctx, sel_dev):
    _check(lib.wnw_set_selection_override(ctx, _dev(sel_dev, _I32, None, "sel_dev")), ctx)


def wnw_debug_set_slot_offset_limit(ctx, nbytes: int):
    _check(lib.wnw_debug_set_slot_offset_limit(ctx, nbytes), ctx)


def wnw_debug_set_recall_delay(ctx, us: int):
    _check(lib.wnw_debug_set_recall_delay(ctx, us), ctx)


def wnw_debug_read_slot(ctx, b: int, chunk: int, host_dst, nbytes: int):
    _check(lib.wnw_debug_read_slot(ctx, b, chunk, _host_out(host_dst, nbytes), nbytes), ctx)


def wnw_debug_read_host_chunk(ctx, b: int, chunk: int, host_dst, nbytes: int):
    _check(lib.wnw_debug_read_host_chunk(ctx, b, chunk, _host_out(host_dst, nbytes), nbytes), ctx)


def wnw_debug_read_resident(ctx, host_dst):
    """host_dst: writable uint8 [B][n_segments]."""
    seg = C.c_int32()
    _check(lib.wnw_query_segments(ctx, C.byref(seg)), ctx)
    c = _cfg(ctx)
    need = c.batch * seg.value if c is not None else 0
    if not isinstance(host_dst, np.ndarray) or not host_dst.flags.c_contiguous or not host_dst.flags.writeable \
            or host_dst.dtype != np.uint8 or host_dst.nbytes < need:
        raise ValueError(f"host_dst must be a writable contiguous uint8 array of at least {need} elements")
    _check(lib.wnw_debug_read_resident(ctx, _ptr(host_dst)), ctx)


def wnw_last_error(ctx=None) -> str:
    return lib.wnw_last_error(ctx).decode()


def wnw_destroy(ctx):
    _CFG.pop(getattr(ctx, "value", ctx), None)
    lib.wnw_destroy(ctx)


def make_config(batch, layers, q_heads, kv_heads, audio_len, text_len, chunk_len, budget_bp,
                head_dim=128, top_k=0, evict_lag=0, flags=0, max_new_tokens=0) -> wnw_config:
    return wnw_config(batch, layers, q_heads, kv_heads, head_dim, audio_len, text_len, chunk_len, budget_bp,
                      top_k, evict_lag, flags, max_new_tokens)
