"""Lock-step comparison of the HIP decode step (through the C ABI) with the CPU oracle.

Both sides consume the same seeded inputs (synth.gen).  The GPU runs free: it selects its own
chunks.  Each step its selection is checked against the oracle's chunk scores (a valid top-k,
up to chunks whose oracle score lies within 1e-6 of the k-th score), and the oracle is then
stepped with that same selection so that the two keep one trajectory.

Tolerances (bf16 storage, fp32 accumulation on the GPU, double in the oracle):
  outputs       max |gpu - oracle| <= 2e-2 over every compared head
  chunk scores  |gpu - oracle| <= 1e-5 * |oracle| per chunk
  selection     equal sets, except chunks within 1e-6 (relative) of the k-th oracle score
  residency     equal sets of resident chunks after every step
"""
from __future__ import annotations

import sys
import time

import numpy as np

from oracle import oracle as O
from synth import gen

OUT_TOL = 2e-2
SCORE_RTOL = 1e-5
# Prefill scores on the device: bf16 products are exact in fp32 and 128 of them are summed in
# fp32, so a logit carries at most ~128 * 2^-24 * sum|q_i k_i| (<= 2e-4 after the 1/sqrt(d)
# scale for these inputs) absolute error, which is the relative error of every softmax weight
# and so of every sum of them; 1e-3 leaves a margin.
PREFILL_RTOL = 1e-3
SEL_EXCUSE = 1e-6


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(a: np.ndarray):
    import torch
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def check_selection(gpu_sel: np.ndarray, oracle_scores: np.ndarray, k: int) -> int:
    """Raise unless gpu_sel is the top-k of the oracle's fp32 scores up to excused near-ties.
    Returns the number of excused differences."""
    if k == 0:
        assert gpu_sel.size == 0
        return 0
    s32 = oracle_scores.astype(np.float32)
    ref = O.topk(s32, k)
    diff = set(int(c) for c in gpu_sel) ^ set(int(c) for c in ref)
    if not diff:
        return 0
    kth = float(np.sort(s32)[::-1][k - 1])
    tol = SEL_EXCUSE * abs(kth)
    bad = [c for c in diff if abs(float(s32[c]) - kth) > tol]
    assert not bad, f"selection differs beyond near-ties: chunks {sorted(bad)} (k-th score {kth:.9g})"
    assert len(set(int(c) for c in gpu_sel)) == k and all(0 <= c < len(s32) for c in gpu_sel)
    return len(diff) // 2


def check_prefill(w, seg, seqs, host, gpu_scores, roles, importance, lam, global_=False) -> float:
    """Device prefill scores against the oracle's (double), relative per entry; the keep sets
    that the fp32 scores give (per-segment ranking, the library's rule) must be those of the
    double scores except at positions whose score lies within PREFILL_RTOL of the segment's
    boundary.  Returns the largest relative error."""
    L, H, Ta, Tt, D = w.layers, w.kv_heads, w.audio_len, w.text_len, w.head_dim
    cfg1 = O.cfg_from_workload(w, batch=1)
    worst = 0.0
    for b in seqs:
        ref = O.prefill_scores(cfg1, host[b]["k"][None], host[b]["q_text"][None])[0]
        got = gpu_scores[b].astype(np.float64)
        rel = np.abs(got - ref) / np.maximum(np.abs(ref), 1e-300)
        worst = max(worst, float(rel.max(initial=0.0)))
        assert (rel <= PREFILL_RTOL).all(), f"seq {b}: prefill score rel err {rel.max():.3g}"
        for l in range(L):
            for kv in range(H):
                if roles[l, kv] == 0:
                    continue
                def count(n):
                    if importance is None:
                        return (w.budget_bp * n) // 10000
                    return int(np.floor(min(float(importance[l, kv]) * float(np.float32(lam)), 1.0) * n))
                segs = [(c0, min(c0 + seg, Ta)) for c0 in range(0, Ta, seg)]
                # the global variant ranks the per-segment total over the whole audio
                groups = [(0, Ta, sum(count(e - a) for a, e in segs))] if global_ else \
                    [(a, e, count(e - a)) for a, e in segs]
                for c0, e0, kc in groups:
                    n = e0 - c0
                    if kc in (0, n):
                        continue
                    r, gsc = ref[l, kv, c0:e0], gpu_scores[b, l, kv, c0:e0]
                    ko = set(sorted(range(n), key=lambda i: (-r[i], i))[:kc])
                    kg = set(sorted(range(n), key=lambda i: (-float(gsc[i]), i))[:kc])
                    bound = sorted(r, reverse=True)[kc - 1]
                    for i in ko ^ kg:
                        assert abs(r[i] - bound) <= PREFILL_RTOL * bound, \
                            f"seq {b} head ({l},{kv}) segment {c0}: keep sets differ beyond near-ties"
    return worst


class Lockstep:
    """One workload, a subset `seqs` of its sequences checked against the oracle (the GPU runs
    all w.batch sequences)."""

    def __init__(self, w, flags: int = 0, seqs=None, budget_bp=None, data=None, top_k=0, importance=None, lam=None,
                 prefill_device=False, append=False):
        """prefill_device: the prefill scores come from wnw_prefill_scores over the synthetic text
        queries, the keep sets from wnw_set_roles_device; the scores are checked against the
        oracle's (double) and then given to the oracle as its prefill input.
        append: before every step the K/V rows of a synthetic generated token (N(0,1), bf16, seeded
        by step) are appended on both sides (room for w.steps tokens)."""
        self.append = append
        import torch
        from paper_2608_22704_amd import wnw as W
        self.W, self.torch = W, torch
        if budget_bp is not None:
            w = w.with_(budget_bp=budget_bp)
        self.w = w
        self.seqs = list(range(w.batch)) if seqs is None else list(seqs)
        B, L, H, T, D = w.batch, w.layers, w.kv_heads, w.total_len, w.head_dim
        t0 = time.time()
        self.roles = gen.roles(w)
        kd = torch.empty((B, L, H, T, D), dtype=torch.int16, device="cuda")
        vd = torch.empty_like(kd)
        self.q = np.empty((w.steps, B, L, w.q_heads, D), dtype=np.uint16)
        self.prefill = np.empty((B, L, H, w.audio_len), dtype=np.float32)
        qt = torch.empty((B, L, w.q_heads, w.text_len, D), dtype=torch.int16, device="cuda") if prefill_device else None
        host = {}
        for b in range(B):
            if data is not None:
                seq = data[b]
            else:
                seq = gen.sequence(w, b)
            kd[b].copy_(to_dev(seq["k"]))
            vd[b].copy_(to_dev(seq["v"]))
            self.q[:, b] = seq["q"]
            self.prefill[b] = seq["prefill"]
            if prefill_device:
                seq["q_text"] = np.stack([gen.text_queries(w, b, l, kv, seq["k"][l, kv])
                                          for l in range(L) for kv in range(H)]).reshape(L, w.q_heads, w.text_len, D)
                qt[b].copy_(to_dev(seq["q_text"]))
            if b in self.seqs:
                host[b] = seq
        torch.cuda.synchronize()
        log(f"[harness] {w.name}: inputs ready in {time.time() - t0:.1f}s")
        self.cfg = W.make_config(B, L, w.q_heads, H, w.audio_len, w.text_len, w.chunk_len, w.budget_bp,
                                 top_k=top_k, flags=flags, max_new_tokens=w.steps if append else 0)
        self.ctx = W.wnw_init_cache(self.cfg, kd, vd)
        if importance is not None:
            W.wnw_set_retention(self.ctx, importance, lam)
        if prefill_device:
            sc = torch.empty((B, L, H, w.audio_len), dtype=torch.float32, device="cuda")
            W.wnw_prefill_scores(self.ctx, qt, sc)
            torch.cuda.synchronize()
            self.prefill = sc.cpu().numpy()
            seg = w.chunk_len // 2 if flags & W.WNW_F_OVERLAP_CHUNKS else w.chunk_len
            self.prefill_err = check_prefill(w, seg, self.seqs, host, self.prefill, self.roles, importance, lam,
                                             bool(flags & W.WNW_F_PREFILL_GLOBAL))
            W.wnw_set_roles_device(self.ctx, self.roles, sc)
            del qt, sc
        else:
            W.wnw_set_roles(self.ctx, self.roles, self.prefill)
        del kd, vd
        torch.cuda.empty_cache()
        self.geo = W.wnw_query_geometry(self.ctx)
        self.next_step = 1 if flags & W.WNW_F_SELECT_NEXT_STEP else 0
        span = 2 if flags & W.WNW_F_OVERLAP_CHUNKS else 1
        ocfg = O.cfg_from_workload(w, batch=len(self.seqs), top_k=top_k, next_step=self.next_step,
                                   chunk_span=span, prefill_global=1 if flags & W.WNW_F_PREFILL_GLOBAL else 0,
                                   max_new=w.steps if append else 0)
        self.ok_ = np.stack([host[b]["k"] for b in self.seqs])
        self.ov_ = np.stack([host[b]["v"] for b in self.seqs])
        self.oracle = O.Oracle(ocfg, self.ok_, self.ov_, self.roles, self.prefill[self.seqs], importance=importance,
                               lam=lam)
        assert (self.oracle.n_chunks, self.oracle.k) == (self.geo["n_chunks"], self.geo["k"])
        assert self.geo["keep_total"] == (self.oracle.keep_total if importance is None else -1)
        # kept audio rows of every head against the oracle's keep sets
        self.head_keep = W.wnw_query_head_keep(self.ctx, L, H)
        okeep = np.array([[self.oracle.keep_mask(0, l, h).sum() for h in range(H)] for l in range(L)])
        assert np.array_equal(self.head_keep, okeep), "per-head keep counts differ from the oracle"
        assert self.oracle.n_segments == self.geo["n_segments"]
        self.k, self.nc, self.nseg = self.geo["k"], self.geo["n_chunks"], self.geo["n_segments"]
        self.out = torch.empty((B, L, w.q_heads, D), dtype=torch.float32, device="cuda")
        self.scores = torch.empty((B, max(self.nc, 1)), dtype=torch.float32, device="cuda")
        self.sel = torch.empty((B, max(self.k, 1)), dtype=torch.int32, device="cuda")
        self.flips = 0
        self.max_err = 0.0
        self.max_score_rel = 0.0
        self.step_i = 0

    def close(self):
        if getattr(self, "ctx", None) is not None:
            try:
                # a step that ran out of recall slots fails the context: get_stats raises then
                st = self.W.wnw_get_stats(self.ctx)
                assert st["slot_exhausted"] == 0
                self.final_stats = st
                self.recalled_total = st["recalled_chunks"]
            finally:
                self.W.wnw_destroy(self.ctx)
                self.ctx = None
        if getattr(self, "oracle", None) is not None:
            self.oracle.close()

    def new_token(self, s: int):
        """K, V rows [B][L][H_kv][d] (bf16 bit patterns) of the token generated before step s."""
        w = self.w
        rng = np.random.default_rng(7000 + s)
        shape = (w.batch, w.layers, w.kv_heads, w.head_dim)
        return (gen.f32_to_bf16(rng.standard_normal(shape, dtype=np.float32)),
                gen.f32_to_bf16(rng.standard_normal(shape, dtype=np.float32)))

    def gpu_step(self, s: int):
        if self.append:
            kn, vn = self.new_token(s)
            self.W.wnw_append_kv(self.ctx, to_dev(kn), to_dev(vn))
        qd = to_dev(self.q[s])
        self.W.wnw_decode_step(self.ctx, qd, self.out, self.scores, self.sel)
        self.torch.cuda.synchronize()
        res = np.empty((self.w.batch, max(self.nseg, 1)), dtype=np.uint8)
        self.W.wnw_debug_read_resident(self.ctx, res)
        return (self.out.cpu().numpy(), self.scores.cpu().numpy()[:, : self.nc],
                self.sel.cpu().numpy()[:, : self.k], res[:, : self.nseg])

    def step(self, s: int, head_mask=None):
        out, sc, sel, res = self.gpu_step(s)
        idx = self.seqs
        if self.append:
            kn, vn = self.new_token(s)
            self.oracle.append(kn[idx], vn[idx])
        r = self.oracle.step(self.q[s][idx], forced=sel[idx] if self.k else None, head_mask=head_mask)
        for j, b in enumerate(idx):
            so = r["scores"][j]
            rel = np.abs(sc[b].astype(np.float64) - so) / np.maximum(np.abs(so), 1e-300)
            self.max_score_rel = max(self.max_score_rel, float(rel.max(initial=0.0)))
            assert (np.abs(sc[b].astype(np.float64) - so) <= SCORE_RTOL * np.abs(so)).all(), \
                f"step {s} seq {b}: chunk score rel err {rel.max():.3g}"
            self.flips += check_selection(sel[b], so, self.k)
            assert (res[b] == r["resident"][j]).all(), f"step {s} seq {b}: resident sets differ"
        # outputs: anchors always, non-anchor heads where the mask asks for them
        L, H, g = self.w.layers, self.w.kv_heads, self.w.group
        m = np.ones((L, H), dtype=bool) if head_mask is None else np.asarray(head_mask, dtype=bool).reshape(L, H)
        m = m | (self.roles == 0)
        mq = np.repeat(m, g, axis=1)                          # [L][Hq]
        for j, b in enumerate(idx):
            err = np.abs(out[b][mq].astype(np.float64) - r["out"][j][mq]).max(initial=0.0)
            self.max_err = max(self.max_err, float(err))
            assert err <= OUT_TOL, f"step {s} seq {b}: output max abs err {err:.4g}"
        self.step_i += 1
        return out, sc, sel, res
