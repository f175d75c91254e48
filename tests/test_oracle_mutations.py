"""Plant plausible mistakes in copies of the oracle (on the CPU) and require the pins to fail.

Each mutant is compiled from the oracle's source with one textual change and the pin suite
is run against it in a subprocess; a mutant that passes every pin would mean the pins leave
that part of the oracle unchecked.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "wnw_oracle.c")

MUTANTS = {
    "score is a sum, not a mean": (
        "double sc = a / (double)(seg_end(c, s1) - seg_begin(c, ch));", "double sc = a;"),
    "text rows left out of the anchor softmax": (
        "attend(qh, o->kc + hoff, o->vc + hoff, rows, T, D, x, oh, p);",
        "attend(qh, o->kc + hoff, o->vc + hoff, rows, Ta, D, x, oh, p);"),
    "chunk ties prefer the higher id": (
        "return (x->id > y->id) - (x->id < y->id);\n}\n\nstatic int by_int",
        "return (x->id < y->id) - (x->id > y->id);\n}\n\nstatic int by_int"),
    "eviction lag one step too long": (
        "            if (st[ch] < o->delta)\n", "            if (st[ch] <= o->delta)\n"),
    "keep count rounds up": (
        "return (int32_t)(((int64_t)c->budget_bp * len) / 10000);",
        "return (int32_t)(((int64_t)c->budget_bp * len + 9999) / 10000);"),
    "tidal heads ignore recalled chunks": (
        "(o->roles[hh] == 1 && ru[sg])", "(o->roles[hh] == 1 && 0 && ru[sg])"),
    "logit scale 1/d": ("1.0 / sqrt((double)d)", "1.0 / (double)d"),
    "prefill ranking keeps the lowest scores": (
        "    const ranked *x = a, *y = b;\n    if (x->s > y->s) return -1;",
        "    const ranked *x = a, *y = b;\n    if (x->s < y->s) return -1;"),
    "selection state not reset on selection": ("if (sel[i] >= 0) st[sel[i]] = 0;", "if (sel[i] >= 0) st[sel[i]] += 0;"),
    "fixed heads see recalled chunks": ("(o->roles[hh] == 1 && ru[sg])", "(o->roles[hh] >= 1 && ru[sg])"),
    "an overlapping chunk covers one segment": (
        "int32_t last = ch + span_of(c) - 1, ns = seg_count(c);", "int32_t last = ch, ns = seg_count(c);"),
    "overlapping chunk scored on its first segment": (
        "for (int32_t sg = ch; sg <= s1; ++sg) a +=", "for (int32_t sg = ch; sg <= ch; ++sg) a +="),
    "overlapping chunks start every other segment": (
        "return (span_of(c) == 2 && ns >= 2) ? ns - 1 : ns;", "return (span_of(c) == 2 && ns >= 2) ? ns / 2 : ns;"),
    "per-head retention ignores lambda": (
        "double r = (double)importance[h] * (double)lambda;", "double r = (double)importance[h];"),
    "per-head keep count rounds to nearest": (
        "return (int32_t)floor(r * (double)len);", "return (int32_t)floor(r * (double)len + 0.5);"),
    "per-head retention ignored": ("if (!importance) return keep_count(c, len);", "return keep_count(c, len);"),
    "prefill text tokens see every text row": (
        "attend(qv, K, K, rows, Ta + t + 1, D, x, o, w);", "attend(qv, K, K, rows, T, D, x, o, w);"),
    "prefill scores from the first q-head only": (
        "        for (int32_t j = 0; j < g; ++j)\n            for (int32_t t = 0; t < Tt; ++t) {",
        "        for (int32_t j = 0; j < 1; ++j)\n            for (int32_t t = 0; t < Tt; ++t) {"),
    "tidal and fixed heads miss the appended rows": (
        "for (int32_t t = Ta; t < T; ++t) rows[n++] = t;", "for (int32_t t = Ta; t < Ta + c->text_len; ++t) rows[n++] = t;"),
    "append overwrites the last prompt row": (
        "const size_t row = (size_t)c->audio_len + c->text_len + o->n_gen;",
        "const size_t row = (size_t)c->audio_len + c->text_len + o->n_gen - 1;"),
    "voice hits count the span's end": (
        "c += x[r].pos >= span[2 * t] && x[r].pos < span[2 * t + 1];",
        "c += x[r].pos >= span[2 * t] && x[r].pos <= span[2 * t + 1];"),
    "voice scores pooled over tokens instead of per sample": (
        "out[m] += sum[(size_t)s * M + m] / cnt[s];", "out[m] += sum[(size_t)s * M + m] * used / n;"),
    "head ranking ties to the higher head": (
        "    return (x->id > y->id) - (x->id < y->id);\n}\n\n/* Three-way",
        "    return (x->id < y->id) - (x->id > y->id);\n}\n\n/* Three-way"),
    "importance normalised by its sum": (
        "if (rk[h].s > mx) mx = rk[h].s;", "mx += rk[h].s;"),
    "global prefill keeps the last segment's count": (
        "for (int32_t j = 0; j < ns; ++j) total += keep_count_head(",
        "for (int32_t j = 0; j < ns; ++j) total = keep_count_head("),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor not unique/found: {old!r}"
    mpath = tmp_path / "mutant.c"
    mpath.write_text(src.replace(old, new))
    so = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O1", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-I", os.path.join(ROOT, "oracle"),
                    "-o", str(so), str(mpath), "-lm"], check=True)
    env = dict(os.environ, WNW_ORACLE_LIB=str(so))
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant '{name}' passed every pin:\n{r.stdout[-2000:]}"
