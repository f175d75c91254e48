"""The C-ABI library on the CPU: it builds, loads, exports every declared entry point, its
header compiles as C99 and C++17, and argument validation answers without a GPU."""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "wnw.h")


@pytest.fixture(scope="module")
def W():
    from paper_2608_22704_amd import build
    if not os.path.exists(build.LIB):
        build.build()
    from paper_2608_22704_amd import wnw
    return wnw


def declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"\b(wnw_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported(W):
    names = declared()
    assert len(names) >= 11
    assert set(names) == set(W.EXPORTS)
    out = subprocess.run(["nm", "-D", "--defined-only", W.LIB_PATH], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r" T (wnw_[a-z_]+)", out))
    assert set(names) <= exported


def test_flag_and_status_values_match_the_header(W):
    src = open(HEADER).read()
    values = {m.group(1): int(m.group(2), 0) for m in re.finditer(r"\b(WNW_(?:F|ERR)_[A-Z0-9_]+)\s*=\s*(-?(?:0x)?[0-9a-fA-F]+)u?", src)}
    assert {k for k in values if k.startswith("WNW_F_")} >= {"WNW_F_SELECT_NEXT_STEP", "WNW_F_OUT_BF16"}
    for name, v in values.items():
        assert getattr(W, name) == v, name


@pytest.mark.parametrize("cmd", [["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-x", "c"],
                                 ["g++", "-std=c++17", "-Wall", "-Wextra", "-pedantic", "-x", "c++"]])
def test_header_compiles(cmd, tmp_path):
    src = tmp_path / "use.c"
    src.write_text('#include "wnw.h"\nint main(void){ wnw_config c = {0}; (void)c; return (int)WNW_OK; }\n')
    subprocess.run(cmd + ["-I", os.path.join(ROOT, "include"), "-fsyntax-only", str(src)], check=True)


def test_validation_without_gpu(W):
    good = dict(batch=1, layers=1, q_heads=24, kv_heads=8, audio_len=1000, text_len=64, chunk_len=32, budget_bp=2000)
    cases = [
        (dict(head_dim=64), W.WNW_ERR_UNSUPPORTED),
        (dict(q_heads=20), W.WNW_ERR_INVALID),          # not a multiple of kv_heads
        (dict(q_heads=40), W.WNW_ERR_UNSUPPORTED),      # group 5
        (dict(budget_bp=10001), W.WNW_ERR_INVALID),
        (dict(chunk_len=0), W.WNW_ERR_INVALID),
        (dict(chunk_len=300), W.WNW_ERR_UNSUPPORTED),
        (dict(top_k=100), W.WNW_ERR_INVALID),           # more than the 32 chunks
        (dict(audio_len=0, text_len=0), W.WNW_ERR_INVALID),
        (dict(flags=1 << 10), W.WNW_ERR_INVALID),
    ]
    for over, want in cases:
        kw = dict(good)
        kw.update(over)
        cfg = W.make_config(**kw)
        with pytest.raises(W.WnwError) as e:
            W.wnw_init_cache(cfg, 1, 1, stream=0)
        assert e.value.status == want, (over, str(e.value))
        assert W.wnw_last_error(None)
    with pytest.raises(W.WnwError) as e:
        W.wnw_init_cache(W.make_config(**good), None, 1, stream=0)
    assert e.value.status == W.WNW_ERR_INVALID
    # NULL context everywhere
    assert W.lib.wnw_set_roles(None, None, None) == W.WNW_ERR_INVALID
    assert W.lib.wnw_decode_step(None, None, None, None, None, None) == W.WNW_ERR_INVALID
    assert W.lib.wnw_append_kv(None, None, None, None) == W.WNW_ERR_INVALID
    assert W.lib.wnw_set_selection_override(None, None) == W.WNW_ERR_INVALID
    assert W.lib.wnw_debug_set_slot_offset_limit(None, 0) == W.WNW_ERR_INVALID
    W.wnw_destroy(None)


def test_triage_host_ranking_matches_oracle():
    """wnw_triage (host code of the library, no GPU) on the hand-worked example and on random
    scores against the oracle's triage."""
    import json
    import os
    import numpy as np
    from oracle import oracle as O
    from paper_2608_22704_amd import wnw as W
    ex = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "triage_example.json")))
    roles, imp, vs, hs = W.wnw_triage(np.array(ex["hits"]), ex["K"], np.array(ex["sens"]), np.array(ex["sample"]),
                                      ex["n_voice"], ex["n_anchor"])
    assert roles.tolist() == ex["roles"]
    np.testing.assert_allclose(vs, ex["vs"], rtol=0, atol=1e-15)
    np.testing.assert_allclose(hs, ex["hs"], rtol=0, atol=1e-15)
    np.testing.assert_allclose(imp, ex["importance_norm"], rtol=0, atol=0)
    rng = np.random.default_rng(5)
    for trial in range(20):
        n, L, H, g = int(rng.integers(1, 9)), int(rng.integers(1, 5)), int(rng.integers(1, 9)), int(rng.choice([1, 2, 4]))
        hits = rng.integers(0, 5, size=(n, L, H * g)).astype(np.int32)
        sens = (rng.integers(0, 4, size=(n, L, H)) / 4).astype(np.float32)   # ties in the ranking
        sample = np.sort(rng.integers(0, 3, size=n)).astype(np.int32)
        nv = int(rng.integers(0, L * H + 1))
        na = int(rng.integers(0, nv + 1))
        r1, i1, v1, h1 = W.wnw_triage(hits, 4, sens, sample, nv, na)
        r2, v2, h2, i2 = O.triage(hits, 4, sens.astype(np.float64), sample, nv, na)
        assert np.array_equal(r1, r2), trial
        np.testing.assert_allclose(v1, v2, rtol=1e-15, atol=1e-15)
        np.testing.assert_allclose(h1, h2, rtol=1e-15, atol=1e-15)
        np.testing.assert_allclose(i1, i2.astype(np.float32), rtol=0, atol=0)


def test_binding_checks_buffers_before_passing_them():
    """The binding refuses buffers the library would misread: wrong element type, a
    non-contiguous view, too few elements; host inputs are converted to the library's types."""
    import numpy as np
    import torch
    from paper_2608_22704_amd import wnw as W
    x = torch.zeros(64, dtype=torch.int16)
    assert W._dev(x, W._BF16, 64) == x.data_ptr()
    assert W._dev(torch.zeros(8, dtype=torch.bfloat16), W._BF16, 8)
    with pytest.raises(TypeError):
        W._dev(torch.zeros(64, dtype=torch.float32), W._BF16, 64)
    with pytest.raises(TypeError):
        W._dev(torch.zeros(64, dtype=torch.int64), W._I32, 64)
    with pytest.raises(ValueError):
        W._dev(torch.zeros(8, 8, dtype=torch.float32).t(), W._F32, 64)
    with pytest.raises(ValueError):
        W._dev(torch.zeros(63, dtype=torch.float32), W._F32, 64)
    assert W._dev(None, W._F32, 64) is None
    r = W._host_in(np.array([[0, 1], [2, 1]], dtype=np.int64), np.uint8, 4, "roles")
    assert r.dtype == np.uint8 and r.flags.c_contiguous and r.tolist() == [[0, 1], [2, 1]]
    p = W._host_in(np.zeros((3, 4), dtype=np.float64)[:, ::2], np.float32, 6)
    assert p.dtype == np.float32 and p.flags.c_contiguous
    with pytest.raises(ValueError):
        W._host_in(np.zeros(5), np.uint8, 4)
    buf = np.empty(16, dtype=np.uint16)
    assert W._host_out(buf, 32) == buf.ctypes.data
    with pytest.raises(ValueError):
        W._host_out(buf, 30)
    with pytest.raises(TypeError):
        W._host_out(np.empty(32, dtype=np.uint8)[::2], 16)


def test_structs_match_the_header(W, tmp_path):
    """The binding's ctypes structures have the header's size and field offsets (a C program
    compiled against the header prints them)."""
    import ctypes
    lines = []
    for st in (W.wnw_config, W.wnw_stats):
        name = st.__name__
        lines.append(f'printf("{name} sizeof %zu\\n", sizeof({name}));')
        for f, _ in st._fields_:
            lines.append(f'printf("{name} {f} %zu\\n", offsetof({name}, {f}));')
    src = tmp_path / "layout.c"
    src.write_text('#include <stddef.h>\n#include <stdio.h>\n#include "wnw.h"\nint main(void){\n' + "\n".join(lines) +
                   "\nreturn 0; }\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-Wall", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l}
    for st in (W.wnw_config, W.wnw_stats):
        name = st.__name__
        assert got[(name, "sizeof")] == ctypes.sizeof(st), name
        for f, _ in st._fields_:
            assert got[(name, f)] == getattr(st, f).offset, (name, f)
    # every field of the header's structures is in the binding
    src_h = open(HEADER).read()
    for st in (W.wnw_config, W.wnw_stats):
        body = src_h[:src_h.index("} " + st.__name__ + ";")]
        body = body[body.rindex("typedef struct {"):]
        fields = re.findall(r"^\s+(?:int32_t|int64_t|uint32_t|double|float)\s+(\w+);", body, re.M)
        assert fields == [f for f, _ in st._fields_], st.__name__
