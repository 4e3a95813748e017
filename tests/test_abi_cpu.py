"""Host-side checks of the C ABI (no GPU needed): exported symbols, the exact
Eq. 3 table against the oracle, and argument validation."""
import math
import re
import os

import numpy as np
import pytest

import oracle
import paper_2512_11221_amd as A

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    with open(os.path.join(ROOT, "include", "asrkf.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(asrkf_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    lib = A.load()
    names = _declared()
    assert {"asrkf_init", "asrkf_decode_step", "asrkf_restore", "asrkf_stats"} <= set(names)
    for name in names:
        assert hasattr(lib, name), name


@pytest.mark.parametrize("k", [2.0, 1.5, 0.75, 3.0, 1.0, 2.5, 0.3, 7.25])
def test_schedule_table_matches_oracle(k):
    tab = A.asrkf_schedule_table(k, 3000)
    ref = oracle.duration_table(2999, k)
    np.testing.assert_array_equal(tab, ref)


def test_schedule_table_extremes_and_random_k():
    """The ends of the accepted k range and 24 seeded log-uniform k values,
    each rounded to float32 (the value the library sees): the table is the
    exact floor of sqrt(c) / k for every count."""
    rng = np.random.default_rng(0x5CED)
    ks = [2.0 ** -8, 2.0 ** 16, 1.7, 0.1, 1.0 / 3.0]
    ks += list(2.0 ** rng.uniform(-8, 16, size=24))
    for k in ks:
        k32 = float(np.float32(k))
        # the oracle searches d one step at a time: keep its work near 3e5 steps per k
        n = int(min(5000, max(100, (4.5e5 * k32) ** (2.0 / 3.0))))
        np.testing.assert_array_equal(A.asrkf_schedule_table(k32, n), oracle.duration_table(n - 1, k32),
                                      err_msg=f"k = {k32!r}")


def test_schedule_table_rejects_bad_k():
    for k in (0.0, -1.0, math.inf, math.nan, 1e-5, 1e6):
        with pytest.raises(A.AsrkfError):
            A.asrkf_schedule_table(k, 10)


BASE = dict(n_layers=1, batch=1, n_q_heads=8, n_kv_heads=2, head_dim=64, max_ctx=600,
            window_K=32, tau=0.5, k_soft=2.0, vocab=1024)


@pytest.mark.parametrize("bad", [
    dict(head_dim=96), dict(head_dim=256, dtype="f32"), dict(n_kv_heads=3), dict(n_q_heads=24, n_kv_heads=2),
    dict(n_kv_heads=64, n_q_heads=64), dict(n_kv_heads=16, n_q_heads=128),
    dict(n_kv_heads=32, n_q_heads=128), dict(n_kv_heads=32, n_q_heads=32, head_dim=128, dtype="f32"),
    dict(batch=0), dict(batch=5000), dict(n_layers=0),
    dict(max_ctx=1), dict(window_K=-1), dict(k_soft=0.0), dict(tau=math.nan), dict(vocab=0),
    dict(spill_min_D=-1), dict(device_rows=64), dict(spill_min_D=2, device_rows=1),
    dict(spill_min_D=2, device_rows=602), dict(candidates=2), dict(candidates=-1),
    dict(relevance=2), dict(scope=2), dict(dtype=7),
])
def test_init_rejects_invalid_config(bad):
    cfg = A.make_config(**{**BASE, **bad})
    with pytest.raises(A.AsrkfError) as e:
        A.asrkf_init(cfg)
    assert e.value.code == A._lib.EINVAL


def test_unknown_option_names_are_refused_by_the_binding():
    for kw in (dict(candidates="all"), dict(relevance="cosine"), dict(scope="head"),
               dict(dtype="f16")):
        with pytest.raises(ValueError):
            A.make_config(**{**BASE, **kw})


def test_null_context_is_einval():
    lib = A.load()
    assert lib.asrkf_set_timing(None, 1) == A._lib.EINVAL
    assert lib.asrkf_timing_series(None, None, 0, None) == A._lib.EINVAL
    assert lib.asrkf_reset(None) == A._lib.EINVAL
    assert lib.asrkf_debug_delay_side(None, 5) == A._lib.EINVAL
    assert lib.asrkf_restore(None, None, 0, None) == A._lib.EINVAL
    assert "null context" in A.asrkf_last_error()
    lib.asrkf_destroy(None)


def test_c_program_uses_the_abi(tmp_path):
    """The header is plain C: a C99 program includes it, links libasrkf.so and
    runs the host-only calls (tests/c_abi/abi_check.c)."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    lib = A.load()._name                       # the build the binding loads
    exe = str(tmp_path / "abi_check")
    subprocess.run([gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
                    os.path.join(ROOT, "tests", "c_abi", "abi_check.c"),
                    "-I", os.path.join(ROOT, "include"), lib,
                    "-Wl,-rpath-link,/opt/rocm/lib", "-o", exe],
                   check=True, capture_output=True, text=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    assert "C ABI checks passed" in r.stdout


def test_binding_structs_match_the_header(tmp_path):
    """The ctypes mirrors of asrkf_config and asrkf_stats_t have the size and
    field offsets the C compiler gives the header's structs (a field added to
    the header and not to the binding, or the reverse, fails here)."""
    import ctypes
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    from paper_2512_11221_amd import _lib as L
    lines = ["#include <stddef.h>", "#include <stdio.h>", '#include "asrkf.h"', "int main(void) {"]
    for cname, py in (("asrkf_config", L.asrkf_config), ("asrkf_stats_t", L.asrkf_stats_t)):
        lines.append(f'    printf("{cname} size %zu\\n", sizeof({cname}));')
        for field, _ in py._fields_:
            lines.append(f'    printf("{cname} {field} %zu\\n", offsetof({cname}, {field}));')
    lines += ["    return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = str(tmp_path / "layout")
    subprocess.run([gcc, "-std=c99", "-Wall", "-Werror", str(src), "-I", os.path.join(ROOT, "include"),
                    "-o", exe], check=True, capture_output=True, text=True)
    out = subprocess.run([exe], capture_output=True, text=True, timeout=60).stdout.split("\n")
    got = {(a, b): int(c) for a, b, c in (x.split() for x in out if x)}
    for cname, py in (("asrkf_config", L.asrkf_config), ("asrkf_stats_t", L.asrkf_stats_t)):
        assert got[(cname, "size")] == ctypes.sizeof(py), cname
        for field, _ in py._fields_:
            assert got[(cname, field)] == getattr(py, field).offset, (cname, field)
