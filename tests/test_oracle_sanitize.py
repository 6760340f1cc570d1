"""The CPU oracle under AddressSanitizer and UndefinedBehaviorSanitizer (host only).

A small C driver (tests/native/oracle_sanitize_main.c) calls every oracle entry
-- model creation and its error paths, the forward passes, heads, decision
primitives, AR and speculative frames in all three draft modes, traced and
untraced -- on a small fp32 and a small bf16 model; any out-of-bounds access,
use after free, leak or undefined operation aborts the run.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

from paper_2609_37007_amd import synth as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("dtype", [S.DTYPE_F32, S.DTYPE_BF16])
def test_oracle_is_clean_under_asan_and_ubsan(tmp_path, dtype):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path / "orc_san")
    cmd = ["gcc", "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-ffp-contract=off",
           os.path.join(ROOT, "oracle", "rvqsd_oracle.c"), os.path.join(ROOT, "tests", "native", "oracle_sanitize_main.c"),
           "-o", exe, "-lm"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0 and "asan" in (r.stderr or "").lower():
        pytest.skip("sanitizer runtime not available: " + r.stderr[-300:])
    assert r.returncode == 0, r.stderr
    s = S.ModelShape(n_layers=2, hidden=64, n_q_heads=4, n_kv_heads=2, head_dim=16, ffn=96, n_codes=7, vocab=40,
                     max_draft=4, dtype=dtype)
    blob = tmp_path / "w.bin"
    blob.write_bytes(S.make_weights(s, seed=2, std=0.3, offset_std=0.5))
    f, c0 = S.frame_inputs(s, 1)
    u = S.uniforms(1, s.n_codes)
    inp = tmp_path / "in.bin"
    inp.write_bytes(f[0].tobytes() + u[0].tobytes() + np.int32(c0[0]).tobytes())
    args = [str(blob), s.n_layers, s.hidden, s.n_q_heads, s.n_kv_heads, s.head_dim, s.ffn, s.n_codes, s.vocab,
            s.max_draft, s.dtype, 5, 3, str(inp), "x"]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:verify_asan_link_order=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe] + [str(a) for a in args], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert "ALL OK" in r.stdout
    assert "runtime error" not in r.stderr, r.stderr[-4000:]
