"""Host-side checks of the C ABI that need no GPU.

* librvqsd.so loads and exports every function include/rvqsd.h declares;
* the library's SplitMix64 uniform table equals the oracle's independent
  implementation and the published first outputs of the generator;
* argument errors come back as status codes with a message;
* the benchmark refuses more than one GPU.
"""
from __future__ import annotations

import ctypes
import json
import os
import re
import subprocess
import sys

import numpy as np
import pytest

from oracle import oracle as O
from paper_2609_37007_amd import rvqsd as R

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rvqsd.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rvqsd_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(R.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(R.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_uniform_table_matches_oracle_and_golden():
    gold = json.load(open(os.path.join(ROOT, "tests", "golden", "splitmix64_seed0.json")))
    first = [int(x, 16) for x in gold["outputs"]]
    u = R.uniforms_from_seed(0)
    for i, x in enumerate(first):
        assert u.reshape(-1)[i] == np.float32((x >> 40) / 2.0 ** 24)
    for seed in (0, 1, 2**32 + 5, 2**64 - 1):
        for n in (1, 7, 15):
            assert np.array_equal(R.uniforms_from_seed(seed, n), O.uniforms_from_seed(seed, n))
    u = R.uniforms_from_seed(99)
    assert (u >= 0).all() and (u < 1).all()


def test_argument_errors():
    L = R.lib()
    out = np.zeros((15, 3), dtype=np.float32)
    assert L.rvqsd_uniforms_from_seed(0, 0, out.ctypes.data_as(ctypes.c_void_p)) == R.EINVAL
    assert L.rvqsd_uniforms_from_seed(0, 16, out.ctypes.data_as(ctypes.c_void_p)) == R.EINVAL
    assert L.rvqsd_uniforms_from_seed(0, 15, None) == R.EINVAL
    assert L.rvqsd_last_error()
    h = ctypes.c_void_p()
    assert L.rvqsd_create(None, None, ctypes.byref(h)) == R.EINVAL
    assert b"null" in L.rvqsd_last_error()
    assert L.rvqsd_stream_create(None, None, 1, ctypes.byref(h)) == R.EINVAL
    assert L.rvqsd_set_trace(None, None) == R.EINVAL
    assert L.rvqsd_stream_reset(None) == R.EINVAL
    assert L.rvqsd_decode_frame_u(None, None, 0, None, None, None) == R.EINVAL
    assert L.rvqsd_decode_frame_async(None, None, None, None, None, None) == R.EINVAL
    assert L.rvqsd_decode_frames_async(None, 2, None, None, None, None, None) == R.EINVAL
    info = R.rvqsd_info()
    assert L.rvqsd_model_info(None, ctypes.byref(info)) == R.EINVAL
    L.rvqsd_destroy(None)
    L.rvqsd_stream_destroy(None)


def test_status_strings():
    L = R.lib()
    seen = set()
    for st in (R.OK, R.EINVAL, R.EBLOB, R.ENOMEM, R.EHIP, R.EUNSUPPORTED, R.ENUMERIC, R.ETIMEOUT):
        s = L.rvqsd_status_str(st)
        assert s and s not in seen
        seen.add(s)
    assert L.rvqsd_status_str(-100)


def test_bench_refuses_several_gpus():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=60)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


PRODUCT_SOURCES = sorted(
    [os.path.join("paper_2609_37007_amd", "csrc", f) for f in os.listdir(os.path.join(ROOT, "paper_2609_37007_amd", "csrc"))]
    + [os.path.join("paper_2609_37007_amd", f) for f in ("rvqsd.py", "build_ext.py", "__init__.py")]
    + [os.path.join("include", f) for f in os.listdir(os.path.join(ROOT, "include"))])


@pytest.mark.parametrize("name", PRODUCT_SOURCES)
def test_gpu_sources_do_not_touch_the_oracle(name):
    """The product path shares no code with the oracle: no source of the library, its
    header or its binding names the oracle or one of its symbols."""
    text = open(os.path.join(ROOT, name)).read()
    assert "oracle" not in text.lower() and "orc_" not in text
