"""The allocation-free frame decode (rvqsd_decode_frame_noalloc) against the
stream path it is a variant of (rvqsd_decode_frame_async on a fresh stream):
the same kernel over the same inputs, so the codes and statistics must be equal
bit for bit, and both must pass the oracle's parity rule. Two models in a row
(the second with smaller frame buffers), then the first again, show that each
call starts from a clean region of the shared array.
"""
from __future__ import annotations

import numpy as np
import pytest

from paper_2609_37007_amd import synth as S
from tests import gpu_checks as GC
from tests.helpers import make_oracle, shape_kwargs

torch = pytest.importorskip("torch")
from paper_2609_37007_amd import rvqsd as R  # noqa: E402

pytestmark = pytest.mark.gpu

KEYS = ("target_calls", "rounds", "drafted", "accepted", "accept_mask", "status")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    R.lib()


def _decode(s, blob, K, topk, frames, use_noalloc):
    """Decode frames of s through one of the two entry points on torch's stream."""
    ts = torch.cuda.current_stream()
    model = R.Model(blob, R.make_cfg(**shape_kwargs(s), topk=topk, temperature=0.9, draft_len=K))
    stream = None if use_noalloc else R.Stream(model, hip_stream=ts.cuda_stream)
    N = max(frames) + 1
    f, c0 = S.frame_inputs(s, N)
    u = S.uniforms(N, s.n_codes)
    d_f = torch.from_numpy(f).cuda()
    d_c0 = torch.from_numpy(c0).cuda()
    d_u = torch.from_numpy(np.ascontiguousarray(u)).cuda()
    n, H, sb = s.n_codes, s.hidden, R.STATS_DTYPE.itemsize
    d_codes = torch.full((N, n), -7, dtype=torch.int32, device="cuda")
    d_st = torch.zeros(N * sb, dtype=torch.uint8, device="cuda")
    for i in frames:
        args = (d_f.data_ptr() + i * H * 4, d_c0.data_ptr() + i * 4, d_u.data_ptr() + i * n * 12,
                d_codes.data_ptr() + i * n * 4, d_st.data_ptr() + i * sb)
        if use_noalloc:
            model.decode_frame_noalloc(ts.cuda_stream, *args)
        else:
            stream.decode_frame_async(*args)
    torch.cuda.synchronize()
    codes = d_codes.cpu().numpy()
    st = np.frombuffer(d_st.cpu().numpy().tobytes(), dtype=R.STATS_DTYPE)
    if stream is not None:
        stream.close()
    model.close()
    return codes, st, f, c0, u


def _same(a, b, frames):
    ca, sa = a[0], a[1]
    cb, sb = b[0], b[1]
    for i in frames:
        assert np.array_equal(ca[i], cb[i]), (i, ca[i].tolist(), cb[i].tolist())
        for k in KEYS:
            assert int(sa[k][i]) == int(sb[k][i]), (i, k)


def _oracle_rule(s, blob, K, topk, res, frames):
    codes, st, f, c0, u = res
    orc = make_oracle(s, blob, topk=topk, temperature=0.9, draft_len=K)
    rig = type("Rig", (), dict(s=s, K=K, topk=topk, T=0.9, greedy=0, orc=orc))()
    for i in frames:
        assert int(st["status"][i]) == 0
        assert GC.untraced_divergence_near(rig, f[i], int(c0[i]), u[i], codes[i], 1e-4), i
    orc.close()


def test_noalloc_matches_the_stream_path_on_two_models_in_a_row():
    big = S.MCD_1024
    small = S.TINY
    bblob = S.make_weights(big, seed=0)
    sblob = S.make_weights(small, seed=0)
    frames = [0, 1, 2]
    print("noalloc: mcd1024 K=4, 3 frames", flush=True)
    ref = _decode(big, bblob, 4, 50, frames, use_noalloc=False)
    got = _decode(big, bblob, 4, 50, frames, use_noalloc=True)
    _same(ref, got, frames)
    _oracle_rule(big, bblob, 4, 50, got, frames)
    # second call with a smaller input: the tiny model's frame region is a prefix of the last one
    print("noalloc: tiny K=3, 4 frames", flush=True)
    sf = [0, 1, 2, 3]
    sref = _decode(small, sblob, 3, 8, sf, use_noalloc=False)
    sgot = _decode(small, sblob, 3, 8, sf, use_noalloc=True)
    _same(sref, sgot, sf)
    _oracle_rule(small, sblob, 3, 8, sgot, sf)
    # and the large model again, after the small one left its state in the array
    again = _decode(big, bblob, 4, 50, [2], use_noalloc=True)
    _same(ref, again, [2])


def test_noalloc_rejects_oversize_models_and_null_arguments():
    # 4096 codes at draft length 14: 18.8 MB of frame buffers, more than the 16 MiB array
    s = S.ModelShape(n_layers=1, hidden=256, n_q_heads=4, n_kv_heads=4, head_dim=64, ffn=512, n_codes=15,
                     vocab=4096, max_draft=14, dtype=S.DTYPE_F32)
    model = R.Model(S.make_weights(s, seed=0), R.make_cfg(**shape_kwargs(s), topk=8, temperature=0.9, draft_len=14))
    buf = torch.zeros(1 << 16, dtype=torch.uint8, device="cuda")
    p = buf.data_ptr()
    with pytest.raises(R.RvqsdError) as e:
        model.decode_frame_noalloc(torch.cuda.current_stream().cuda_stream, p, p + 4096, p + 8192, p + 12288,
                                   p + 16384)
    assert e.value.status == R.EUNSUPPORTED and "16777216" in str(e.value)
    with pytest.raises(R.RvqsdError) as e:
        model.decode_frame_noalloc(torch.cuda.current_stream().cuda_stream, 0, p, p, p, p)
    assert e.value.status == R.EINVAL
    model.close()
