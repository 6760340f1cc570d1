"""GPU parity of the W8A16 weight path (Sec. 3.4): int8 codes with fp32 per-output-
channel scales, decoded on MFMA, against the oracle over the same int8 blob (the
dequantized weights s * q in fp64). Same rule as the bf16 model: logits within
2e-2, decisions replayed exactly, the oracle end to end."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2609_37007_amd import synth as S
from tests.helpers import shape_kwargs

torch = pytest.importorskip("torch")
from paper_2609_37007_amd import rvqsd as R  # noqa: E402
from tests.test_gpu_parity import Rig, blob_of, check_frames, shape_with  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    R.lib()


@pytest.mark.parametrize("K", [0, 2, 4, 7])
def test_mcd1024_w8_frames(K):
    """The 1024-wide model with int8 weights, every matrix-core instantiation (2, 4, 5, 8 rows)."""
    s = S.MCD_1024_W8
    rig = Rig(s, topk=50, K=K)
    f, c0 = S.frame_inputs(s, 3)
    u = S.uniforms(3)
    print(f"mcd1024 int8 K={K}: frames 0..2", flush=True)
    worst, excused = check_frames(rig, range(3), f, c0, u)
    print(f"max logit error {worst:.3g}, excused {excused}", flush=True)
    if K == 0:
        for i in range(3):
            codes, _ = rig.stream.decode_frame_u(f[i], int(c0[i]), u[i])
            assert np.array_equal(codes, rig.orc.ar_frame(f[i], int(c0[i]), u[i]))
    rig.close()


def test_small_w8_async_and_noalloc_agree():
    """A 512-wide int8 model: the async stream path and the allocation-free decode give the same
    codes, and both match the oracle."""
    s = S.ModelShape(n_layers=2, hidden=512, n_q_heads=8, n_kv_heads=4, head_dim=64, ffn=1024, n_codes=15,
                     vocab=128, max_draft=14, dtype=S.DTYPE_I8)
    rig = Rig(s, topk=16, K=3, hip_stream=torch.cuda.current_stream().cuda_stream)
    f, c0 = S.frame_inputs(s, 4)
    u = S.uniforms(4)
    check_frames(rig, range(4), f, c0, u)
    d_f = torch.from_numpy(f).cuda()
    d_c0 = torch.from_numpy(c0).cuda()
    d_u = torch.from_numpy(np.ascontiguousarray(u)).cuda()
    n, H, sb = s.n_codes, s.hidden, R.STATS_DTYPE.itemsize
    a = torch.full((4, n), -1, dtype=torch.int32, device="cuda")
    b = torch.full((4, n), -1, dtype=torch.int32, device="cuda")
    sa = torch.zeros(4 * sb, dtype=torch.uint8, device="cuda")
    sbuf = torch.zeros(4 * sb, dtype=torch.uint8, device="cuda")
    ts = torch.cuda.current_stream().cuda_stream
    for i in range(4):
        args = (d_f.data_ptr() + i * H * 4, d_c0.data_ptr() + i * 4, d_u.data_ptr() + i * n * 12)
        rig.stream.decode_frame_async(*args, a.data_ptr() + i * n * 4, sa.data_ptr() + i * sb)
        rig.model.decode_frame_noalloc(ts, *args, b.data_ptr() + i * n * 4, sbuf.data_ptr() + i * sb)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    for i in range(4):
        codes, _ = rig.stream.decode_frame_u(f[i], int(c0[i]), u[i])
        assert np.array_equal(codes, a[i].cpu().numpy())
    rig.close()


def test_w8_limits():
    s = S.ModelShape(n_layers=1, hidden=512, n_q_heads=8, n_kv_heads=4, head_dim=64, ffn=1024, n_codes=15,
                     vocab=128, max_draft=14, dtype=S.DTYPE_I8)
    blob = S.make_weights(s, seed=0)
    with pytest.raises(R.RvqsdError) as e:  # 15 rows: beyond the matrix-core path
        R.Model(blob, R.make_cfg(**shape_kwargs(s), topk=16, temperature=0.9, draft_len=14))
    assert e.value.status == R.EUNSUPPORTED
    with pytest.raises(R.RvqsdError) as e:  # int8 codes are widened for the matrix cores only
        R.Model(blob, R.make_cfg(**shape_kwargs(s), topk=16, temperature=0.9, draft_len=3, matrix_path=1))
    assert e.value.status == R.EUNSUPPORTED
    model = R.Model(blob, R.make_cfg(**shape_kwargs(s), topk=16, temperature=0.9, draft_len=3))
    with pytest.raises(R.RvqsdError) as e:  # the batched kernel reads bf16 only
        R.Stream(model, max_streams=4)
    assert e.value.status == R.EUNSUPPORTED
    info = model.info()
    assert info["emb_row_bytes"] == s.hidden + 4
    assert info["head_bytes"] == S.mat_bytes(s, (s.vocab, s.hidden))
    model.close()
