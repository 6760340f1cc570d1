"""GPU parity of sparse-tree verification (Sec. 2.2, "Tree attention increases
acceptance rate", Fig. 2): the batched kernel's tree lanes against the oracle's
tree frame, through the C ABI (rvqsd_tree_stream_create).

Every traced frame: every verify and draft logit row within 2e-2 of the oracle's
fp64 logits over the same packed rows (bf16 weights); every decision (the ranked
candidates of each depth, the sibling walks, the residual draws) replayed bit for
bit from the kernel's own logits; and the codes and statistics of the oracle from
scratch, a difference excused only when the first round where the two runs part
lies within reach of the measured logit error.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import oracle as O
from paper_2609_37007_amd import synth as S
from paper_2609_37007_amd import tree as TR
from tests import gpu_checks as GC
from tests.helpers import make_oracle, shape_kwargs

torch = pytest.importorskip("torch")
from paper_2609_37007_amd import rvqsd as R  # noqa: E402

pytestmark = pytest.mark.gpu

LOGIT_TOL = 2e-2
ROUND_INTS = 128
SMALL = S.ModelShape(n_layers=2, hidden=512, n_q_heads=8, n_kv_heads=4, head_dim=64, ffn=1024, n_codes=15,
                     vocab=128, max_draft=14, dtype=S.DTYPE_BF16)
FIG2 = ([0, 0, 1, 1, 2, 3, 5, 5], [0, 1, 0, 1, 0, 0, 0, 1])


def calibrated(N, K, decay=0.5, depth_decay=0.8):
    """A greedy tree from a geometric per-depth, per-rank acceptance table."""
    P = [[(decay ** (r + 1)) * (depth_decay ** d) for r in range(8)] for d in range(K)]
    return TR.pack(TR.greedy_tree(P, N, K))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    R.lib()


_blobs = {}


def blob_of(s):
    if s not in _blobs:
        _blobs[s] = S.make_weights(s, seed=0)
    return _blobs[s]


class TreeRig:
    def __init__(self, s, tree, topk, K, lanes=1, T=0.9):
        self.s, self.tree, self.topk, self.K, self.T, self.greedy = s, tree, topk, K, T, 0
        blob = blob_of(s)
        self.model = R.Model(blob, R.make_cfg(**shape_kwargs(s), topk=topk, temperature=T, draft_len=K))
        self.stream = R.Stream(self.model, max_streams=lanes, tree=tree)
        self.orc = make_oracle(s, blob, topk=topk, temperature=T, draft_len=K)
        self.otree = O.make_tree(*tree)
        self.slot0 = max(16, len(tree[0]) + 1)
        self.slots = self.slot0 + (len(tree[0]) + 1) * K

    def close(self):
        self.stream.close()
        self.model.close()
        self.orc.close()

    def traced(self, f, c0, u, n_traced, max_rounds=16):
        V = self.s.vocab
        lg = torch.zeros((n_traced, max_rounds, self.slots, V), dtype=torch.float32, device="cuda")
        rd = torch.full((n_traced, max_rounds, ROUND_INTS), -1, dtype=torch.int32, device="cuda")
        torch.cuda.synchronize()
        self.stream.set_batch_trace(lg.data_ptr(), rd.data_ptr(), max_rounds, n_traced)
        try:
            codes, st = self.stream.decode_frames_batched(f, c0, u)
        finally:
            self.stream.set_batch_trace()
        torch.cuda.synchronize()
        lgh, rdh = lg.cpu().numpy(), rd.cpu().numpy()

        def get(i):
            sd = {k: int(st[k][i]) for k in st.dtype.names}
            return codes[i], sd, lgh[i], rdh[i][:sd["target_calls"]]

        return codes, st, get


def run_case(s, tree, topk, K, n, lanes=1, n_traced=None, excuse=1):
    rig = TreeRig(s, tree, topk, K, lanes=lanes)
    f, c0 = S.frame_inputs(s, n)
    u = S.uniforms(n, s.n_codes)
    codes, st, get = rig.traced(f, c0, u, n_traced or n)
    assert (st["status"] == 0).all()
    assert ((codes >= 0) & (codes < s.vocab)).all()
    worst, ex = GC.check_tree_frames(rig, range(n_traced or n), f, c0, u, get, LOGIT_TOL, excuse_frac=1.0)
    assert ex <= excuse, ex
    calls = int(st["target_calls"].sum())
    print(f"{len(tree[0])} nodes, {lanes} lane(s): max logit error {worst:.3g}, excused {ex}, "
          f"tokens/call {s.n_codes * n / calls:.3f}", flush=True)
    rig.close()
    return codes, st


def test_fig2_tree_small_model():
    """The tree of Fig. 2 (8 nodes, depth 3) on a 2-layer bf16 model, 12 frames."""
    run_case(SMALL, FIG2, topk=16, K=3, n=12)


def test_calibrated_tree_two_lanes():
    """A 15-node greedy tree of depth 4, two frames in flight (32 rows per pass)."""
    run_case(SMALL, calibrated(15, 4), topk=16, K=4, n=8, lanes=2)


def test_63_node_tree_fills_four_mfma_tiles():
    """64 rows (63 nodes of depth <= 4): four 16-row MFMA tiles, 79 KV slots."""
    run_case(SMALL, calibrated(63, 4), topk=32, K=4, n=4)


@pytest.mark.timeout(600)
def test_mcd1024_16_node_tree():
    """The 1024-wide model with a 16-node greedy tree (17 rows), draft depth 4, top-k 50."""
    run_case(S.MCD_1024, calibrated(16, 4), topk=50, K=4, n=3)


def test_width1_tree_is_the_greedy_chain_on_the_gpu():
    """A chain of rank-0 candidates: the same codes as the oracle's greedy chain."""
    K = 3
    codes, st = run_case(SMALL, (list(range(K)), [0] * K), topk=16, K=K, n=6)
    blob = blob_of(SMALL)
    orc = make_oracle(SMALL, blob, topk=16, temperature=0.9, draft_len=K, draft_mode=O.DRAFT_GREEDY)
    f, c0 = S.frame_inputs(SMALL, 6)
    u = S.uniforms(6)
    same = sum(int(np.array_equal(orc.spec_frame(f[i], int(c0[i]), u[i])[0], codes[i])) for i in range(6))
    assert same >= 5, same
    orc.close()


def test_single_frame_calls_on_a_tree_stream():
    """rvqsd_decode_frame_u on a tree stream runs the frame through the tree kernel."""
    rig = TreeRig(SMALL, FIG2, topk=16, K=3)
    f, c0 = S.frame_inputs(SMALL, 3)
    u = S.uniforms(3)
    batched, _ = rig.stream.decode_frames_batched(f, c0, u)
    for i in range(3):
        one, st = rig.stream.decode_frame_u(f[i], int(c0[i]), u[i])
        assert np.array_equal(one, batched[i]) and st["status"] == 0
    rig.close()


def test_malformed_and_oversize_trees_are_rejected():
    model = R.Model(blob_of(SMALL), R.make_cfg(**shape_kwargs(SMALL), topk=16, temperature=0.9, draft_len=3))
    bad = [([1], [0]),                 # parent not an earlier row
           ([0, 0], [0, 0]),            # siblings of the same rank
           ([0, 1, 0], [0, 0, 1]),      # not breadth first
           ([0, 1, 2, 3], [0, 0, 0, 0]),  # deeper than draft_len 3
           ([0], [16])]                 # rank outside the top-16
    for tree in bad:
        with pytest.raises(R.RvqsdError) as e:
            R.Stream(model, tree=tree)
        assert e.value.status == R.EINVAL, tree
    with pytest.raises(R.RvqsdError) as e:
        R.Stream(model, max_streams=8, tree=calibrated(15, 3))  # 8 x 16 rows > 80
    assert e.value.status == R.EUNSUPPORTED
    model.close()
