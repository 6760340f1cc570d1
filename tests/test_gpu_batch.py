"""GPU parity of the batched path (several frame streams verified together).

Every frame decoded by rvqsd_decode_frames_batched is the same problem as a
single-frame decode, and is held to the same rule: with the per-frame trace
(rvqsd_set_batch_trace), every verify and draft logit row within 2e-2 of the
oracle's fp64 logits (bf16 weights), every decision replayed bit for bit from
the kernel's own logits, and the codes and statistics equal to the oracle's
from scratch unless the first round where the two runs part lies within reach
of the measured logit error.  Untraced frames use the largest logit error
measured on the traced ones (MEASURED) for the same rule, applied to the
oracle rounds up to the one that commits the first differing code.  The
single-stream path of the same library is a second reference.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import oracle as O
from paper_2609_37007_amd import synth as S
from tests import gpu_checks as GC
from tests.helpers import make_oracle, shape_kwargs

torch = pytest.importorskip("torch")
from paper_2609_37007_amd import rvqsd as R  # noqa: E402

pytestmark = pytest.mark.gpu

LOGIT_TOL = 2e-2
# largest logit error the traced frames of this module measured (updated as they run;
# the untraced frames' excuse rule uses it); starts at the single-stream path's level
MEASURED = {"err": 1e-4}
# 2 layers, hidden 512, GQA 8 q / 4 kv heads of 64, FFN 1024, 128 codes, bf16
SMALL = S.ModelShape(n_layers=2, hidden=512, n_q_heads=8, n_kv_heads=4, head_dim=64, ffn=1024, n_codes=15,
                     vocab=128, max_draft=14, dtype=S.DTYPE_BF16)


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


class BRig:
    """A model, a batched stream of `lanes` lanes, a single-frame stream and the oracle."""

    def __init__(self, s, lanes, topk, K, T=0.9, greedy=0):
        self.s, self.T, self.K, self.topk, self.greedy, self.lanes = s, T, K, topk, greedy, lanes
        blob = blob_of(s)
        self.model = R.Model(blob, R.make_cfg(**shape_kwargs(s), topk=topk, temperature=T, draft_len=K,
                                              draft_greedy=greedy))
        self.batch = R.Stream(self.model, max_streams=lanes)
        self.single = R.Stream(self.model)
        self.orc = make_oracle(s, blob, topk=topk, temperature=T, draft_len=K,
                               draft_mode=O.DRAFT_GREEDY if greedy else O.DRAFT_SAMPLED)

    def close(self):
        self.batch.close()
        self.single.close()
        self.model.close()
        self.orc.close()

    def traced_batch(self, f, c0, u, n_traced, max_rounds=16):
        """Batched decode with the first n_traced frames traced; returns codes, stats and
        get(i) -> (codes, stats dict, logits, round records) for a traced frame."""
        slots = self.model.info()["trace_slots"]
        V = self.s.vocab
        lg = torch.zeros((n_traced, max_rounds, slots, V), dtype=torch.float32, device="cuda")
        rd = torch.full((n_traced, max_rounds, R.TRACE_ROUND_INTS), -1, dtype=torch.int32, device="cuda")
        torch.cuda.synchronize()
        self.batch.set_batch_trace(lg.data_ptr(), rd.data_ptr(), max_rounds, n_traced)
        try:
            codes, st = self.batch.decode_frames_batched(f, c0, u)
        finally:
            self.batch.set_batch_trace()
        torch.cuda.synchronize()
        lgh, rdh = lg.cpu().numpy(), rd.cpu().numpy()

        def get(i):
            sd = {k: int(st[k][i]) for k in st.dtype.names}
            return codes[i], sd, lgh[i], rdh[i][:sd["target_calls"]]

        return codes, st, get


def near_threshold(rig, f, c0, u, codes):
    """The oracle rounds up to the one committing the first differing code: some decision
    within reach of the largest logit error measured on traced batched frames."""
    return GC.untraced_divergence_near(rig, f, c0, u, codes, MEASURED["err"])


def check_traced(rig, f, c0, u, get, frames, max_excused):
    worst, excused = GC.check_traced_frames(rig, frames, f, c0, u, get, LOGIT_TOL, excuse_frac=1.0)
    MEASURED["err"] = max(MEASURED["err"], worst)
    assert excused <= max_excused, excused
    return worst, excused


def check_against_oracle(rig, f, c0, u, codes, st, frames, max_excused):
    excused = []
    for i in frames:
        assert st["status"][i] == 0, (i, st["status"][i])
        oc, ost, _ = rig.orc.spec_frame(f[i], int(c0[i]), u[i])
        if np.array_equal(oc, codes[i]):
            for k in ("target_calls", "rounds", "drafted", "accepted", "accept_mask"):
                assert st[k][i] == ost[k], (i, k, st[k][i], ost[k])
        else:
            assert near_threshold(rig, f[i], c0[i], u[i], codes[i]), \
                f"frame {i}: codes differ with no decision near a threshold: {codes[i].tolist()} vs {oc.tolist()}"
            excused.append(i)
    assert len(excused) <= max_excused, excused
    return excused


def check_against_single(rig, f, c0, u, codes, frames):
    """The single-frame path of the same library: equal codes, or a near-threshold frame."""
    differ = []
    for i in frames:
        sc, _ = rig.single.decode_frame_u(f[i], int(c0[i]), u[i])
        if not np.array_equal(sc, codes[i]):
            assert near_threshold(rig, f[i], c0[i], u[i], codes[i]) or \
                near_threshold(rig, f[i], c0[i], u[i], sc), (i, sc.tolist(), codes[i].tolist())
            differ.append(i)
    return differ


def test_small_4_lanes_matches_oracle():
    """24 frames, 4 lanes (6 frames per lane in sequence), draft length 3, top-k 16;
    every frame traced: logits, decision replay and the oracle from scratch."""
    rig = BRig(SMALL, lanes=4, topk=16, K=3)
    n = 24
    f, c0 = S.frame_inputs(SMALL, n)
    u = S.uniforms(n)
    print("small bf16, 4 lanes, K=3: 24 frames, traced", flush=True)
    codes, st, get = rig.traced_batch(f, c0, u, n)
    assert ((codes >= 0) & (codes < SMALL.vocab)).all()
    assert (st["target_calls"] == st["rounds"] + 1).all()
    worst, ex = check_traced(rig, f, c0, u, get, range(n), max_excused=2)
    d = check_against_single(rig, f, c0, u, codes, range(n))
    untraced, _ = rig.batch.decode_frames_batched(f, c0, u)
    assert np.array_equal(untraced, codes)  # the trace changes nothing
    passes, nbytes = rig.batch.batch_totals()
    # every lane runs its frames one after another inside the shared passes
    per_lane = [int(st["target_calls"][i::4].sum()) for i in range(4)]
    assert passes >= max(per_lane) and passes <= sum(per_lane)
    assert nbytes > 0
    print(f"max logit error {worst:.3g}, excused {ex}, differ from single-stream {d}, passes {passes} "
          f"(lanes {per_lane})", flush=True)
    rig.close()


@pytest.mark.timeout(900)
def test_mcd1024_16_lanes_matches_oracle():
    """The 1024-wide bf16 model, 16 lanes (M = 80 rows), draft length 4, top-k 50:
    48 frames; the first 16 traced (logits within 2e-2, decisions replayed, oracle
    end to end), the others against the oracle (every third) and the single-stream
    path under the rule with the measured logit error."""
    s = S.MCD_1024
    rig = BRig(s, lanes=16, topk=50, K=4)
    n = 48
    f, c0 = S.frame_inputs(s, n)
    u = S.uniforms(n)
    print("mcd1024 bf16, 16 lanes, K=4: 48 frames, 16 traced", flush=True)
    codes, st, get = rig.traced_batch(f, c0, u, 16)
    assert ((codes >= 0) & (codes < s.vocab)).all()
    worst, ex = check_traced(rig, f, c0, u, get, range(16), max_excused=2)
    print(f"traced frames: max logit error {worst:.3g}, excused {ex}", flush=True)
    ex2 = check_against_oracle(rig, f, c0, u, codes, st, range(18, n, 3), max_excused=2)
    d = check_against_single(rig, f, c0, u, codes, range(n))
    assert len(d) <= 3, d
    print(f"untraced excused vs oracle {ex2}, differ from single-stream {d}", flush=True)
    rig.close()


def test_frames_do_not_depend_on_lane_or_neighbours():
    """The same frames in another order (other lanes, other neighbours) give the same codes."""
    rig = BRig(SMALL, lanes=5, topk=16, K=3)
    n = 20
    f, c0 = S.frame_inputs(SMALL, n)
    u = S.uniforms(n)
    codes, _ = rig.batch.decode_frames_batched(f, c0, u)
    perm = np.random.default_rng(7).permutation(n)
    codes_p, _ = rig.batch.decode_frames_batched(f[perm], c0[perm], u[perm])
    assert np.array_equal(codes_p, codes[perm])
    again, _ = rig.batch.decode_frames_batched(f, c0, u)
    assert np.array_equal(again, codes)
    rig.close()


def test_ragged_counts_and_invalid_c0_async():
    """n not a multiple of the lanes, n below the lanes, and (async) one frame with a bad c0
    and one with a uniform outside [0, 1)."""
    rig = BRig(SMALL, lanes=4, topk=16, K=2)
    n = 7
    f, c0 = S.frame_inputs(SMALL, n)
    u = S.uniforms(n)
    codes, st, get = rig.traced_batch(f, c0, u, n)
    check_traced(rig, f, c0, u, get, range(n), max_excused=1)
    two, _ = rig.batch.decode_frames_batched(f[:2], c0[:2], u[:2])
    assert np.array_equal(two, codes[:2])
    bad = c0.copy()
    bad[3] = SMALL.vocab + 5
    d_f = torch.from_numpy(f).cuda()
    d_c0 = torch.from_numpy(bad).cuda()
    ubad = np.ascontiguousarray(u).copy()
    ubad[5, 0, 1] = np.nan
    d_u = torch.from_numpy(ubad).cuda()
    d_codes = torch.zeros((n, SMALL.n_codes), dtype=torch.int32, device="cuda")
    sb = R.STATS_DTYPE.itemsize
    d_st = torch.zeros(n * sb, dtype=torch.uint8, device="cuda")
    rig.batch.decode_frames_batched_async(n, d_f.data_ptr(), d_c0.data_ptr(), d_u.data_ptr(), d_codes.data_ptr(),
                                          d_st.data_ptr())
    torch.cuda.synchronize()
    acodes = d_codes.cpu().numpy()
    ast = np.frombuffer(d_st.cpu().numpy().tobytes(), dtype=R.STATS_DTYPE)
    for i in (3, 5):
        assert ast["status"][i] == R.EINVAL and (acodes[i] == -1).all(), i
    ok = [i for i in range(n) if i not in (3, 5)]
    assert (ast["status"][ok] == 0).all()
    assert np.array_equal(acodes[ok], codes[ok])
    with pytest.raises(R.RvqsdError):
        rig.batch.decode_frames_batched(f, bad, u)
    rig.close()


def test_k0_batched_is_autoregressive():
    """Draft length 0: two rows per lane (prefix) then one; codes = plain top-k sampling."""
    rig = BRig(SMALL, lanes=8, topk=16, K=0)
    n = 16
    f, c0 = S.frame_inputs(SMALL, n)
    u = S.uniforms(n)
    codes, st, get = rig.traced_batch(f, c0, u, n)
    assert (st["target_calls"] == SMALL.n_codes).all()
    _, excused = check_traced(rig, f, c0, u, get, range(n), max_excused=1)
    for i in range(n):
        ar = rig.orc.ar_frame(f[i], int(c0[i]), u[i])
        oc, _, _ = rig.orc.spec_frame(f[i], int(c0[i]), u[i])
        assert np.array_equal(ar, oc)  # draft length 0 is plain top-k sampling
        if not np.array_equal(ar, codes[i]):
            excused -= 1
    assert excused >= 0
    rig.close()


def test_greedy_drafts_batched():
    rig = BRig(SMALL, lanes=4, topk=16, K=4, greedy=1)
    n = 12
    f, c0 = S.frame_inputs(SMALL, n)
    u = S.uniforms(n)
    codes, st, get = rig.traced_batch(f, c0, u, n)
    check_traced(rig, f, c0, u, get, range(n), max_excused=1)
    rig.close()


def test_batched_needs_a_batched_stream():
    rig = BRig(SMALL, lanes=2, topk=16, K=3)
    f, c0 = S.frame_inputs(SMALL, 2)
    u = S.uniforms(2)
    with pytest.raises(R.RvqsdError) as e:
        rig.single.decode_frames_batched(f, c0, u)
    assert e.value.status == R.EUNSUPPORTED
    rig.close()
    # 16 lanes x (K + 1 = 6 rows) exceeds the 80 rows of a pass
    model = R.Model(blob_of(SMALL), R.make_cfg(**shape_kwargs(SMALL), topk=16, temperature=0.9, draft_len=5))
    with pytest.raises(R.RvqsdError) as e:
        R.Stream(model, max_streams=16)
    assert e.value.status == R.EUNSUPPORTED
    model.close()
