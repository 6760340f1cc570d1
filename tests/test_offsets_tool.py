"""The offline offset-training tool (paper_2609_37007_amd/offsets.py), on the CPU.

Its PyTorch forward must be the target model (checked against the oracle's fp64
forward), the drafter pairs must cover every anchor k >= 1 and distance j <= K with
k + j <= n, and one epoch on the tiny model must run and return offsets of the
blob's shape."""
import numpy as np
import pytest

from paper_2609_37007_amd import offsets as OF
from paper_2609_37007_amd import synth as S
from tests import helpers as Hh

torch = pytest.importorskip("torch")


def test_torch_forward_is_the_target_model():
    s = S.ModelShape(n_layers=2, hidden=64, n_q_heads=4, n_kv_heads=2, head_dim=16, ffn=96, n_codes=7, vocab=24,
                     max_draft=3, dtype=S.DTYPE_BF16)
    blob = S.make_weights(s, seed=5, std=0.2)
    dec = OF.Decoder(s, blob, "cpu")
    orc = Hh.make_oracle(s, blob, topk=4, temperature=0.9, draft_len=1)
    f, c0 = S.frame_inputs(s, 2)
    rng = np.random.default_rng(1)
    for i in range(2):
        codes = [int(c0[i])] + [int(x) for x in rng.integers(0, s.vocab, s.n_codes - 1)]
        ref = orc.forward(f[i], codes)
        x = dec.inputs(torch.from_numpy(f[i:i + 1]), torch.tensor([codes]))
        got = dec.forward(x)[0].double().numpy()
        assert np.abs(got - ref).max() < 1e-4
    orc.close()


def test_draft_pairs_cover_the_drafter():
    pairs = OF.draft_pairs(15, 4)
    seen = {(k, t - k) for t, ks, js in pairs for k in ks}
    want = {(k, j) for k in range(1, 15) for j in range(1, 5) if k + j <= 15}
    assert seen == want


def test_one_epoch_on_the_tiny_model():
    s = S.TINY
    blob = S.make_weights(s, seed=0)
    b, hist = OF.train(s, blob, frames=64, K=3, topk=8, T=0.9, epochs=1, device="cpu", log=lambda m: None,
                       compare={"seed": S.unpack_weights(s, blob)["offsets"]})
    assert b.shape == (3, s.hidden) and b.dtype == np.float32
    assert len(hist) == 2 and len(hist[0]["accept"]) == 3 and "seed_accept" in hist[0]
    assert all(0.0 <= a <= 1.0 for a in hist[-1]["accept"])
