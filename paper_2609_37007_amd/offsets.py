"""Offline training of the position-aware draft offsets b_1..b_K by self-distillation.

The method's drafter reads the hidden state h_k of the anchor position k, adds a
per-distance offset b_j and projects through the frozen head of position k + j
(Sec. 2.2, Fig. 3). The paper trains only these offsets, with the backbone,
tables and heads frozen: teacher forcing gives h_k at every inner position, and a
cross entropy of LMH_{k+j}(h_k + b_j) against the code c_{k+j} that followed is
summed over draft distances j <= K and all valid positions, with Adam at learning
rate 1e-3 and batch 32 (Sec. 2.2, "Training the offsets").

The paper's training data (VoxPopuli audio codes of the trained TTS model) is not
available here, so the codes come from the model itself: plain top-k sampling
(top-k, temperature T) from seeded synthetic frame inputs, i.e. the target
distribution the verifier accepts against. The logits are divided by T in the loss
so that the trained draft distribution is the one the runtime samples from.

This is an offline tool (PyTorch, any device), not part of the decode path: it
writes a float32 array [K][hidden] that replaces the offsets of a weight blob
(synth.make_weights(offsets=...)).

    python -m paper_2609_37007_amd.offsets --workload mcd1024 --frames 4096 \
        --out paper_2609_37007_amd/assets/offsets_mcd1024.npy
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
if os.path.dirname(HERE) not in sys.path:
    sys.path.insert(0, os.path.dirname(HERE))

from paper_2609_37007_amd import synth as S  # noqa: E402


class Decoder:
    """The target decoder as plain PyTorch modules-free math (fp32), for training only."""

    def __init__(self, s: S.ModelShape, blob: bytes, device, eps: float = 1e-6, base: float = 1e6):
        import torch
        self.torch = torch
        self.s, self.eps, self.dev = s, eps, device
        W = S.unpack_weights(s, blob)
        self.W = {k: torch.from_numpy(np.ascontiguousarray(v, dtype=np.float32)).to(device) for k, v in W.items()}
        d = s.head_dim
        pos = torch.arange(s.n_codes + 1, dtype=torch.float64)
        inv = base ** (-torch.arange(0, d // 2, dtype=torch.float64) * 2.0 / d)
        ang = pos[:, None] * inv[None, :]
        self.cos = torch.cos(ang).float().to(device)
        self.sin = torch.sin(ang).float().to(device)

    def _rms(self, x, g):
        return x * self.torch.rsqrt((x * x).mean(-1, keepdim=True) + self.eps) * g

    def _rope(self, v):  # v [B, S, heads, d], rotate-half on (i, i + d/2)
        n = v.shape[1]
        h = v.shape[-1] // 2
        c, sn = self.cos[:n, None, :], self.sin[:n, None, :]
        a, b = v[..., :h], v[..., h:]
        return self.torch.cat([a * c - b * sn, b * c + a * sn], dim=-1)

    def inputs(self, f, codes):
        """x_0 = f, x_s = E_{s-1}[codes[:, s-1]] for s = 1..codes.shape[1]."""
        torch = self.torch
        rows = [f[:, None, :]]
        for i in range(codes.shape[1]):
            rows.append(self.W[f"emb{i}"][codes[:, i]][:, None, :])
        return torch.cat(rows, dim=1)

    def forward(self, x):
        """Final-normed hidden states of x [B, S, H] (causal)."""
        torch = self.torch
        s = self.s
        B, n, H = x.shape
        nq, nkv, d = s.n_q_heads, s.n_kv_heads, s.head_dim
        mask = torch.full((n, n), float("-inf"), device=x.device).triu(1)
        for l in range(s.n_layers):
            a = self._rms(x, self.W[f"l{l}.attn_norm"])
            q = (a @ self.W[f"l{l}.wq"].T).view(B, n, nq, d)
            k = (a @ self.W[f"l{l}.wk"].T).view(B, n, nkv, d)
            v = (a @ self.W[f"l{l}.wv"].T).view(B, n, nkv, d)
            q = self._rope(self._rms(q, self.W[f"l{l}.q_norm"]))
            k = self._rope(self._rms(k, self.W[f"l{l}.k_norm"]))
            rep = nq // nkv
            k = k.repeat_interleave(rep, dim=2)
            v = v.repeat_interleave(rep, dim=2)
            sc = torch.einsum("bqhd,bkhd->bhqk", q, k) / math.sqrt(d) + mask
            o = torch.einsum("bhqk,bkhd->bqhd", sc.softmax(-1), v).reshape(B, n, nq * d)
            x = x + o @ self.W[f"l{l}.wo"].T
            b = self._rms(x, self.W[f"l{l}.mlp_norm"])
            x = x + (torch.nn.functional.silu(b @ self.W[f"l{l}.wgate"].T) * (b @ self.W[f"l{l}.wup"].T)) \
                @ self.W[f"l{l}.wdown"].T
        return self._rms(x, self.W["final_norm"])

    def topk_probs(self, logits, topk, T):
        """Top-k restricted, temperature-T softmax over the last axis (dense)."""
        torch = self.torch
        k = min(topk, logits.shape[-1])
        vals, idx = logits.topk(k, dim=-1)
        p = torch.zeros_like(logits)
        p.scatter_(-1, idx, torch.softmax(vals / T, dim=-1))
        return p

    def sample_frames(self, f, c0, topk, T, gen):
        """Plain top-k sampling of codes c_1..c_n for every frame (batched)."""
        torch = self.torch
        n = self.s.n_codes
        codes = c0[:, None]
        for s in range(1, n + 1):
            h = self.forward(self.inputs(f, codes))[:, s]
            p = self.topk_probs(h @ self.W[f"lmh{s}"].T, topk, T)
            nxt = torch.multinomial(p, 1, generator=gen)
            codes = torch.cat([codes, nxt], dim=1)
        return codes  # [B, n + 1]: c_0 .. c_n


def draft_pairs(n_codes, K):
    """(target position t, anchors k, distances j = t - k) of the drafter: anchors 1..n-1."""
    out = []
    for t in range(2, n_codes + 1):
        ks = [k for k in range(max(1, t - K), t)]
        if ks:
            out.append((t, ks, [t - k for k in ks]))
    return out


def loss_and_accept(dec, hs, codes, b, K, topk, T, with_accept=False):
    """Cross entropy of LMH_t((h_k + b_{t-k}) / T) against c_t summed over the drafter's
    (t, k) pairs, averaged over frames; optionally the expected acceptance
    sum_x min(p_t, q_t) per distance j (top-k restricted, temperature T)."""
    torch = dec.torch
    total = 0.0
    acc = torch.zeros(K, device=hs.device)
    cnt = torch.zeros(K, device=hs.device)
    for t, ks, js in draft_pairs(dec.s.n_codes, K):
        v = hs[:, ks, :] + b[[j - 1 for j in js]][None, :, :]          # [B, nk, H]
        lg = v @ dec.W[f"lmh{t}"].T / T                                  # [B, nk, V]
        tgt = codes[:, t][:, None].expand(-1, len(ks))
        total = total + torch.nn.functional.cross_entropy(lg.reshape(-1, lg.shape[-1]), tgt.reshape(-1),
                                                          reduction="sum")
        if with_accept:
            with torch.no_grad():
                p = dec.topk_probs(hs[:, t] @ dec.W[f"lmh{t}"].T, topk, T)[:, None, :]
                q = dec.topk_probs(lg * T, topk, T)
                a = torch.minimum(p, q).sum(-1).mean(0)                  # [nk]
                for j, aj in zip(js, a):
                    acc[j - 1] += aj
                    cnt[j - 1] += 1
    out = total / hs.shape[0]
    return (out, acc / cnt.clamp(min=1)) if with_accept else out


def train(s, blob, *, frames, K, topk, T, epochs, lr=1e-3, batch=32, seed=0, device=None, log=print,
          compare=None):
    """Returns the trained offsets [K][H] and the per-epoch history; compare: named
    offset arrays [>= K][H] whose validation loss and expected acceptance are reported
    in the history's first entry (e.g. the blob's own draw)."""
    import torch
    dev = torch.device(device or ("cuda" if torch.cuda.is_available() else "cpu"))
    dec = Decoder(s, blob, dev)
    f, c0 = S.frame_inputs(s, frames, seed_hidden=seed + 40, seed_c0=seed + 41)
    gen = torch.Generator(device=dev).manual_seed(seed)
    t0 = time.time()
    with torch.no_grad():
        fT = torch.from_numpy(f).to(dev)
        cT = torch.from_numpy(c0.astype(np.int64)).to(dev)
        codes, hs = [], []
        for a in range(0, frames, 512):
            c = dec.sample_frames(fT[a:a + 512], cT[a:a + 512], topk, T, gen)
            codes.append(c)
            hs.append(dec.forward(dec.inputs(fT[a:a + 512], c[:, :-1])))
        codes = torch.cat(codes)
        hs = torch.cat(hs)
    log(f"sampled {frames} frames and their hidden states in {time.time() - t0:.1f} s on {dev}")
    n_val = max(frames // 8, 1)
    hv, cv = hs[:n_val], codes[:n_val]
    ht, ct = hs[n_val:], codes[n_val:]
    b = torch.zeros(K, s.hidden, device=dev, requires_grad=True)
    opt = torch.optim.Adam([b], lr=lr)
    hist = []
    with torch.no_grad():
        l0, a0 = loss_and_accept(dec, hv, cv, b, K, topk, T, with_accept=True)
    hist.append(dict(epoch=0, val_loss=float(l0), accept=[float(x) for x in a0]))
    for name, arr in (compare or {}).items():
        with torch.no_grad():
            bc = torch.from_numpy(np.ascontiguousarray(arr[:K], dtype=np.float32)).to(dev)
            lc, ac = loss_and_accept(dec, hv, cv, bc, K, topk, T, with_accept=True)
        hist[0][f"{name}_val_loss"] = float(lc)
        hist[0][f"{name}_accept"] = [float(x) for x in ac]
        log(f"{name} offsets: val loss {float(lc):.4f}, expected acceptance {np.round(ac.cpu().numpy(), 4).tolist()}")
    log(f"epoch 0: val loss {float(l0):.4f}, expected acceptance by distance {np.round(a0.cpu().numpy(), 4).tolist()}")
    for ep in range(1, epochs + 1):
        perm = torch.randperm(ht.shape[0], generator=torch.Generator().manual_seed(seed + ep)).to(dev)
        for a in range(0, ht.shape[0], batch):
            idx = perm[a:a + batch]
            opt.zero_grad()
            loss = loss_and_accept(dec, ht[idx], ct[idx], b, K, topk, T)
            loss.backward()
            opt.step()
        with torch.no_grad():
            l1, a1 = loss_and_accept(dec, hv, cv, b, K, topk, T, with_accept=True)
        hist.append(dict(epoch=ep, val_loss=float(l1), accept=[float(x) for x in a1]))
        log(f"epoch {ep}: val loss {float(l1):.4f}, expected acceptance by distance "
            f"{np.round(a1.cpu().numpy(), 4).tolist()}")
    return b.detach().cpu().numpy().astype(np.float32), hist


WORKLOADS = {"mcd1024": ("MCD_1024", 50), "tiny": ("TINY", 8)}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--workload", default="mcd1024", choices=sorted(WORKLOADS))
    ap.add_argument("--frames", type=int, default=4096)
    ap.add_argument("--epochs", type=int, default=4)
    ap.add_argument("--max-draft", type=int, default=None, help="offsets to train (default: the blob's max_draft)")
    ap.add_argument("--temperature", type=float, default=0.9)
    ap.add_argument("--head-scale", type=float, default=1.0)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--device", default=None)
    ap.add_argument("--out", required=True)
    a = ap.parse_args(argv)
    shape_name, topk = WORKLOADS[a.workload]
    s = getattr(S, shape_name)
    K = a.max_draft or s.max_draft
    blob = S.make_weights(s, seed=0, head_scale=a.head_scale)
    seed_ofs = S.unpack_weights(s, blob)["offsets"]
    b, hist = train(s, blob, frames=a.frames, K=K, topk=topk, T=a.temperature, epochs=a.epochs, seed=a.seed,
                    device=a.device, compare={"seed_draw": seed_ofs})
    full = np.zeros((s.max_draft, s.hidden), dtype=np.float32)
    full[:K] = b
    os.makedirs(os.path.dirname(os.path.abspath(a.out)), exist_ok=True)
    np.save(a.out, full)
    with open(os.path.splitext(a.out)[0] + ".json", "w") as fh:
        json.dump(dict(workload=a.workload, frames=a.frames, epochs=a.epochs, trained=K, topk=topk,
                       temperature=a.temperature, head_scale=a.head_scale, seed=a.seed, lr=1e-3, batch=32,
                       history=hist), fh, indent=1)
    print(f"wrote {a.out}")
    return 0


if __name__ == "__main__":
    sys.exit(main())
