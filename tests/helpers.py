"""Test helpers: shape plumbing and the exact-law enumerator (no method arithmetic)."""
from __future__ import annotations

import collections
import math

import numpy as np

from oracle import oracle as O
from paper_2609_37007_amd import synth as S


def shape_kwargs(s: S.ModelShape) -> dict:
    return dict(n_layers=s.n_layers, hidden=s.hidden, n_q_heads=s.n_q_heads, n_kv_heads=s.n_kv_heads,
                head_dim=s.head_dim, ffn=s.ffn, n_codes=s.n_codes, vocab=s.vocab, max_draft=s.max_draft,
                dtype=s.dtype)


def make_oracle(s: S.ModelShape, blob: bytes, **kw) -> O.Oracle:
    args = shape_kwargs(s)
    args.update(kw)
    return O.Oracle(blob, **args)


def micro_shape(vocab: int, n_codes: int, max_draft: int | None = None) -> S.ModelShape:
    """A one-layer model small enough for exact enumeration."""
    return S.ModelShape(n_layers=1, hidden=16, n_q_heads=2, n_kv_heads=1, head_dim=8, ffn=32, n_codes=n_codes,
                        vocab=vocab, max_draft=max(1, n_codes - 1) if max_draft is None else max_draft,
                        dtype=S.DTYPE_F32)


def enumerate_law(run, n_slots: int, rng: np.random.Generator | None = None, check_points: int = 2):
    """Exact law of the output of ``run`` over i.i.d. U[0,1) uniforms.

    ``run(u)`` takes float32 uniforms [n_slots] and returns (outcome, events) where
    events lists (uniform index, breakpoints) in consumption order: the decision
    taken with that uniform changes only at those points.  Each uniform's
    interval is split at the breakpoints that fall inside it, depth first, until
    every consumed uniform sits in an interval with no breakpoint inside; the
    leaf's probability is the product of the interval widths.  At each leaf the
    outcome is re-checked at random points of the box.
    """
    rng = rng or np.random.default_rng(0)
    law = collections.defaultdict(float)
    stack = [dict()]
    leaves = 0
    while stack:
        fixed = stack.pop()
        u = np.full(n_slots, 0.5, dtype=np.float32)
        for i, (lo, hi) in fixed.items():
            mid = np.float32(0.5 * (lo + hi))
            if not (lo < float(mid) < hi):
                raise AssertionError(f"interval too narrow for float32 uniforms: {lo} {hi}")
            u[i] = mid
        outcome, events = run(u)
        split = None
        for idx, bps in events:
            lo, hi = fixed.get(idx, (0.0, 1.0))
            inner = sorted(set(b for b in bps if lo < b < hi))
            if idx not in fixed or inner:
                split = (idx, lo, hi, inner)
                break
        if split is None:
            w = math.prod(hi - lo for lo, hi in fixed.values())
            law[outcome] += w
            leaves += 1
            for _ in range(check_points):
                v = u.copy()
                for i, (lo, hi) in fixed.items():
                    x = np.float32(lo + (hi - lo) * rng.uniform(0.05, 0.95))
                    if lo < float(x) < hi:
                        v[i] = x
                o2, _ = run(v)
                assert o2 == outcome, "outcome not constant on an enumeration box"
            continue
        idx, lo, hi, inner = split
        pts = [lo] + inner + [hi]
        for a, b in zip(pts[:-1], pts[1:]):
            if b > a:
                stack.append({**fixed, idx: (a, b)})
    return dict(law), leaves


def spec_runner(orc: O.Oracle, f, c0):
    n = orc.n

    def run(u):
        events = []

        def probe(ctx, idx, bps, nb):
            events.append((int(idx), [bps[i] for i in range(nb)]))

        codes, _, _ = orc.spec_frame(f, c0, u.reshape(n, 3), probe=probe)
        return tuple(int(c) for c in codes), events

    return run


def ar_law(orc: O.Oracle, f, c0, topk: int, temperature: float) -> dict:
    """Joint law of plain top-k sampling from its definition: prod_s p_s(c_s | c_<s)."""
    n = orc.n
    law = {}

    def rec(prefix, prob):
        s = len(prefix) + 1
        if s > n:
            law[tuple(prefix)] = prob
            return
        h = orc.forward(f, [c0] + prefix)
        lg = orc.logits(h[s], s)
        idx, p = O.topk_softmax(lg, topk, temperature)
        for t, pt in zip(idx, p):
            if pt > 0:
                rec(prefix + [int(t)], prob * pt)

    rec([], 1.0)
    return law
