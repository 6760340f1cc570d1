"""Parity checks shared by the GPU test files (no GPU code here).

A "rig" is any object with the attributes s (ModelShape), K, topk, T, greedy
and orc (an oracle of the same configuration).  A traced frame is given as its
codes, the kernel's logits lg[pass][slot][vocab] (slot r < 16: verify row r;
16 + r*K + j - 1: draft row (r, j)) and its round records rd[pass][32]
(m, K', first_pos, rows, m_new, accepted, token, pass, drafts...).

Three checks, in order of strength (the GPU parity rule of the method's
decisions):

* logit_error: every traced verify and draft logit row against the oracle's fp64
  forward and heads on the same inputs;
* replay: the kernel's own fp32 logits through the oracle's decision primitives
  reproduce every draft, accept and code bit for bit, except a threshold within
  1e-6 of its uniform (summation-order rounding);
* compare_end_to_end: the oracle from scratch.  A frame may differ only if the
  first round where the oracle's and the kernel's decisions part lies within
  reach of the measured logit error (its uniform margin or its top-k / argmax
  gap).
"""
from __future__ import annotations

import numpy as np

from oracle import oracle as O

SLOT_DRAFT0 = 16
CDF_EXCUSE = 1e-6


def pass_rows(K, n, row):
    """Verify rows and (row, j) draft slots the kernel computes in one pass."""
    fp, R_, ps = int(row[2]), int(row[3]), int(row[7])
    verify = [r for r in range(R_) if (ps > 0 or r == 1) and fp + r >= 1]
    drafts = []
    for r in range(R_):
        s = fp + r
        if s < 1 or s > n - 1 or (ps == 0 and r != 1):
            continue
        drafts += [(r, j) for j in range(1, min(K, n - s) + 1)]
    return verify, drafts


def pass_inputs(codes_full, row):
    """Codes consumed by positions 1 .. first_pos+rows-1 of a traced pass:
    committed codes up to the anchor m, then the round's drafts."""
    m, fp, R_ = int(row[0]), int(row[2]), int(row[3])
    ic = []
    for s in range(1, fp + R_):
        x = s - 1
        ic.append(int(codes_full[x]) if x <= m else int(row[8 + (x - m - 1)]))
    return ic


def logit_error(rig, f, c0, codes, lg, rd):
    """Max-abs difference of every traced logit row from the oracle's fp64 logits."""
    K, n = rig.K, rig.s.n_codes
    codes_full = [int(c0)] + [int(c) for c in codes]
    worst = 0.0
    for i, row in enumerate(rd):
        h = rig.orc.forward(f, pass_inputs(codes_full, row))
        fp = int(row[2])
        verify, drafts = pass_rows(K, n, row)
        for r in verify:
            ref = rig.orc.logits(h[fp + r], fp + r, 0)
            worst = max(worst, float(np.abs(lg[i, r].astype(np.float64) - ref).max()))
        for r, j in drafts:
            ref = rig.orc.logits(h[fp + r], fp + r + j, j)
            worst = max(worst, float(np.abs(lg[i, SLOT_DRAFT0 + r * K + j - 1].astype(np.float64) - ref).max()))
    return worst


def cdf_margin(prob, u):
    """Distance of u from the nearest step of the normalised ascending-index CDF."""
    c = np.cumsum(prob) / prob.sum()
    return float(np.min(np.abs(c - u)))


def residual_probs(pi, pp, qi, qp):
    q = dict(zip((int(x) for x in qi), (float(x) for x in qp)))
    r = np.array([max(0.0, float(p) - q.get(int(i), 0.0)) for i, p in zip(pi, pp)])
    return r if r.sum() > 0 else np.asarray(pp, dtype=np.float64)


class _Excused(Exception):
    pass


def replay(rig, lg, rd, u, codes):
    """Re-take every decision of the frame from the kernel's own logits with the
    oracle's primitives.  Returns 1 when the frame diverged at a decision whose
    threshold lies within 1e-6 of its uniform (summation-order rounding), else 0."""
    K, n, topk, T = rig.K, rig.s.n_codes, rig.topk, rig.T

    def check(gpu, mine, margin, what):
        if gpu == mine:
            return
        assert margin < CDF_EXCUSE, f"{what}: kernel {gpu}, oracle primitives {mine}, margin {margin:.3g}"
        raise _Excused

    mine = {}
    try:
        for i, row in enumerate(rd):
            m, kp, fp, R_, m_new, acc, tok = (int(x) for x in row[:7])
            if i == 0:
                pi, pp = O.topk_softmax(lg[0, 1], topk, T)
                us = float(u[0, 2])
                check(tok, O.sample(pi, pp, us), cdf_margin(pp, us), "prefix sample")
                assert m_new == 1
                mine[1] = tok
                continue
            arow = m - int(rd[i - 1][2])
            n_acc, my_new = 0, None
            for j in range(1, kp + 1):
                ud, ua, us = (float(x) for x in u[m + j - 1])
                qi, qp = O.topk_softmax(lg[i - 1, SLOT_DRAFT0 + arow * K + j - 1], topk, T)
                d = int(row[8 + j - 1])
                if rig.greedy:
                    check(d, int(qi[int(np.argmax(qp))]), 0.0, f"greedy draft {m + j}")
                    qi, qp = np.array([d], dtype=np.int32), np.array([1.0])
                else:
                    check(d, O.sample(qi, qp, ud), cdf_margin(qp, ud), f"draft {m + j}")
                pi, pp = O.topk_softmax(lg[i, j - 1], topk, T)
                ok, t = O.accept_or_resample(pi, pp, qi, qp, d, ua, us)
                pd = dict(zip(pi.tolist(), pp.tolist())).get(d, 0.0)
                qd = dict(zip(qi.tolist(), qp.tolist())).get(d, 0.0)
                gpu_ok = j <= acc
                check(gpu_ok, ok, abs(ua - pd / qd) if qd > 0 else 1.0, f"accept {m + j}")
                if not ok:
                    check(tok, t, cdf_margin(residual_probs(pi, pp, qi, qp), us), f"residual {m + j}")
                    my_new = m + j
                    break
                mine[m + j] = d
                n_acc += 1
            if my_new is None:
                if m + kp < n:
                    pi, pp = O.topk_softmax(lg[i, kp], topk, T)
                    us = float(u[m + kp, 2])
                    check(tok, O.sample(pi, pp, us), cdf_margin(pp, us), f"bonus {m + kp + 1}")
                    my_new = m + kp + 1
                else:
                    my_new = n
            assert (m_new, acc) == (my_new, n_acc), (i, row[:8].tolist(), my_new, n_acc)
            if my_new > m + n_acc:
                mine[my_new] = tok
    except _Excused:
        return 1
    assert sorted(mine) == list(range(1, n + 1))
    assert [mine[s] for s in range(1, n + 1)] == [int(c) for c in codes]
    return 0


def first_divergence(orounds, rd):
    """Index of the first round whose decisions differ between the oracle's trace
    and the kernel's round records (None when every round agrees)."""
    for i in range(max(len(orounds), len(rd))):
        if i >= len(orounds) or i >= len(rd):
            return i
        o, g = orounds[i], [int(x) for x in rd[i]]
        kp = o["kp"]
        if (o["m"], kp) != (g[0], g[1]) or list(o["drafts"][:kp]) != g[8:8 + kp]:
            return i
        if (o["m_new"], o["accepted"], o["token"]) != (g[4], g[5], g[6]):
            return i
    return None


def argmax_gap(logits):
    """Gap between the two largest logits of a row (where a greedy draft could flip)."""
    a = np.sort(np.asarray(logits, dtype=np.float64))[::-1]
    return float(a[0] - a[1]) if a.size > 1 else np.inf


def near_enough(rig, ornd, err, draft_rows=None):
    """Whether an oracle round's decision margin, top-k gap or (greedy drafts) argmax gap
    is within what a logit error of err can flip."""
    e = max(err, 1e-7)
    if ornd["margin"] < 5.0 * e / rig.T or ornd["topk_gap"] < 2 * e:
        return True
    if rig.greedy and draft_rows is not None:
        return any(argmax_gap(r) < 2 * e for r in draft_rows[:ornd["kp"]])
    return False


def compare_end_to_end(rig, f, c0, u, codes, stats, logit_err, rd):
    """True when the oracle from scratch gives the same frame; False when it differs
    and the first round where the two part is within reach of the measured logit
    error (the GPU parity rule's end-to-end clause); fails otherwise."""
    oc, ost, otr = rig.orc.spec_frame(f, int(c0), u, trace=True, logits=bool(rig.greedy))
    if np.array_equal(oc, codes):
        for k in ("target_calls", "rounds", "drafted", "accepted", "accept_mask"):
            assert stats[k] == ost[k], (k, stats[k], ost[k])
        return True
    i = first_divergence(otr["rounds"], rd)
    assert i is not None, "codes differ but every round agrees"
    dl = otr["draft_logits"][i] if rig.greedy and i < len(otr["rounds"]) else None
    assert i < len(otr["rounds"]) and near_enough(rig, otr["rounds"][i], logit_err, dl), \
        f"first differing round {i} is not near a threshold: gpu {codes.tolist()} oracle {oc.tolist()}"
    return False


def check_traced_frames(rig, frames, f, c0, u, get, tol, excuse_frac=0.1):
    """get(i) -> (codes, stats dict, lg, rd) of frame i; every check above per frame."""
    excused = 0
    worst = 0.0
    for i in frames:
        codes, st, lg, rd = get(i)
        assert st["status"] == 0
        err = logit_error(rig, f[i], c0[i], codes, lg, rd)
        worst = max(worst, err)
        assert err <= tol, f"frame {i}: logit max-abs {err:.3g} > {tol}"
        ex = replay(rig, lg, rd, u[i], codes)
        if not compare_end_to_end(rig, f[i], c0[i], u[i], codes, st, err, rd) or ex:
            excused += 1
    assert excused <= max(1, int(excuse_frac * len(frames))), excused
    return worst, excused


def committing_round(orounds, pos):
    """Index of the oracle round that committed code position pos."""
    for i, r in enumerate(orounds):
        if r["m"] < pos <= r["m_new"]:
            return i
    return len(orounds) - 1


def untraced_divergence_near(rig, f, c0, u, codes, err):
    """For a frame with no kernel trace: the oracle rounds up to the one that commits the
    first differing code hold every decision that could have parted the two runs; at
    least one of them must be within reach of err."""
    oc, _, otr = rig.orc.spec_frame(f, int(c0), u, trace=True, logits=bool(rig.greedy))
    diff = [s for s in range(len(oc)) if int(oc[s]) != int(codes[s])]
    if not diff:
        return True
    last = committing_round(otr["rounds"], diff[0] + 1)
    for i in range(last + 1):
        dl = otr["draft_logits"][i] if rig.greedy else None
        if near_enough(rig, otr["rounds"][i], err, dl):
            return True
    return False


# ------------------------------------------------------------ sparse-tree lanes
# A tree rig adds tree (parents, ranks of rows 1..N), otree (oracle.make_tree of it)
# and slot0 (the first draft slot: max(16, N + 1)). Tree round records (128 ints):
# [0..7] m, K', first, rows, m_new, accepted, token, pass; [8] candidate rows;
# [16..) accepted rows; [32..) candidate tokens (row 0 = c_m).

def tree_depths(tree):
    parents, _ = tree
    d = [0]
    for p in parents:
        d.append(d[p] + 1)
    return d


def tree_logit_error(rig, f, c0, codes, lg, rd):
    """Max-abs difference of every traced verify and draft row of a tree frame from the
    oracle's fp64 logits over the same packed rows."""
    K, n = rig.K, rig.s.n_codes
    depth = tree_depths(rig.tree)
    full = [int(c0)] + [int(c) for c in codes]
    worst = 0.0
    for i, row in enumerate(rd):
        m, fp, R = int(row[0]), int(row[2]), int(row[3])
        if i == 0:
            h = rig.orc.forward(f, [int(c0)])
            rows = [(1, h[1], 1)]  # (row, hidden, position)
        else:
            toks = [int(x) for x in row[32:32 + R]]
            hr = rig.orc.tree_hidden(rig.otree, f, full[:m + 1], toks[1:])
            rows = [(r, hr[r], fp + depth[r]) for r in range(R)]
        for r, h, pos in rows:
            ref = rig.orc.logits(h, pos, 0)
            worst = max(worst, float(np.abs(lg[i, r].astype(np.float64) - ref).max()))
            if pos <= n - 1:
                for j in range(1, min(K, n - pos) + 1):
                    ref = rig.orc.logits(h, pos + j, j)
                    got = lg[i, rig.slot0 + r * K + j - 1].astype(np.float64)
                    worst = max(worst, float(np.abs(got - ref).max()))
    return worst


def tree_replay(rig, lg, rd, u, codes):
    """Re-take every decision of a tree frame from the kernel's own logits: the ranked
    candidates of every depth, the sibling walks and the residual draws. Returns 1 when a
    decision diverged within 1e-6 of its uniform, else 0."""
    K, n, topk, T = rig.K, rig.s.n_codes, rig.topk, rig.T
    parents, ranks = rig.tree
    depth = tree_depths(rig.tree)
    mine = {}
    arow = 1
    for i, row in enumerate(rd):
        m, kp, fp, R, m_new, acc, tok = (int(x) for x in row[:7])
        if i == 0:
            pi, pp = O.topk_softmax(lg[0, 1], topk, T)
            us = float(u[0, 2])
            if tok != O.sample(pi, pp, us):
                assert cdf_margin(pp, us) < CDF_EXCUSE
                return 1
            mine[1] = tok
            arow = 1
            continue
        ncand = int(row[8])
        cand = [int(x) for x in row[32:32 + ncand]]
        # candidates: the anchor row's draft logits of the previous pass, ranked
        for r in range(1, ncand):
            d = depth[r]
            order = np.lexsort((np.arange(rig.s.vocab), -lg[i - 1, rig.slot0 + arow * K + d - 1].astype(np.float64)))
            assert cand[r] == int(order[ranks[r - 1]]), (i, r, cand[r], int(order[ranks[r - 1]]))
        assert cand[0] == (mine[m] if m in mine else None), (i, cand[0])
        cur, pos, path = 0, m + 1, []
        while True:
            pi, pp = O.topk_softmax(lg[i, cur], topk, T)
            kids = sorted((c for c in range(cur + 1, ncand) if parents[c - 1] == cur), key=lambda c: ranks[c - 1])
            pmap = dict(zip(pi.tolist(), pp.tolist()))
            ua, us = float(u[pos - 1, 1]), float(u[pos - 1, 2])
            cum, taken = 0.0, None
            for c in kids:
                cum += pmap.get(cand[c], 0.0)
                if taken is None and ua < cum:
                    taken = c
            gpu_taken = int(row[16 + len(path)]) if len(path) < acc else None
            if taken != gpu_taken:
                cums = np.cumsum([pmap.get(cand[c], 0.0) for c in kids]) if kids else np.array([])
                assert kids and np.min(np.abs(cums - ua)) < CDF_EXCUSE, (i, pos, taken, gpu_taken)
                return 1
            if taken is not None:
                mine[pos] = cand[taken]
                path.append(taken)
                cur = taken
                pos += 1
                if pos > n:
                    break
                continue
            kid_toks = {cand[c] for c in kids}
            res = np.array([0.0 if int(x) in kid_toks else float(p) for x, p in zip(pi, pp)])
            if not res.sum() > 0:
                res = np.asarray(pp, dtype=np.float64)
            t = O.sample(pi, res, us)
            if t != tok:
                assert cdf_margin(res, us) < CDF_EXCUSE, (i, pos, t, tok)
                return 1
            mine[pos] = t
            break
        assert (len(path), min(pos, n)) == (acc, m_new), (i, path, pos, acc, m_new)
        arow = cur
    assert sorted(mine) == list(range(1, n + 1))
    assert [mine[s] for s in range(1, n + 1)] == [int(c) for c in codes]
    return 0


def tree_first_divergence(orounds, rd):
    for i in range(max(len(orounds), len(rd))):
        if i >= len(orounds) or i >= len(rd):
            return i
        o, g = orounds[i], [int(x) for x in rd[i]]
        if (o["m"], o["m_new"], o["accepted"], o["token"]) != (g[0], g[4], g[5], g[6]):
            return i
        if i > 0:
            nc = o["n_cand"]
            if nc != g[8] or o["tokens"][:nc] != g[32:32 + nc] or o["path"] != g[16:16 + o["accepted"]]:
                return i
    return None


def tree_compare_end_to_end(rig, f, c0, u, codes, stats, logit_err, rd):
    oc, ost, otr = rig.orc.tree_frame(rig.otree, f, int(c0), u, trace=True)
    if np.array_equal(oc, codes):
        for k in ("target_calls", "rounds", "drafted", "accepted", "accept_mask"):
            assert stats[k] == ost[k], (k, stats[k], ost[k])
        return True
    i = tree_first_divergence(otr["rounds"], rd)
    assert i is not None and i < len(otr["rounds"]) and near_enough(rig, otr["rounds"][i], logit_err), \
        f"first differing round {i} is not near a threshold: gpu {codes.tolist()} oracle {oc.tolist()}"
    return False


def check_tree_frames(rig, frames, f, c0, u, get, tol, excuse_frac=0.1):
    excused, worst = 0, 0.0
    for i in frames:
        codes, st, lg, rd = get(i)
        assert st["status"] == 0
        err = tree_logit_error(rig, f[i], c0[i], codes, lg, rd)
        worst = max(worst, err)
        assert err <= tol, f"frame {i}: logit max-abs {err:.3g} > {tol}"
        ex = tree_replay(rig, lg, rd, u[i], codes)
        if not tree_compare_end_to_end(rig, f[i], c0[i], u[i], codes, st, err, rd) or ex:
            excused += 1
    assert excused <= max(1, int(excuse_frac * len(frames))), excused
    return worst, excused
