"""Staged parity checker: the HIP path against the CPU oracle.

Each stage of the GPU result is checked given the GPU's previous stage, because
the top-k boundary of the synthetic workloads is dense with near-ties:

1. per-key scores within ``1e-3 * D`` where ``D = (1/sqrt d) sum_e |qbar_e||K_e|``
   is the magnitude of the score's terms (fp32 accumulation of bf16 inputs);
2. each GPU top-k list is tolerance-valid against the oracle's scores (every
   selected row scores at least the oracle's k-th score minus the tolerance,
   every other row at most that score plus it); exact swaps are counted;
3. votes equal exactly the oracle's votes recomputed from the GPU lists; mass
   within 1e-3 of the magnitude of the summed scores;
4. the pool is a valid vote ranking of the GPU's votes and mass (mass ties up to
   the tolerance are exempt); the selection is a valid greedy max-min run over
   the oracle's descriptors (argmax near-ties below 1e-5 exempt);
5. end to end, frame ids equal the pure oracle's when no stage needed an exemption.
"""
from __future__ import annotations

import math

import numpy as np
import torch

from oracle import oracle as O

SCORE_RTOL = 1e-3
MAXMIN_EPS = 1e-5


def dev_bf16(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


def score_scale(oidx: O.Index, queries, head_mode: int = 0):
    """Per list, per candidate row: ``(1/sqrt d) sum_e |qbar_e| |K_e|`` (head_mode 0),
    or the head mean of those magnitudes (head_mode 1): the scale of the scaled
    logits' terms."""
    lo, hi = oidx.first_candidate_row(), oidx.candidate_rows()
    N = hi - lo
    qm = O.query_means(queries)
    out = []
    for l in range(oidx.L):
        K = oidx.rows(l)
        per_head = np.empty((oidx.Hq, N))
        for g in range(oidx.Hk):
            Ka = np.abs(O.decode_bf16(K[g, lo:hi, :]))
            Qa = np.abs(qm[l][g * oidx.G:(g + 1) * oidx.G])
            per_head[g * oidx.G:(g + 1) * oidx.G] = (Ka @ Qa.T).T / math.sqrt(oidx.d)
        if head_mode == 0:
            out.extend(per_head)
        else:
            out.append(per_head.mean(axis=0))
    return out


def value_scale(oidx: O.Index, queries, head_mode: int = 0, score_mode: int = 0):
    """The scale of each list value's error under the logit tolerance: the logit
    scale of ``score_scale`` for scaled logits; for attention probabilities a
    logit error of 1e-3 D moves ``p = exp(s - lse)`` by at most
    ``p (1e-3 D_row + 1e-3 max_rows D)`` (the row's own logit and the
    log-sum-exp, which moves by at most the largest row error), so the scale of
    a per-head probability is ``p (D_row + max D)``, averaged over heads in
    head mode 1."""
    if score_mode == 0:
        return score_scale(oidx, queries, head_mode)
    P = O.score_lists(oidx, queries, 0, 1)
    D = score_scale(oidx, queries, 0)
    # plus 0.01 p: a floor of 1e-5 relative for the fp32 exp and log of the
    # probability itself (all-zero queries make every D zero)
    per_head = [p * (d + d.max() + 0.01) if d.size else d for p, d in zip(P, D)]
    if head_mode == 0:
        return per_head
    return [np.mean(per_head[l * oidx.Hq:(l + 1) * oidx.Hq], axis=0) for l in range(oidx.L)]


def check_topk_list(so, dscale, pos, gscore, kk, report, name=""):
    """Stage 2 for one list; returns the oracle-exact top-k positions."""
    assert pos.shape == (kk,), name
    assert np.all(pos >= 0) and np.all(pos < so.size), name
    assert np.unique(pos).size == kk, f"{name}: duplicate rows"
    tol = SCORE_RTOL * dscale
    # GPU scores of the selected rows
    err = np.abs(gscore - so[pos])
    assert np.all(err <= tol[pos]), f"{name}: score error {err.max()} above tolerance"
    report["max_rel_score_err"] = max(report.get("max_rel_score_err", 0.0),
                                      float(np.max(err / np.maximum(dscale[pos], 1e-300))))
    # rank order of the GPU list: scores non-increasing, equal scores by row
    assert np.all(np.diff(gscore) <= 0), f"{name}: GPU list not sorted"
    tied = np.diff(gscore) == 0
    assert np.all(np.diff(pos)[tied] > 0), f"{name}: equal scores not in row order"
    if kk == 0:
        return np.zeros(0, dtype=np.int64)
    exact = O.topk(so, kk)
    kth = exact[-1]
    sel = np.zeros(so.size, dtype=bool)
    sel[pos] = True
    lo = so[kth] - tol[kth]
    hi = so[kth] + tol[kth]
    assert np.all(so[pos] + tol[pos] >= lo), f"{name}: a selected row is clearly below the k-th score"
    assert np.all(so[~sel] - tol[~sel] <= hi), f"{name}: an unselected row is clearly above the k-th score"
    sw = int(np.setdiff1d(exact, pos).size)
    report["swaps"] = report.get("swaps", 0) + sw
    if sw:
        report["lists_with_swaps"] = report.get("lists_with_swaps", 0) + 1
    return exact


def check_pool(pool, votes, mass, mass_tol, P, report):
    """Stage 4a: ``pool`` (frame ids) is a valid ranking of frames with >= 1 vote by
    (votes desc, mass desc, id asc), mass ties within ``mass_tol`` exempt."""
    voted = np.nonzero(votes >= 1)[0]
    assert pool.size == min(P, voted.size)
    assert np.unique(pool).size == pool.size
    assert np.all(votes[pool] >= 1)
    for a, b in zip(pool[:-1], pool[1:]):
        assert votes[a] >= votes[b], "pool not ordered by votes"
        if votes[a] == votes[b]:
            t = mass_tol[a] + mass_tol[b]
            assert mass[a] >= mass[b] - t, "pool not ordered by mass"
            if abs(mass[a] - mass[b]) <= t and not (mass[a] > mass[b] or (mass[a] == mass[b] and a < b)):
                report["pool_exempt"] = report.get("pool_exempt", 0) + 1
    rest = np.setdiff1d(voted, pool)
    if pool.size and rest.size:
        last = pool[-1]
        for f in rest:
            better = votes[f] > votes[last] or (votes[f] == votes[last] and
                                                mass[f] > mass[last] + mass_tol[f] + mass_tol[last])
            assert not better, f"frame {f} should have entered the pool"
    ref = O.vote_pool(votes, mass, P)
    if not np.array_equal(ref, pool):
        report["pool_differs"] = report.get("pool_differs", 0) + 1


def check_maxmin(pool, desc, K, selected, report):
    """Stage 4b: ``selected`` is a greedy max-min run over ``pool`` (oracle descriptors)."""
    want = min(K, pool.size)
    assert selected.size == want
    if want == 0:
        return
    assert selected[0] == pool[0], "max-min must start from the top of the vote ranking"
    chosen = [int(selected[0])]
    rank = {int(f): i for i, f in enumerate(pool)}
    for f in selected[1:]:
        f = int(f)
        assert f in rank and f not in chosen
        cand = [u for u in pool if int(u) not in chosen]
        val = {int(u): min(1.0 - float(desc[u] @ desc[c]) for c in chosen) for u in cand}
        best = max(val.values())
        assert val[f] >= best - MAXMIN_EPS, "selection is not the max-min choice"
        winners = [u for u in cand if val[int(u)] == best]
        if val[f] != best or rank[f] != min(rank[int(u)] for u in winners):
            report["maxmin_exempt"] = report.get("maxmin_exempt", 0) + 1
        chosen.append(f)


def staged_check(oidx: O.Index, queries, gpu: dict, s: int, top_k: int, n_select: int,
                 pool_mult: int = 4, head_mode: int = 0, score_mode: int = 0):
    """Run stages 2-5 for stream ``s`` of a ``Retriever.debug`` result; returns a
    report with the swap and exemption counts."""
    report = {}
    S_or = O.score_lists(oidx, queries, head_mode, score_mode)
    Dsc = value_scale(oidx, queries, head_mode, score_mode)
    N = oidx.candidate_rows() - oidx.first_candidate_row()     # positions are window-relative
    kk = min(top_k, N)
    NL = len(S_or)
    gpu_lists, exact_lists = [], []
    for j in range(NL):
        pos = gpu["topk_pos"][s, j]
        assert np.all(pos[kk:] == -1)
        p = pos[:kk].astype(np.int64)
        exact = check_topk_list(S_or[j], Dsc[j], p, gpu["topk_score"][s, j, :kk].astype(np.float64), kk,
                                report, name=f"list {j}")
        gpu_lists.append(p)
        exact_lists.append(exact)
    F = oidx.n_frames
    v_re, m_re = O.votes_and_mass(oidx, gpu_lists, S_or)
    gv = gpu["vote_hist"][s, :F].astype(np.int64)
    gm = gpu["mass_hist"][s, :F].astype(np.float64)
    assert np.array_equal(gv, v_re), "votes differ from the oracle's votes of the GPU lists"
    assert gv.sum() == NL * kk
    # mass tolerance: 1e-3 of the summed magnitudes of the frame's selected scores
    f_of = oidx.frame_of_row()[oidx.first_candidate_row():oidx.candidate_rows()]
    mag = np.zeros(F)
    for p, dsc in zip(gpu_lists, Dsc):
        np.add.at(mag, f_of[p], dsc[p])
    mass_tol = SCORE_RTOL * mag + 1e-12
    assert np.all(np.abs(gm - m_re) <= mass_tol), "mass outside tolerance"
    P = pool_mult * n_select
    pn = int(gpu["pool_n"][s])
    pool = gpu["pool"][s, :pn].astype(np.int64)
    assert np.all(gpu["pool"][s, pn:] == -1)
    check_pool(pool, gv, gm, mass_tol, P, report)
    desc = np.array(oidx.desc)
    n_out = int(gpu["n_out"][s])
    sel = gpu["frame_ids"][s, :n_out].astype(np.int64)
    assert np.all(gpu["frame_ids"][s, n_out:] == -1)
    check_maxmin(pool, desc, n_select, sel, report)
    assert np.array_equal(gpu["votes"][s, :n_out], gv[sel])
    np.testing.assert_allclose(gpu["mass"][s, :n_out], gm[sel], rtol=1e-6, atol=1e-6)
    # end to end against the pure oracle
    ids, v, m, n = O.retrieve(oidx, queries, top_k, n_select, pool_mult, head_mode, score_mode=score_mode)
    report["lists"] = NL
    report["end_to_end_equal"] = bool(np.array_equal(ids[:n], sel) and n == n_out)
    clean = not any(report.get(k, 0) for k in ("swaps", "pool_exempt", "pool_differs", "maxmin_exempt"))
    if clean:
        assert report["end_to_end_equal"], "no exemption was needed, yet the frame ids differ"
    return report
