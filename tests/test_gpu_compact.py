"""GPU parity of the memory side of long-history compression (Eq.
optional_context_compression): a stream several times longer than its index
arena runs through budget-driven absorption (ss_index_budget_split,
ss_clusters_absorb) and compaction (ss_index_compact).  Every compaction
leaves retrieval, pooled ranking and cluster retrieval bit-identical, and the
results are staged against the oracle, which keeps the whole stream."""
import sys

import numpy as np
import pytest

import workloads as W
from oracle import oracle as O

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_02780_amd  # noqa: F401  (fails loudly without the built library)


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


def scene_keys(rng, L, Hk, d, F, T, scene_len):
    """Keys with piecewise-constant scene centroids, so that clusters form with
    clear joining margins."""
    n_sc = -(-F // scene_len)
    scene = rng.standard_normal((n_sc, L, Hk, d)).astype(np.float32)
    keys = []
    for l in range(L):
        base = scene[np.arange(F * T) // (scene_len * T), l].transpose(1, 0, 2)
        keys.append(W.bf16_bits(base + rng.standard_normal((Hk, F * T, d)).astype(np.float32) * 0.5))
    return keys


def absolute_hists(out, first_stored, F):
    """The debug histograms are indexed by frame id - first stored frame; the
    staged checker reads them by frame id."""
    for k in ("vote_hist", "mass_hist"):
        h = np.zeros((out[k].shape[0], F), dtype=out[k].dtype)
        n = min(out[k].shape[1], F - first_stored)
        h[:, first_stored:first_stored + n] = out[k][:, :n]
        out[k] = h
    return out


def same_outputs(a, b):
    for k in ("frame_ids", "votes", "mass", "n_out", "topk_pos", "topk_score", "pool", "pool_n", "list_stats"):
        assert np.array_equal(np.asarray(a[k]).view(np.uint8), np.asarray(b[k]).view(np.uint8)), k


def test_budgeted_stream_through_a_small_arena():
    import paper_2609_02780_amd as P
    from parity import staged_check
    rng = np.random.default_rng(91)
    L, Hq, Hk, d, T, nr, F = 2, 8, 2, 64, 16, 4, 150
    keys = scene_keys(rng, L, Hk, d, F, T, 6)
    q = [W.bf16_bits(rng.standard_normal((Hq, 3, d)).astype(np.float32)) for _ in range(L)]
    qd = [dev(x) for x in q]
    cap = 48                                              # frames the arena can hold
    g = P.ShallowIndex(L, Hq, Hk, d, cap, cap * T, nr)
    cl = P.LongClusters(g, T, 256, 0.8)
    o = O.Index(L, Hq, Hk, d, nr)
    ocl = O.LongClusters(0.8, 256)
    budget = 24 * O.frame_bytes(T, L, Hk, d)              # about 24 detailed frames
    r = P.Retriever([g], 24, 4)
    pr = P.PooledRanker([g], 5)
    compactions = 0
    for f0 in range(0, F, 12):
        f1 = min(F, f0 + 12)
        blk = [np.ascontiguousarray(k[:, f0 * T:f1 * T, :]) for k in keys]
        g.append([dev(b) for b in blk], f1 - f0, T)
        o.append(blk, f1 - f0, T)
        first_stored, first_detail = g.window()
        hi = g.budget_split(budget)
        want = O.budget_split([T] * f1, first_detail, nr, L, Hk, d, budget)
        assert hi == want, (f1, hi, want)
        if hi > first_detail:
            cl.absorb(hi, hi - first_detail)
            ocl.absorb(o, hi)
            before = r.debug([qd])
            pb = [t.cpu().numpy().copy() for t in pr([qd])]
            cb = [t.cpu().numpy().copy() for t in cl.retrieve(qd, 5)]
            g.compact()
            compactions += 1
            assert g.window() == (hi, hi)
            after = r.debug([qd])
            same_outputs(before, after)
            pa = [t.cpu().numpy() for t in pr([qd])]
            ca = [t.cpu().numpy() for t in cl.retrieve(qd, 5)]
            for x, y in zip(pb + cb, pa + ca):
                assert np.array_equal(x.view(np.uint8), y.view(np.uint8))
        n_frames, n_rows = g.info()
        assert n_frames == f1 and n_rows == (f1 - g.window()[0]) * T and n_rows <= cap * T
    log("frames", F, "compactions", compactions, "window", g.window(), "clusters", len(ocl.sizes))
    assert compactions >= 8 and F > 2 * cap
    # the final state against the oracle, which keeps the whole stream
    first_stored, first_detail = g.window()
    assert first_detail == o.first_detail
    ex = cl.export()
    assert ex["n_clusters"] == len(ocl.sizes) and ex["sizes"].tolist() == ocl.sizes
    assert ex["span"].tolist() == [[a, b] for a, b in zip(ocl.first, ocl.last)]
    np.testing.assert_allclose(ex["centroids"], np.array(ocl.centroids), atol=2e-6)
    reps = np.array(ocl.rep)
    np.testing.assert_allclose(ex["reps"], reps, atol=2e-5 * max(1.0, np.abs(reps).max()))
    out = absolute_hists(r.debug([qd]), first_stored, F)
    rep = staged_check(o, q, out, 0, 24, 4)
    log("after the stream", rep)
    ids, sc, n = (t.cpu().numpy() for t in pr([qd]))
    w_ids, w_sc, w_n = O.pooled_retrieve(o, q, 5)
    s_all = O.pooled_scores(o, q)
    assert int(n[0]) == w_n
    if not np.any(np.abs(np.diff(np.sort(s_all)[::-1][:6])) < 1e-6):
        assert ids[0, :w_n].tolist() == w_ids[:w_n].tolist()
    np.testing.assert_allclose(sc[0, :w_n], s_all[ids[0, :w_n] - o.first_candidate_frame()], atol=2e-6)
    cids, csc, cfirst, clast, cn = cl.retrieve(qd, 5)
    ev_ids, ev_kinds, ev_n = P.assemble_evidence([g], r.frame_ids, nr, 1, 0, True, clusters=[cl],
                                                 cluster_ids=cids[None, :].contiguous())
    torch.cuda.synchronize()
    m = int(ev_n.cpu()[0])
    wi, wk = O.evidence_items(F, out["frame_ids"][0], nr, 1, 0, True, o.first_detail, ocl.first,
                              cids.cpu().numpy())
    assert ev_ids.cpu().numpy()[0, :m].tolist() == wi.tolist()
    assert ev_kinds.cpu().numpy()[0, :m].tolist() == wk.tolist()


def test_compaction_of_a_compressed_stream_and_full_capacity():
    """Frames stored as k-means centroids compact the same way (member counts
    move with their rows); compacting everything up to the recent window, and
    a capacity error when the arena is full without compaction."""
    import paper_2609_02780_amd as P
    rng = np.random.default_rng(92)
    L, Hq, Hk, d, T, nr = 2, 4, 2, 64, 40, 3
    keys = scene_keys(rng, L, Hk, d, 60, T, 5)
    q = [W.bf16_bits(rng.standard_normal((Hq, 2, d)).astype(np.float32)) for _ in range(L)]
    qd = [dev(x) for x in q]
    g = P.ShallowIndex(L, Hq, Hk, d, 30, 30 * 8, nr)
    cl = P.LongClusters(g, 8, 64, 0.8)
    blk = [np.ascontiguousarray(k[:, :30 * T, :]) for k in keys]
    g.append([dev(b) for b in blk], 30, T, (8, 3))
    with pytest.raises(P.SSError) as e:
        g.append([dev(np.ascontiguousarray(k[:, 30 * T:31 * T, :])) for k in keys], 1, T, (8, 3))
    assert e.value.status == 3
    full = g.export()
    cl.absorb(27, 27)                      # everything but the recent window
    r = P.Retriever([g], 6, 2)
    before = r.debug([qd])
    g.compact()
    after = r.debug([qd])
    same_outputs(before, after)
    ex = g.export()
    assert ex["frame_offsets"] == [8 * i for i in range(4)]
    np.testing.assert_array_equal(ex["rows"], full["rows"][:, :, 27 * 8:, :])
    np.testing.assert_array_equal(ex["counts"], full["counts"][:, :, 27 * 8:])
    np.testing.assert_array_equal(ex["desc"], full["desc"][27:])
    blk2 = [np.ascontiguousarray(k[:, 30 * T:57 * T, :]) for k in keys]
    g.append([dev(b) for b in blk2], 27, T, (8, 3))     # the freed space is reused
    assert g.info() == (57, 30 * 8)
    ex2 = g.export()
    np.testing.assert_array_equal(ex2["rows"][:, :, :3 * 8], ex["rows"])
