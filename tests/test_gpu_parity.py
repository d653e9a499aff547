"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Inputs come from the seeded generators in ``workloads``; expected values only
from ``oracle``.  Tolerances: per-key scores within 1e-3 of the magnitude of
their terms (fp32 accumulation of bf16 products); integer results (votes, row
positions, frame ids) exact, with the boundary near-tie exemptions of
``parity.staged_check``.
"""
import math
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


def _P():
    import paper_2609_02780_amd as P
    return P


from parity import dev_bf16, score_scale, staged_check  # noqa: E402


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def make_pair(cfg, spec, keys, compress=None, n_recent=0, max_frames=None, max_rows=None):
    P = _P()
    T = cfg.tokens_per_frame
    F = spec.n_frames
    rpf = T if compress is None else min(compress[0], T)
    gidx = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim,
                          max_frames or F, max_rows or F * rpf, n_recent)
    gidx.append([dev_bf16(k) for k in keys], F, T, compress)
    oidx = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, n_recent)
    if compress is None:
        oidx.append(keys, F, T)
    return gidx, oidx


def debug_run(gidxs, queries, top_k, n_select, pool_mult=4, head_mode=0):
    P = _P()
    r = P.Retriever(gidxs, top_k, n_select, pool_mult, head_mode)
    qd = [[dev_bf16(q) for q in qs] for qs in queries]
    return r.debug(qd)


def c1():
    cfg = W.CONFIGS["C1"]
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec)
    return cfg, spec, q, keys


# ---------------------------------------------------------------------------


def test_scores_c1():
    cfg, spec, q, keys = c1()
    log("scores C1")
    gidx, oidx = make_pair(cfg, spec, keys)
    S = O.score_lists(oidx, q)
    D = score_scale(oidx, q)
    qd = [dev_bf16(x) for x in q]
    worst = 0.0
    for l in range(cfg.n_layers):
        for h in range(cfg.n_q_heads):
            g = gidx.debug_scores(qd, l, h).cpu().numpy().astype(np.float64)
            j = l * cfg.n_q_heads + h
            err = np.abs(g - S[j])
            assert np.all(err <= 1e-3 * D[j])
            worst = max(worst, float(np.max(err / D[j])))
    log("max |err|/D", worst)
    assert worst < 1e-5       # the hi/lo query split keeps fp32-level accuracy


def test_scores_ragged_row_range():
    """A row range that starts mid-tile and ends in a ragged tail."""
    cfg, spec, q, keys = c1()
    gidx, oidx = make_pair(cfg, spec, keys)
    S = O.score_lists(oidx, q)
    qd = [dev_bf16(x) for x in q]
    g = gidx.debug_scores(qd, 1, 3, row0=37, n_rows=501).cpu().numpy()
    np.testing.assert_allclose(g, S[1 * 4 + 3][37:538], rtol=0, atol=1e-4)


def test_descriptors_and_rows_c1():
    cfg, spec, q, keys = c1()
    gidx, oidx = make_pair(cfg, spec, keys)
    ex = gidx.export()
    np.testing.assert_allclose(ex["desc"], np.array(oidx.desc), rtol=0, atol=2e-6)
    for l in range(cfg.n_layers):
        np.testing.assert_array_equal(ex["rows"][l], keys[l])
    assert ex["frame_offsets"] == [16 * i for i in range(65)]
    assert np.all(ex["counts"] == 1)


def test_retrieve_c1_staged_and_planted():
    cfg, spec, q, keys = c1()
    log("retrieve C1")
    gidx, oidx = make_pair(cfg, spec, keys)
    out = debug_run([gidx], [q], cfg.top_k, cfg.n_select)
    rep = staged_check(oidx, q, out, 0, cfg.top_k, cfg.n_select)
    log(rep)
    assert rep["end_to_end_equal"]
    planted = set(spec.planted)
    assert out["frame_ids"][0, 0] in planted                          # P2
    assert out["list_stats"][0, :, 1].sum() == 0    # no list needed the fallback
    # P3: with a pool of K frames diversity cannot displace a planted frame
    out1 = debug_run([gidx], [q], cfg.top_k, cfg.n_select, pool_mult=1)
    assert planted <= set(out1["frame_ids"][0].tolist())


def test_small_grid_handed_out_tail_covers_last_tiles():
    """The tiny workload runs the streaming pass on 16 blocks with the handed-out
    tail on (4 segments against a 16-block grid).  The last frame gets twice the
    keys of a planted frame, so the top rows of the last segment's lists sit in
    its last tile, inside the last handed-out chunk: every chunk counter must
    have waves, or those rows are never scored and the lists fall back."""
    cfg, spec, q, keys = c1()
    F, T = spec.n_frames, cfg.tokens_per_frame
    src = spec.planted[-1]
    for l in range(cfg.n_layers):
        x = O.decode_bf16(keys[l])
        x[:, (F - 1) * T:F * T, :] = 2.0 * x[:, src * T:(src + 1) * T, :]   # exact in bf16
        keys[l] = W.bf16_bits(x.astype(np.float32))
    gidx, oidx = make_pair(cfg, spec, keys)
    out = debug_run([gidx], [q], cfg.top_k, cfg.n_select)
    assert out["list_stats"][0, :, 1].sum() == 0    # no list needed the fallback
    rep = staged_check(oidx, q, out, 0, cfg.top_k, cfg.n_select)
    log(rep)
    assert F - 1 in out["frame_ids"][0].tolist()


def test_selected_scores_have_the_recompute_bits():
    """Every path scores a row with the same arithmetic: the scores the retrieval
    selects (query prep fused with the sample pass, then the streaming pass) are
    bit-equal to the standalone prep and recompute kernels' scores of the same
    rows, in both head modes."""
    cfg, spec, q, keys = c1()
    gidx, _ = make_pair(cfg, spec, keys)
    qd = [dev_bf16(x) for x in q]
    for head_mode, n_lists in ((0, cfg.n_layers * cfg.n_q_heads), (1, cfg.n_layers)):
        out = debug_run([gidx], [q], cfg.top_k, cfg.n_select, head_mode=head_mode)
        for j in range(n_lists):
            l, h = (j // cfg.n_q_heads, j % cfg.n_q_heads) if head_mode == 0 else (j, 0)
            full = gidx.debug_scores(qd, l, h, head_mode=head_mode).cpu().numpy()
            pos = out["topk_pos"][0, j]
            got = out["topk_score"][0, j]
            assert np.array_equal(got.view(np.uint32), full[pos].view(np.uint32)), (head_mode, j)


def test_zero_queries_tie_rule():
    """All-zero queries: every score is 0, so each list keeps rows 0..k-1."""
    cfg, spec, q, keys = c1()
    gidx, oidx = make_pair(cfg, spec, keys)
    zq = [np.zeros_like(x) for x in q]
    out = debug_run([gidx], [zq], cfg.top_k, cfg.n_select)
    for j in range(cfg.n_layers * cfg.n_q_heads):
        np.testing.assert_array_equal(out["topk_pos"][0, j], np.arange(32))
    assert out["vote_hist"][0, 0] == 128 and out["vote_hist"][0, 1] == 128
    assert out["vote_hist"][0, 2:64].sum() == 0
    assert out["n_out"][0] == 2 and out["frame_ids"][0, 0] == 0


def test_fallback_too_many_candidates():
    """Zero queries over 8192 rows: every row ties at the cut-off, the candidate
    buffer overflows and the exact fallback must still return rows 0..k-1."""
    cfg = W.Config("fb", 1, 2, 1, 64, 16, 1, 40, 3, n_frames=512)
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec)
    gidx, oidx = make_pair(cfg, spec, keys)
    zq = [np.zeros_like(x) for x in q]
    out = debug_run([gidx], [zq], cfg.top_k, cfg.n_select)
    assert np.all(out["list_stats"][0, :, 1] == 1)
    for j in range(2):
        np.testing.assert_array_equal(out["topk_pos"][0, j], np.arange(40))
    rep = staged_check(oidx, zq, out, 0, cfg.top_k, cfg.n_select)
    assert rep["end_to_end_equal"]


def test_fallback_too_few_candidates():
    """Rows on the sample lattice score highest, so the sample cut-off keeps fewer
    than k rows; the exact fallback must take over and match the oracle."""
    P = _P()
    L, Hq, Hk, d, T, F = 1, 1, 1, 64, 100, 1000
    n = F * T
    k = 512
    m, r, cap, E = P.sample_plan(n, k)        # the library's own plan of this list
    assert m < n
    step = (n << 32) // m                     # the documented sample lattice, 32.32 fixed point
    rows = (np.arange(m, dtype=np.uint64) * np.uint64(step) + np.uint64(step >> 1)) >> np.uint64(32)
    rows = rows.astype(np.int64)
    rng = np.random.default_rng(11)
    x = rng.standard_normal((1, n, d)).astype(np.float32) * 0.01
    x[0, rows, 0] = 5.0 + rng.random(m).astype(np.float32)      # only sampled rows score high
    keys = [W.bf16_bits(x)]
    qv = np.zeros((Hq, 1, d), np.float32)
    qv[0, 0, 0] = 1.0
    q = [W.bf16_bits(qv)]
    cfg = W.Config("few", L, Hq, Hk, d, T, 1, k, 4, n_frames=F)
    spec = W.stream_specs(cfg)[0]
    gidx, oidx = make_pair(cfg, spec, keys)
    out = debug_run([gidx], [q], k, 4)
    assert out["list_stats"][0, 0, 1] == 1, "no fallback: the planted rows are not the library's sample"
    rep = staged_check(oidx, q, out, 0, k, 4)
    log(rep)
    assert rep.get("swaps", 0) == 0


def test_head_mode_paper_reduction_c1():
    """head_mode 1: scores averaged over all query heads, top-k per layer."""
    cfg, spec, q, keys = c1()
    gidx, oidx = make_pair(cfg, spec, keys)
    qd = [dev_bf16(x) for x in q]
    S = O.score_lists(oidx, q, 1)
    D = score_scale(oidx, q, 1)
    for l in range(cfg.n_layers):
        g = gidx.debug_scores(qd, l, 0, head_mode=1).cpu().numpy()
        assert np.all(np.abs(g - S[l]) <= 1e-3 * D[l])
    out = debug_run([gidx], [q], 64, 4, 4, head_mode=1)
    rep = staged_check(oidx, q, out, 0, 64, 4, 4, head_mode=1)
    log(rep)
    assert out["vote_hist"][0].sum() == cfg.n_layers * 64


def test_k_beyond_rows_and_recent_window():
    cfg = W.Config("small", 2, 4, 2, 64, 5, 3, 100, 3, n_frames=9, n_planted=1)
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec)
    gidx, oidx = make_pair(cfg, spec, keys, n_recent=2)
    out = debug_run([gidx], [q], 100, 3)
    n = 7 * 5
    assert np.all(out["topk_pos"][0, :, n:] == -1)
    assert out["vote_hist"][0].sum() == 8 * n
    assert np.all(out["vote_hist"][0, 7:] == 0)
    staged_check(oidx, q, out, 0, 100, 3)


def test_no_candidates():
    cfg = W.Config("none", 1, 2, 1, 64, 4, 2, 8, 3, n_frames=3)
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec)
    gidx, oidx = make_pair(cfg, spec, keys, n_recent=5)
    out = debug_run([gidx], [q], 8, 3)
    assert out["n_out"][0] == 0 and np.all(out["frame_ids"][0] == -1)
    assert out["pool_n"][0] == 0


def test_ragged_batch_one_call():
    """Three streams of different lengths, token counts and recent windows, one
    of them compressed, retrieved in one call; each checked on its own."""
    P = _P()
    base = W.Config("rag", 2, 8, 2, 128, 49, 6, 48, 5, n_frames=0)
    lens, nrec, comp = [37, 120, 81], [0, 3, 0], [None, None, (8, 4)]
    gidxs, oidxs, qs = [], [], []
    for s, (F, nr, cp) in enumerate(zip(lens, nrec, comp)):
        cfg = W.Config("rag", 2, 8, 2, 128, 49, 6 + 3 * s, 48, 5, n_frames=F, n_planted=2)
        spec = W.StreamSpec(s, F, 2, cp, W.planted_frames(F, 2))
        q, keys = W.make_stream(cfg, spec)
        g, o = make_pair(cfg, spec, keys, compress=cp, n_recent=nr)
        if cp is not None:
            ex = g.export()
            o.append_stored([ex["rows"][l] for l in range(cfg.n_layers)], [8] * F,
                            [O.descriptor(O.decode_bf16(keys[-1][:, f * 49:(f + 1) * 49, :])) for f in range(F)])
        gidxs.append(g)
        oidxs.append(o)
        qs.append(q)
    out = debug_run(gidxs, qs, 48, 5)
    for s in range(3):
        rep = staged_check(oidxs[s], qs[s], out, s, 48, 5)
        log(s, rep)


def test_segment_rich_batch_weighted_split_and_handed_out_tail():
    """Sixteen ragged streams of 2 layers x 2 KV heads (64 segments of 60-75
    frames x 32 rows) in one call: the streaming pass takes groups of 16 blocks
    with XCD-weighted ranges and hands the last 15% of its tiles out in chunks
    through the chunk counters, so segments are cut at arbitrary tiles between
    waves.  Every stream checked stage by stage against the oracle."""
    gidxs, oidxs, qs = [], [], []
    for s in range(16):
        F = 60 + s
        cfg = W.Config("segrich", 2, 4, 2, 64, 32, 8, 32, 4, n_frames=F, n_planted=1)
        spec = W.stream_specs(cfg)[0]
        q, keys = W.make_stream(cfg, spec, seed=100 + s)
        g, o = make_pair(cfg, spec, keys)
        gidxs.append(g)
        oidxs.append(o)
        qs.append(q)
    out = debug_run(gidxs, qs, 32, 4)
    assert out["list_stats"][:, :, 1].sum() == 0    # no list needed the fallback
    for s in range(16):
        rep = staged_check(oidxs[s], qs[s], out, s, 32, 4)
        log(s, rep)


def test_pool_cut_many_ties():
    """One selected row per list over 256 lists of an 800-frame stream: almost
    every voted frame has a single vote, so more than 128 frames tie at the
    pool's cut and the pool falls back to the radix cut over the (votes, mass,
    frame) records; checked against the oracle stage by stage."""
    cfg = W.Config("ties", 8, 32, 8, 64, 4, 2, 1, 16, n_frames=800, n_planted=0)
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec)
    g, o = make_pair(cfg, spec, keys)
    out = debug_run([g], [q], cfg.top_k, cfg.n_select)
    v = out["vote_hist"][0, :spec.n_frames]
    P = 4 * cfg.n_select
    vstar = np.sort(v)[::-1][P - 1]
    assert vstar >= 1 and np.count_nonzero(v == vstar) > 128   # the radix cut ran
    rep = staged_check(o, q, out, 0, cfg.top_k, cfg.n_select)
    log(rep)


def test_long_stream_global_paths():
    """A 6,000-frame stream with k = 2048 per list: more than 4,096 frames, so
    the selection adds votes and mass with global atomics; more than 4,096
    voted frames, so the pool keeps its records in global memory and cuts them
    by the 128-bit radix selection; and about 12,000 candidates per list on
    average, above the 8,192 that the selection holds in registers, so lists
    select by radix over their candidates in global memory.  Staged against
    the oracle."""
    cfg = W.Config("long", 2, 8, 2, 64, 4, 3, 2048, 16, n_frames=6000, n_planted=4)
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec)
    g, o = make_pair(cfg, spec, keys)
    out = debug_run([g], [q], cfg.top_k, cfg.n_select)
    stats = out["list_stats"][0]
    voted = int(np.count_nonzero(out["vote_hist"][0, :spec.n_frames]))
    log("long stream: candidates per list", stats[:, 0].min(), stats[:, 0].max(), "fallbacks",
        stats[:, 1].sum(), "voted frames", voted)
    assert stats[:, 0].max() > 8192 and stats[:, 1].sum() == 0
    assert voted > 4096
    rep = staged_check(o, q, out, 0, cfg.top_k, cfg.n_select)
    log("long stream", rep)


def test_sample_of_more_than_8192_rows():
    """A list of 2,000,000 rows with k = 16: the planner samples about 14,300
    rows, so the cut-off holds 16 sample slots per thread (the widest
    instantiation); both head modes staged against the oracle."""
    import paper_2609_02780_amd as P
    cfg = W.Config("bigsample", 1, 2, 1, 64, 500, 2, 16, 4, n_frames=4000, n_planted=2)
    n = cfg.n_frames * cfg.tokens_per_frame
    m = P.sample_plan(n, cfg.top_k)[0]
    log("big sample: rows", n, "sampled", m)
    assert 8192 < m <= 16384
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec)
    g, o = make_pair(cfg, spec, keys)
    for hm in (0, 1):
        out = debug_run([g], [q], cfg.top_k, cfg.n_select, head_mode=hm)
        stats = out["list_stats"][0]
        log("big sample, head mode", hm, "candidates", stats[:, 0].tolist(), "fallbacks", stats[:, 1].tolist())
        assert stats[:, 1].sum() == 0
        rep = staged_check(o, q, out, 0, cfg.top_k, cfg.n_select, head_mode=hm)
        log("big sample, head mode", hm, rep)


def test_group_of_16_query_heads():
    """G = 16 query heads per KV head (the largest group: 16 MFMA columns for
    the hi chain and 16 for the lo chain), d = 64 and d = 128."""
    for d in (64, 128):
        cfg = W.Config(f"g16-{d}", 2, 16, 1, d, 16, 5, 40, 6, n_frames=150, n_planted=2)
        spec = W.stream_specs(cfg)[0]
        q, keys = W.make_stream(cfg, spec)
        g, o = make_pair(cfg, spec, keys)
        worst = _all_row_scores(g, o, q, [(l, h) for l in range(2) for h in range(16)])
        log(f"G=16 d={d}: max |err|/D", worst)
        assert worst < 1e-5
        out = debug_run([g], [q], cfg.top_k, cfg.n_select)
        rep = staged_check(o, q, out, 0, cfg.top_k, cfg.n_select)
        log(f"G=16 d={d}", rep)
        out1 = debug_run([g], [q], cfg.top_k, cfg.n_select, head_mode=1)
        rep1 = staged_check(o, q, out1, 0, cfg.top_k, cfg.n_select, head_mode=1)
        log(f"G=16 d={d} head mode 1", rep1)


def test_more_streams_than_one_launch():
    """40 streams in one call: the host runs them as a group of 32 and a group
    of 8 over one workspace; every stream staged against the oracle."""
    gidxs, oidxs, qs = [], [], []
    for s in range(40):
        F = 20 + (7 * s) % 23
        cfg = W.Config("many", 2, 4, 2, 64, 8, 2 + s % 3, 12, 3, n_frames=F, n_planted=1)
        spec = W.stream_specs(cfg)[0]
        q, keys = W.make_stream(cfg, spec, seed=300 + s)
        g, o = make_pair(cfg, spec, keys)
        gidxs.append(g)
        oidxs.append(o)
        qs.append(q)
    out = debug_run(gidxs, qs, 12, 3)
    for s in range(40):
        staged_check(oidxs[s], qs[s], out, s, 12, 3)
    log("40 streams staged")


def test_largest_pool_and_selection():
    """The largest frame budget the boundary takes (K = 64) with the pool
    multiplier 4: a pool of 256 frames, beyond the 128 whose distances max-min
    keeps in LDS (its block-wide greedy over the Gram matrix in global memory)
    and a 16 x 16 grid of Gram tiles; 10-minute head shape (G = 7, d = 128) on
    300 frames, of which more than 128 get votes.  Staged against the oracle
    (the greedy property of the selection checked on the oracle's
    descriptors)."""
    base = W.CONFIGS["C2"]
    cfg = W.Config("pool256", base.n_layers, base.n_q_heads, base.n_kv_heads, base.head_dim, 196, base.n_q,
                   base.top_k, 64, n_frames=300, n_planted=4)
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec)
    gidx, oidx = make_pair(cfg, spec, keys)
    out = debug_run([gidx], [q], cfg.top_k, 64, 4)
    pn = int(out["pool_n"][0])
    log("voted frames in the pool:", pn)
    assert 128 < pn <= 256          # more than the LDS-resident distances hold
    assert int(out["n_out"][0]) == 64
    rep = staged_check(oidx, q, out, 0, cfg.top_k, 64, 4)
    log("K = 64, pool 256:", rep)
    assert rep["lists"] == cfg.n_layers * cfg.n_q_heads


def test_deterministic_repeat():
    cfg, spec, q, keys = c1()
    gidx, _ = make_pair(cfg, spec, keys)
    a = debug_run([gidx], [q], cfg.top_k, cfg.n_select)
    b = debug_run([gidx], [q], cfg.top_k, cfg.n_select)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k])


def test_append_in_pieces_equals_one_append():
    cfg, spec, q, keys = c1()
    P = _P()
    g1, _ = make_pair(cfg, spec, keys)
    g2 = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, 64, 1024)
    T = cfg.tokens_per_frame
    for f0, f1 in [(0, 10), (10, 11), (11, 64)]:
        first = g2.append([dev_bf16(np.ascontiguousarray(k[:, f0 * T:f1 * T, :])) for k in keys], f1 - f0, T)
        assert first == f0
    e1, e2 = g1.export(), g2.export()
    for k in ("rows", "counts", "desc"):
        np.testing.assert_array_equal(e1[k], e2[k])
    assert e1["frame_offsets"] == e2["frame_offsets"]


def test_capacity_error_leaves_index_unchanged():
    cfg, spec, q, keys = c1()
    P = _P()
    g = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, 10, 160)
    T = cfg.tokens_per_frame
    g.append([dev_bf16(np.ascontiguousarray(k[:, :8 * T, :])) for k in keys], 8, T)
    with pytest.raises(P.SSError) as e:
        g.append([dev_bf16(np.ascontiguousarray(k[:, :3 * T, :])) for k in keys], 3, T)
    assert e.value.status == 3
    assert g.info() == (8, 128)


# ---------------------------------------------------------------------------
# Compression (k-means at append)
# ---------------------------------------------------------------------------


KMEANS_MARGIN = 1e-5


KMEANS_SSE_BAND = 0.02


def _nearest_sse(X, C):
    """Sum over tokens of the squared distance to the nearest centre (float64)."""
    d2 = ((X[:, None, :] - C[None, :, :]) ** 2).sum(axis=2)
    return float(d2.min(axis=1).sum())


def _kmeans_audit(ex, keys, cfg, frames, n_c, n_it):
    """Where every farthest-point and assignment decision of the oracle has a
    relative margin of at least KMEANS_MARGIN (about ten times the relative error
    of a 128-term fp32 squared distance), the GPU's bf16 centroids are within one
    bf16 unit of the oracle's and the member counts are equal.  The other
    problems, where an fp32 near-tie may legitimately flip a decision, are
    checked by tolerance: their counts add up to the tokens, and the tokens'
    squared distance to their nearest stored centroid (the clustering's SSE)
    is within KMEANS_SSE_BAND of the same figure for the oracle's centroids.
    Returns (checked, exempt, largest relative SSE gap over all problems)."""
    T, d = cfg.tokens_per_frame, cfg.head_dim
    checked = exempt = 0
    sse_gap = 0.0
    for f in frames:
        for l in range(cfg.n_layers):
            for g in range(cfg.n_kv_heads):
                X = O.decode_bf16(keys[l][g, f * T:(f + 1) * T, :])
                C, cnt, dg = O.kmeans(X, n_c, n_it)
                got = ex["rows"][l, g, f * n_c:(f + 1) * n_c, :]
                got_cnt = ex["counts"][l, g, f * n_c:(f + 1) * n_c]
                want = O.round_bf16(C)
                s_gpu = _nearest_sse(X, O.decode_bf16(got))
                s_ora = _nearest_sse(X, O.decode_bf16(want))
                gap = abs(s_gpu - s_ora) / max(s_ora, 1e-300)
                sse_gap = max(sse_gap, gap)
                if min(dg["init_margin"], dg["assign_margin"]) < KMEANS_MARGIN:
                    exempt += 1
                    assert int(got_cnt.sum()) == T and np.all(got_cnt >= 0), (f, l, g)
                    assert gap <= KMEANS_SSE_BAND, (f, l, g, gap)
                    continue
                diff = np.abs(got.astype(np.int32) - want.astype(np.int32))
                assert diff.max() <= 1, (f, l, g)
                np.testing.assert_array_equal(got_cnt, cnt)
                checked += 1
    return checked, exempt, sse_gap


def test_compression_small_exact_cases():
    """T <= n_centroids stores the tokens themselves in farthest-point order."""
    cfg = W.Config("cs", 1, 2, 1, 64, 6, 2, 4, 2, n_frames=4)
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec)
    gidx, _ = make_pair(cfg, spec, keys, compress=(8, 3))
    ex = gidx.export()
    assert ex["frame_offsets"] == [0, 6, 12, 18, 24]
    for f in range(4):
        X = O.decode_bf16(keys[0][0, f * 6:(f + 1) * 6, :])
        _, _, dg = O.kmeans(X, 8, 3)
        np.testing.assert_array_equal(ex["rows"][0, 0, f * 6:(f + 1) * 6], keys[0][0, f * 6:(f + 1) * 6][dg["order"]])
        assert np.all(ex["counts"][0, 0, f * 6:(f + 1) * 6] == 1)


def test_compression_exact_ties():
    """Exact ties, which the oracle and the GPU must break the same way (lower
    token, lower centre): frame 0 holds 24 random tokens twice, so every
    farthest-point pick has an equal twin; frame 1 is symmetric (+-2 e_i and
    zero rows), so a zero row is equidistant from the first two centres.  Both
    frames are checked exactly: bf16 centres within one unit, equal counts."""
    P = _P()
    rng = np.random.default_rng(7)
    T, d = 48, 128
    base = rng.standard_normal((T // 2, d)).astype(np.float32)
    f0 = np.concatenate([base, base])
    f1 = np.zeros((T, d), dtype=np.float32)
    for i in range(8):
        f1[2 * i, i] = 2.0
        f1[2 * i + 1, i] = -2.0
    keys_f = np.concatenate([f0, f1])[None]                  # [H_kv = 1][2T][d]
    bits = W.bf16_bits(keys_f)
    for n_c, n_it in ((8, 3), (2, 2), (20, 4)):
        g = P.ShallowIndex(1, 1, 1, d, 2, 2 * n_c)
        g.append([dev_bf16(bits)], 2, T, (n_c, n_it))
        ex = g.export()
        for f in range(2):
            X = O.decode_bf16(bits[0, f * T:(f + 1) * T])
            C, cnt, _ = O.kmeans(X, n_c, n_it)
            got = ex["rows"][0, 0, f * n_c:(f + 1) * n_c]
            diff = np.abs(got.astype(np.int32) - O.round_bf16(C).astype(np.int32))
            assert diff.max() <= 1, (n_c, n_it, f)
            np.testing.assert_array_equal(ex["counts"][0, 0, f * n_c:(f + 1) * n_c], cnt)


def test_compression_c3_shape_audit_and_retrieval():
    """The C3 workload at 60 frames: k-means audit on every problem, then
    retrieval parity on the GPU's stored centroids."""
    base = W.CONFIGS["C3"]
    cfg = W.Config("C3s", base.n_layers, base.n_q_heads, base.n_kv_heads, base.head_dim, 196, base.n_q,
                   base.top_k, base.n_select, n_frames=60, n_planted=1, compress=(32, 10))
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec)
    log("C3-shape compressed append")
    gidx, _ = make_pair(cfg, spec, keys, compress=(32, 10))
    ex = gidx.export()
    checked, exempt, gap = _kmeans_audit(ex, keys, cfg, range(60), 32, 10)
    log("k-means audit", checked, "checked exactly,", exempt, "by tolerance; largest relative SSE gap", gap)
    assert checked >= 0.9 * (checked + exempt)
    oidx = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim)
    desc = [O.descriptor(O.decode_bf16(keys[-1][:, f * 196:(f + 1) * 196, :])) for f in range(60)]
    oidx.append_stored([ex["rows"][l] for l in range(cfg.n_layers)], [32] * 60, desc)
    np.testing.assert_allclose(ex["desc"], np.array(desc), atol=2e-6)
    out = debug_run([gidx], [q], cfg.top_k, cfg.n_select)
    rep = staged_check(oidx, q, out, 0, cfg.top_k, cfg.n_select)
    log(rep)


# ---------------------------------------------------------------------------
# Full-size workloads
# ---------------------------------------------------------------------------


def _build_big(cfg, spec, q, block=600, compress=None):
    P = _P()
    T = cfg.tokens_per_frame
    rpf = T if compress is None else compress[0]
    gidx = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, spec.n_frames,
                          spec.n_frames * rpf)
    host = [[] for _ in range(cfg.n_layers)]
    for f0 in range(0, spec.n_frames, block):
        f1 = min(spec.n_frames, f0 + block)
        kb = W.frame_block_keys(cfg, spec, q, f0, f1)
        gidx.append([dev_bf16(k) for k in kb], f1 - f0, T, compress)
        for l in range(cfg.n_layers):
            host[l].append(kb[l])
    torch.cuda.synchronize()
    keys = [np.concatenate(h, axis=1) for h in host]
    return gidx, keys


def _all_row_scores(gidx, oidx, q, lists, head_mode=0):
    """Per-key scores of every row of the given lists (layer, query head)
    against the oracle's: within 1e-3 D each, and the largest |err|/D."""
    qd = [dev_bf16(x) for x in q]
    S = O.score_lists(oidx, q, head_mode)
    D = score_scale(oidx, q, head_mode)
    Hq = oidx.Hq if head_mode == 0 else 1
    worst = 0.0
    for l, h in lists:
        g = gidx.debug_scores(qd, l, h, head_mode=head_mode).cpu().numpy().astype(np.float64)
        j = l * Hq + (h if head_mode == 0 else 0)
        assert g.shape == S[j].shape
        err = np.abs(g - S[j])
        assert np.all(err <= 1e-3 * D[j]), (l, h)
        worst = max(worst, float(np.max(err / D[j])))
    return worst


def _planted_checks(out, s, spec, F):
    planted = set(spec.planted)
    ranked = O.vote_pool(out["vote_hist"][s, :F].astype(np.int64), out["mass_hist"][s, :F].astype(np.float64), F)
    assert set(ranked[:len(planted)].tolist()) == planted            # P1
    assert out["frame_ids"][s, 0] in planted                          # P2


def _tally(total, rep):
    for k in ("swaps", "lists_with_swaps", "pool_exempt", "pool_differs", "maxmin_exempt"):
        total[k] = total.get(k, 0) + rep.get(k, 0)
    total["end_to_end_equal"] = total.get("end_to_end_equal", 0) + int(rep["end_to_end_equal"])
    total["max_rel_score_err"] = max(total.get("max_rel_score_err", 0.0), rep.get("max_rel_score_err", 0.0))


def test_c2_full_staged():
    """The 10-minute workload: staged in full, the planted evidence (P1-P3), and
    the per-key scores of every row of every list of layers 0 and 3 (all four
    KV-head groups, G = 7) and of every head-mean list."""
    cfg = W.CONFIGS["C2"]
    spec = W.stream_specs(cfg)[0]
    q = W.make_queries(cfg, 0, 0)
    log("C2 build")
    gidx, keys = _build_big(cfg, spec, q)
    oidx = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim)
    oidx.append(keys, spec.n_frames, cfg.tokens_per_frame)
    out = debug_run([gidx], [q], cfg.top_k, cfg.n_select)
    log("C2 list stats: max candidates", out["list_stats"][0, :, 0].max(), "fallbacks",
        out["list_stats"][0, :, 1].sum())
    rep = staged_check(oidx, q, out, 0, cfg.top_k, cfg.n_select)
    log("C2", rep)
    assert out["list_stats"][0, :, 1].sum() == 0
    _planted_checks(out, 0, spec, spec.n_frames)
    out1 = debug_run([gidx], [q], cfg.top_k, cfg.n_select, pool_mult=1)
    assert set(spec.planted) <= set(out1["frame_ids"][0].tolist())   # P3
    worst = _all_row_scores(gidx, oidx, q, [(l, h) for l in (0, 3) for h in range(cfg.n_q_heads)])
    log("C2 all rows, layers 0 and 3, every query head: max |err|/D", worst)
    assert worst < 1e-5
    worst1 = _all_row_scores(gidx, oidx, q, [(l, 0) for l in range(cfg.n_layers)], head_mode=1)
    log("C2 all rows, head-mean lists of every layer: max |err|/D", worst1)
    assert worst1 < 1e-5


def test_scores_all_rows_group_of_8():
    """The 16-stream workload's head shape (6 layers, 16 query / 2 KV heads,
    G = 8: the whole 16-column MFMA tile) at 400 frames: every row of every
    list of layers 0 and 5, and every head-mean list."""
    base = W.CONFIGS["C5"]
    cfg = W.Config("C5-shape", base.n_layers, base.n_q_heads, base.n_kv_heads, base.head_dim, 196, base.n_q,
                   base.top_k, base.n_select, n_frames=400, n_planted=3)
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec)
    gidx, oidx = make_pair(cfg, spec, keys)
    worst = _all_row_scores(gidx, oidx, q, [(l, h) for l in (0, 5) for h in range(cfg.n_q_heads)])
    log("G=8 all rows, layers 0 and 5, every query head: max |err|/D", worst)
    assert worst < 1e-5
    worst1 = _all_row_scores(gidx, oidx, q, [(l, 0) for l in range(cfg.n_layers)], head_mode=1)
    log("G=8 all rows, head-mean lists: max |err|/D", worst1)
    assert worst1 < 1e-5
    out = debug_run([gidx], [q], cfg.top_k, cfg.n_select)
    rep = staged_check(oidx, q, out, 0, cfg.top_k, cfg.n_select)
    log("G=8 staged", rep)


def test_c4_full_size_staged():
    """The 1-hour index at full size, in the launch configuration the benchmark
    times: every one of the 112 lists staged against the oracle (the scores of
    the selected rows, a tolerance-valid top-k, votes exactly, mass against the
    oracle's scores, pool and max-min), the frame ids end to end against the
    pure oracle, and the planted evidence."""
    cfg = W.CONFIGS["C4"]
    spec = W.stream_specs(cfg)[0]
    q = W.make_queries(cfg, 0, 0)
    log("C4 build")
    gidx, keys = _build_big(cfg, spec, q)
    P = _P()
    r = P.Retriever([gidx], cfg.top_k, cfg.n_select)
    qd = [[dev_bf16(x) for x in q]]
    ids, v, m, n = r(qd)
    torch.cuda.synchronize()
    plain = ids.cpu().numpy().copy()
    out = r.debug(qd)
    np.testing.assert_array_equal(plain, out["frame_ids"])
    stats = out["list_stats"][0]
    log("C4 candidates per list: min", stats[:, 0].min(), "max", stats[:, 0].max(), "fallbacks", stats[:, 1].sum())
    assert stats[:, 1].sum() == 0
    oidx = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim)
    oidx.append(keys, spec.n_frames, cfg.tokens_per_frame)
    del keys
    log("C4 oracle, 112 lists")
    rep = staged_check(oidx, q, out, 0, cfg.top_k, cfg.n_select)
    log("C4", rep)
    assert rep["lists"] == cfg.n_layers * cfg.n_q_heads
    _planted_checks(out, 0, spec, spec.n_frames)


def test_p4_paper_settings_full_size_staged():
    """The paper's own selection settings (one query token, head-averaged lists,
    top 64 per layer, pool 32, 8 units) on the 1-hour stream at full size, in
    the benchmark's launch configuration: all four layer lists staged against
    the oracle, the frame ids end to end, and the planted evidence."""
    cfg = W.CONFIGS["P4"]
    spec = W.stream_specs(cfg)[0]
    q = W.make_queries(cfg, 0, 0)
    log("P4 build")
    gidx, keys = _build_big(cfg, spec, q)
    P = _P()
    r = P.Retriever([gidx], cfg.top_k, cfg.n_select, cfg.pool_mult, 1)
    qd = [[dev_bf16(x) for x in q]]
    ids, v, m, n = r(qd)
    torch.cuda.synchronize()
    plain = ids.cpu().numpy().copy()
    out = r.debug(qd)
    np.testing.assert_array_equal(plain, out["frame_ids"])
    stats = out["list_stats"][0]
    log("P4 candidates per list", stats[:, 0].tolist(), "fallbacks", stats[:, 1].sum())
    assert stats[:, 1].sum() == 0
    oidx = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim)
    oidx.append(keys, spec.n_frames, cfg.tokens_per_frame)
    del keys
    log("P4 oracle, 4 layer lists")
    rep = staged_check(oidx, q, out, 0, cfg.top_k, cfg.n_select, cfg.pool_mult, head_mode=1)
    log("P4", rep)
    assert rep["lists"] == cfg.n_layers
    assert out["frame_ids"][0, 0] in set(spec.planted)
    # the paper's rule proper: head-averaged attention probabilities
    rp = P.Retriever([gidx], cfg.top_k, cfg.n_select, cfg.pool_mult, 1, 1)
    outp = rp.debug(qd)
    log("P4 probabilities: candidates per list", outp["list_stats"][0, :, 0].tolist(), "fallbacks",
        outp["list_stats"][0, :, 1].tolist())
    repp = staged_check(oidx, q, outp, 0, cfg.top_k, cfg.n_select, cfg.pool_mult, head_mode=1, score_mode=1)
    log("P4 probabilities", repp)
    assert outp["frame_ids"][0, 0] in set(spec.planted)


def test_c5_full_size_staged():
    """The 16-stream ragged batch at full size (odd streams compressed to 32
    centroids) in one call, the benchmark's launch configuration: every stream
    staged against the oracle in full (compressed streams on the GPU's stored
    centroids with the oracle's own descriptors from the raw keys), frame ids
    end to end, and the planted evidence."""
    cfg = W.CONFIGS["C5"]
    specs = W.stream_specs(cfg)
    P = _P()
    gidxs, qs = [], []
    for sp in specs:
        q = W.make_queries(cfg, 0, sp.stream)
        rpf = 196 if sp.compress is None else 32
        g = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, sp.n_frames,
                           sp.n_frames * rpf)
        for f0 in range(0, sp.n_frames, 600):
            f1 = min(sp.n_frames, f0 + 600)
            kb = W.frame_block_keys(cfg, sp, q, f0, f1)
            g.append([dev_bf16(k) for k in kb], f1 - f0, 196, sp.compress)
        torch.cuda.synchronize()
        gidxs.append(g)
        qs.append(q)
        log(f"C5 stream {sp.stream}: {sp.n_frames} frames, compressed {sp.compress is not None}")
    r = P.Retriever(gidxs, cfg.top_k, cfg.n_select)
    qd = [[dev_bf16(x) for x in q] for q in qs]
    ids, v, m, n = r(qd)
    torch.cuda.synchronize()
    plain = ids.cpu().numpy().copy()
    out = r.debug(qd)
    np.testing.assert_array_equal(plain, out["frame_ids"])
    total = {}
    for s, sp in enumerate(specs):
        assert out["list_stats"][s, :, 1].sum() == 0, f"stream {s} took the fallback"
        keys = W.frame_block_keys(cfg, sp, qs[s], 0, sp.n_frames)     # the same bytes again
        o = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim)
        if sp.compress is None:
            o.append(keys, sp.n_frames, 196)
        else:
            ex = gidxs[s].export()
            desc = [O.descriptor(O.decode_bf16(keys[-1][:, f * 196:(f + 1) * 196, :])) for f in range(sp.n_frames)]
            np.testing.assert_allclose(ex["desc"], np.array(desc), atol=2e-6)
            o.append_stored([ex["rows"][l] for l in range(cfg.n_layers)], [32] * sp.n_frames, desc)
            del ex
        del keys
        rep = staged_check(o, qs[s], out, s, cfg.top_k, cfg.n_select)
        log(f"C5 stream {s} ({sp.n_frames} frames)", rep)
        assert out["frame_ids"][s, 0] in set(sp.planted), f"stream {s}: first pick not planted"
        _tally(total, rep)
        del o
    log("C5 all streams", total)
    assert total["end_to_end_equal"] >= 1


def test_c3_full_size():
    """The compressed 10-minute workload at full size: 600 frames appended with
    per-frame k-means in the benchmark's 600-frame block, a k-means audit of 24
    frames spread over the stream, and retrieval parity (staged, in full) on
    the stored centroids."""
    cfg = W.CONFIGS["C3"]
    spec = W.stream_specs(cfg)[0]
    q = W.make_queries(cfg, 0, 0)
    log("C3 build")
    gidx, keys = _build_big(cfg, spec, q, compress=cfg.compress)
    ex = gidx.export()
    checked, exempt, gap = _kmeans_audit(ex, keys, cfg, range(0, spec.n_frames, 25), *cfg.compress)
    log("C3 k-means audit", checked, "checked exactly,", exempt, "by tolerance; largest relative SSE gap", gap)
    assert checked >= 0.9 * (checked + exempt)
    o = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim)
    desc = [O.descriptor(O.decode_bf16(keys[-1][:, f * 196:(f + 1) * 196, :])) for f in range(spec.n_frames)]
    np.testing.assert_allclose(ex["desc"], np.array(desc), atol=2e-6)
    o.append_stored([ex["rows"][l] for l in range(cfg.n_layers)], [32] * spec.n_frames, desc)
    del keys
    out = debug_run([gidx], [q], cfg.top_k, cfg.n_select)
    assert out["list_stats"][0, :, 1].sum() == 0
    rep = staged_check(o, q, out, 0, cfg.top_k, cfg.n_select)
    log("C3", rep)
    assert out["frame_ids"][0, 0] in set(spec.planted)
