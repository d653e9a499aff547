"""Pins of the CPU oracle against what the paper and the mathematics fix.

Hand-worked fixtures (tests/golden), closed forms, invariants, special cases and
an independent pure-Python brute force.  No GPU.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import brute
from oracle import oracle as O
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def bits(x):
    """Exact float -> bfloat16 bits (test inputs are exactly representable)."""
    a = np.asarray(x, dtype=np.float32)
    u = a.view(np.uint32)
    assert np.all((u & 0xFFFF) == 0), "value not exactly representable in bfloat16"
    return (u >> 16).astype(np.uint16)


def hand_index(spec, n_recent=0):
    sh = spec["shape"]
    idx = O.Index(sh["n_layers"], sh["n_q_heads"], sh["n_kv_heads"], sh["head_dim"], n_recent)
    rows = bits(spec["rows"])                         # [N][d]
    idx.append([rows[None, :, :]], sh["n_frames"], sh["tokens_per_frame"])
    q = [bits(spec["queries"])]                       # [H_q][n_q][d]
    return idx, q


# ---------------------------------------------------------------------------
# bfloat16 handling
# ---------------------------------------------------------------------------

def test_bf16_known_patterns():
    assert O.decode_bf16(np.array([0x3F80], np.uint16))[0] == 1.0
    assert O.decode_bf16(np.array([0xC020], np.uint16))[0] == -2.5
    # 1 + 2^-8 is half-way between 1 and 1 + 2^-7: ties to the even significand (1.0)
    assert O.round_bf16(np.array([1 + 2 ** -8]))[0] == 0x3F80
    # 1 + 3*2^-8 is half-way between 1+2^-7 and 1+2^-6: even is 1+2^-6
    assert O.round_bf16(np.array([1 + 3 * 2 ** -8]))[0] == 0x3F82
    assert O.round_bf16(np.array([1 + 2 ** -8 + 2 ** -30]))[0] == 0x3F81
    with pytest.raises(ValueError):
        O.decode_bf16(np.array([0x7FC0], np.uint16))


def test_bf16_rounding_is_nearest():
    x = np.abs(np.random.default_rng(3).standard_normal(20000)) * np.logspace(-30, 30, 20000)
    b = O.round_bf16(x)
    err = np.abs(O.decode_bf16(b) - x)
    up = np.abs(O.decode_bf16((b + 1).astype(np.uint16)) - x)
    dn = np.abs(O.decode_bf16((b - 1).astype(np.uint16)) - x)
    assert np.all(err <= up) and np.all(err <= dn)


# ---------------------------------------------------------------------------
# Hand-worked end-to-end fixture
# ---------------------------------------------------------------------------

def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_hand_scores():
    spec = _load("hand_retrieval.json")
    idx, q = hand_index(spec)
    S = O.score_lists(idx, q)
    for got, want in zip(S, spec["scores"]):
        np.testing.assert_array_equal(got, np.array(want, dtype=np.float64))
    (hm,) = O.score_lists(idx, q, head_mode=1)
    np.testing.assert_array_equal(hm, np.array(spec["scores_head_mean"], dtype=np.float64))


@pytest.mark.parametrize("case", [c["name"] for c in _load("hand_retrieval.json")["cases"]])
def test_hand_retrieval(case):
    spec = _load("hand_retrieval.json")
    c = next(c for c in spec["cases"] if c["name"] == case)
    idx, q = hand_index(spec, c["n_recent"])
    ids, v, m, n, dbg = O.retrieve(idx, q, c["top_k"], c["n_select"], c["pool_mult"],
                                   head_mode=c.get("head_mode", 0), debug=True)
    assert [list(t) for t in dbg["topk"]] == c["topk"]
    assert list(dbg["votes"]) == c["votes"]
    np.testing.assert_allclose(dbg["mass"], c["mass"], rtol=0, atol=1e-12)
    assert list(dbg["pool"]) == c["pool"]
    assert list(ids) == c["frame_ids"] and list(v) == c["sel_votes"] and n == c["n_out"]
    np.testing.assert_allclose(m, c["sel_mass"], rtol=0, atol=1e-12)


def _closed_form(expr, defs):
    """Evaluates a fixture's hand-derived closed form (exp, sqrt, + - * / and the
    fixture's named normalisers only)."""
    env = {"exp": math.exp, "sqrt": math.sqrt}
    for k, e in defs.items():
        env[k] = eval(e, {"__builtins__": {}}, dict(env))
    return float(eval(expr, {"__builtins__": {}}, env))


@pytest.mark.parametrize("case", [c["name"] for c in _load("hand_attention.json")["cases"]])
def test_hand_attention(case):
    """The logit and the attention-probability readings on a hand-worked index
    where they select different rows (head mode 1) and rank the pool
    differently (head mode 0)."""
    spec = _load("hand_attention.json")
    c = next(c for c in spec["cases"] if c["name"] == case)
    cf = lambda e: _closed_form(e, spec["defs"])
    idx, q = hand_index(spec, c["n_recent"])
    hm, sm = c["head_mode"], c["score_mode"]
    if "values" in c:
        S = O.score_lists(idx, q, hm, sm)
        assert len(S) == len(c["values"])
        for got, want in zip(S, c["values"]):
            np.testing.assert_allclose(got, [cf(e) for e in want], rtol=1e-13, atol=1e-15)
    ids, v, m, n, dbg = O.retrieve(idx, q, c["top_k"], c["n_select"], c["pool_mult"],
                                   head_mode=hm, score_mode=sm, debug=True)
    assert [list(t) for t in dbg["topk"]] == c["topk"]
    assert list(dbg["votes"]) == c["votes"]
    np.testing.assert_allclose(dbg["mass"], [cf(e) for e in c["mass"]], rtol=1e-13, atol=1e-15)
    assert list(dbg["pool"]) == c["pool"]
    assert list(ids) == c["frame_ids"] and list(v) == c["sel_votes"] and n == c["n_out"]
    np.testing.assert_allclose(m, [cf(e) for e in c["sel_mass"]], rtol=1e-13, atol=1e-15)


def test_hand_attention_descriptor_distances():
    spec = _load("hand_attention.json")
    idx, _ = hand_index(spec)
    D = np.array(idx.desc)
    dist = {k: _closed_form(e, {}) for k, e in spec["distances"].items()}
    assert math.isclose(1 - D[0] @ D[1], dist["f0_f1"], abs_tol=1e-14)
    assert math.isclose(1 - D[0] @ D[2], dist["f0_f2"], abs_tol=1e-14)
    assert math.isclose(1 - D[1] @ D[2], dist["f1_f2"], abs_tol=1e-14)


def test_readings_disagree_only_where_expected():
    """On the attention fixture the two readings give different head-mode-1
    lists and different head-mode-0 pools, but the same head-mode-0 lists."""
    spec = _load("hand_attention.json")
    idx, q = hand_index(spec)
    r = {sm: O.retrieve(idx, q, 2, 2, 1, head_mode=0, score_mode=sm, debug=True)[4] for sm in (0, 1)}
    assert [list(t) for t in r[0]["topk"]] == [list(t) for t in r[1]["topk"]]
    assert list(r[0]["pool"]) != list(r[1]["pool"])
    h = {sm: O.retrieve(idx, q, 2, 2, 4, head_mode=1, score_mode=sm, debug=True)[4] for sm in (0, 1)}
    assert list(h[0]["topk"][0]) != list(h[1]["topk"][0])


def test_hand_descriptor_distances():
    spec = _load("hand_retrieval.json")
    idx, _ = hand_index(spec)
    D = np.array(idx.desc)
    assert math.isclose(1 - D[0] @ D[1], spec["distances_to_f0"]["f1"], abs_tol=1e-12)
    assert math.isclose(1 - D[0] @ D[2], spec["distances_to_f0"]["f2"], abs_tol=1e-12)
    assert math.isclose(1 - D[1] @ D[2], spec["distance_f1_f2"], abs_tol=1e-12)


# ---------------------------------------------------------------------------
# Scoring
# ---------------------------------------------------------------------------

def _random_index(rng, L=2, Hq=4, Hk=2, d=8, F=6, T=3, n_recent=0, scale=1.0):
    idx = O.Index(L, Hq, Hk, d, n_recent)
    keys = [bits(np.round(rng.standard_normal((Hk, F * T, d)) * scale * 8) / 8) for _ in range(L)]
    idx.append(keys, F, T)
    return idx, keys


def _random_queries(rng, L=2, Hq=4, nq=3, d=8):
    return [bits(np.round(rng.standard_normal((Hq, nq, d)) * 8) / 8) for _ in range(L)]


def test_score_is_mean_of_token_logits():
    """The pre-averaged query gives the mean of the per-token scaled logits."""
    rng = np.random.default_rng(0)
    idx, keys = _random_index(rng)
    q = _random_queries(rng)
    S = O.score_lists(idx, q)
    d = idx.d
    for l in range(idx.L):
        for h in range(idx.Hq):
            g = h // idx.G
            K = O.decode_bf16(keys[l][g])
            Q = O.decode_bf16(q[l][h])
            want = np.array([math.fsum(math.fsum(Q[j] * K[p]) / math.sqrt(d) for j in range(Q.shape[0])) / Q.shape[0]
                             for p in range(K.shape[0])])
            np.testing.assert_allclose(S[l * idx.Hq + h], want, rtol=1e-13, atol=1e-13)


def test_score_linear_in_query():
    rng = np.random.default_rng(1)
    idx, _ = _random_index(rng)
    q = _random_queries(rng)
    q2 = [bits(2 * O.decode_bf16(x)) for x in q]       # doubling is exact in bfloat16
    for a, b in zip(O.score_lists(idx, q), O.score_lists(idx, q2)):
        np.testing.assert_array_equal(2 * a, b)


def test_gqa_mapping():
    """Query head h reads KV head h // G (contiguous groups)."""
    d, T = 4, 1
    idx = O.Index(1, 4, 2, d)
    k0 = np.zeros((2, 2, d), np.float32)
    k0[0, :, 0] = [1, 2]      # KV head 0: scores along e0
    k0[1, :, 1] = [5, 7]      # KV head 1: scores along e1
    idx.append([bits(k0)], 2, T)
    q = np.zeros((4, 1, d), np.float32)
    q[:, 0, 0] = 2.0
    q[:, 0, 1] = 4.0          # every head probes e0 with weight 2 and e1 with weight 4
    S = O.score_lists(idx, [bits(q)])
    for h in range(4):
        want = [1.0, 2.0] if h < 2 else [10.0, 14.0]    # (1/sqrt(4)) * q.k
        np.testing.assert_array_equal(S[h], want)


def test_head_mean_equal_heads_reduce_to_one_head():
    """Special case: when every query head of a layer carries the same query and
    every KV head the same keys, the head average of either reading is the
    single head's value, a textbook dot product (or its softmax)."""
    rng = np.random.default_rng(2)
    L, Hq, Hk, d, F, T = 2, 4, 2, 8, 5, 3
    k1 = [np.round(rng.standard_normal((1, F * T, d)) * 8) / 8 for _ in range(L)]
    keys = [bits(np.repeat(k, Hk, axis=0)) for k in k1]
    q1 = [np.round(rng.standard_normal((1, 1, d)) * 8) / 8 for _ in range(L)]
    q = [bits(np.repeat(x, Hq, axis=0)) for x in q1]
    idx = O.Index(L, Hq, Hk, d)
    idx.append(keys, F, T)
    for l in range(L):
        K = O.decode_bf16(keys[l][0])
        qv = O.decode_bf16(q[l][0, 0])
        logit = np.array([math.fsum(K[p] * qv) for p in range(F * T)]) / math.sqrt(d)
        m = logit.max()
        prob = np.exp(logit - m) / math.fsum(np.exp(logit - m))
        np.testing.assert_allclose(O.score_lists(idx, q, 1, 0)[l], logit, rtol=1e-14, atol=1e-14)
        np.testing.assert_allclose(O.score_lists(idx, q, 1, 1)[l], prob, rtol=1e-13, atol=1e-16)


def test_attention_probabilities_are_distributions():
    """Each (layer, head)'s probabilities are positive and sum to one over the
    candidates, keep the order of its logits (so head-mode-0 lists are the same
    in both readings), and their head mean sums to one as well."""
    rng = np.random.default_rng(12)
    idx, _ = _random_index(rng, F=7, T=4, n_recent=2)
    q = _random_queries(rng)
    lg = O.score_lists(idx, q, 0, 0)
    pr = O.score_lists(idx, q, 0, 1)
    for a, b in zip(lg, pr):
        assert np.all(b > 0) and math.isclose(math.fsum(b), 1.0, rel_tol=1e-13)
        np.testing.assert_array_equal(O.topk(a, a.size), O.topk(b, b.size))
    for hm in O.score_lists(idx, q, 1, 1):
        assert math.isclose(math.fsum(hm), 1.0, rel_tol=1e-13)
    # shifting every logit of a list by a constant leaves its probabilities unchanged:
    # doubling a query is not a shift, but a zero query gives the uniform distribution
    zq = [np.zeros_like(x) for x in q]
    for b in O.score_lists(idx, zq, 0, 1):
        np.testing.assert_allclose(b, 1.0 / b.size, rtol=1e-15)


def test_attention_probabilities_of_huge_logits():
    """Logits 1024, 1020 and 0 (exp(1024) overflows float64): the probabilities
    are 1/(1+e^-4), e^-4/(1+e^-4) and 0 in closed form."""
    idx = O.Index(1, 1, 1, 4)
    idx.append([bits(np.array([[[1024, 0, 0, 0], [1020, 0, 0, 0], [0, 0, 0, 0]]], np.float32))], 3, 1)
    q = [bits(np.array([[[2, 0, 0, 0]]], np.float32))]
    (b,) = O.score_lists(idx, q, 0, 1)
    e4 = math.exp(-4.0)
    np.testing.assert_allclose(b, [1 / (1 + e4), e4 / (1 + e4), 0.0], rtol=1e-15, atol=0)


# ---------------------------------------------------------------------------
# Top-k and votes
# ---------------------------------------------------------------------------

def test_zero_query_selects_lowest_positions_c1():
    """All-zero queries make every score 0, so each list keeps rows 0..k-1: at
    the C1 shape frames 0 and 1 get 16 rows x 8 lists = 128 votes each."""
    cfg = W.CONFIGS["C1"]
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec, threads=2)
    idx = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim)
    idx.append(keys, spec.n_frames, cfg.tokens_per_frame)
    zq = [np.zeros_like(x) for x in q]
    ids, v, m, n, dbg = O.retrieve(idx, zq, cfg.top_k, cfg.n_select, debug=True)
    for t in dbg["topk"]:
        np.testing.assert_array_equal(t, np.arange(cfg.top_k))
    assert dbg["votes"][0] == 128 and dbg["votes"][1] == 128 and dbg["votes"][2:].sum() == 0
    assert n == 2 and set(ids[:2]) == {0, 1} and ids[0] == 0


def test_topk_ties_and_k_beyond_n():
    s = np.array([1.0, 3.0, 3.0, 0.5, 3.0])
    np.testing.assert_array_equal(O.topk(s, 2), [1, 2])
    np.testing.assert_array_equal(O.topk(s, 4), [1, 2, 4, 0])
    np.testing.assert_array_equal(O.topk(s, 99), [1, 2, 4, 0, 3])


def test_duplicated_keys_tie_to_lower_position():
    d = 4
    idx = O.Index(1, 1, 1, d)
    k = np.tile(np.array([[1, 2, 3, 4]], np.float32), (6, 1))[None]    # six equal rows
    idx.append([bits(k)], 3, 2)
    q = bits(np.array([[[1, 0, 0, 1]]], np.float32))
    ids, v, m, n, dbg = O.retrieve(idx, [q], 3, 2, debug=True)
    np.testing.assert_array_equal(dbg["topk"][0], [0, 1, 2])
    assert list(dbg["votes"]) == [2, 1, 0]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_vote_sum_invariant(seed):
    rng = np.random.default_rng(seed)
    idx, _ = _random_index(rng, F=7, T=4)
    q = _random_queries(rng)
    for k in (1, 5, 28, 100):
        for sm in (0, 1):
            _, _, _, _, dbg = O.retrieve(idx, q, k, 3, debug=True, score_mode=sm)
            assert dbg["votes"].sum() == idx.L * idx.Hq * min(k, idx.candidate_rows())
            # head mode 1: one list per layer, so sum v = L min(k, N)
            _, _, _, _, dbg = O.retrieve(idx, q, k, 3, head_mode=1, debug=True, score_mode=sm)
            assert dbg["votes"].sum() == idx.L * min(k, idx.candidate_rows())
            assert all(len(t) == min(k, idx.candidate_rows()) for t in dbg["topk"])


def test_votes_invariant_under_row_permutation_within_frame():
    rng = np.random.default_rng(5)
    L, Hq, Hk, d, F, T = 2, 4, 2, 8, 5, 4
    keys = [rng.standard_normal((Hk, F * T, d)).astype(np.float32) for _ in range(L)]
    q = _random_queries(rng, L, Hq, 2, d)
    perm = np.concatenate([f * T + rng.permutation(T) for f in range(F)])
    a = O.Index(L, Hq, Hk, d)
    a.append([W.bf16_bits(k) for k in keys], F, T)
    b = O.Index(L, Hq, Hk, d)
    b.append([W.bf16_bits(k[:, perm, :]) for k in keys], F, T)
    ra = O.retrieve(a, q, 6, 3, debug=True)
    rb = O.retrieve(b, q, 6, 3, debug=True)
    np.testing.assert_array_equal(ra[4]["votes"], rb[4]["votes"])
    np.testing.assert_allclose(ra[4]["mass"], rb[4]["mass"], rtol=1e-12)
    np.testing.assert_array_equal(ra[0], rb[0])
    np.testing.assert_allclose(a.desc, b.desc, rtol=0, atol=1e-15)


def test_pool_excludes_unvoted_and_orders():
    votes = np.array([0, 3, 3, 1, 0, 3])
    mass = np.array([9.0, 1.0, 2.0, 5.0, 0.0, 2.0])
    np.testing.assert_array_equal(O.vote_pool(votes, mass, 10), [2, 5, 1, 3])
    np.testing.assert_array_equal(O.vote_pool(votes, mass, 2), [2, 5])


# ---------------------------------------------------------------------------
# Max-min diversity
# ---------------------------------------------------------------------------

def _unit(deg):
    r = math.radians(deg)
    return np.array([math.cos(r), math.sin(r), 0.0])


def test_maxmin_planar_known_order():
    """Unit vectors at 0, 10, 90 and 180 degrees in pool order: from 0 the farthest
    is 180 (distance 2), then 90 (min distance 1), then 10."""
    desc = np.array([_unit(0), _unit(10), _unit(90), _unit(180)])
    sel, margins = O.maxmin_select(np.arange(4), desc, 4)
    np.testing.assert_array_equal(sel, [0, 3, 2, 1])
    assert margins[0] == pytest.approx(2 - 1)        # 180 vs 90 at the first step
    sel2, _ = O.maxmin_select(np.arange(4), desc, 2)
    np.testing.assert_array_equal(sel2, [0, 3])


def test_maxmin_orthonormal_keeps_pool_order():
    desc = np.eye(6)
    pool = np.array([4, 1, 5, 0])
    sel, _ = O.maxmin_select(pool, desc, 3)
    np.testing.assert_array_equal(sel, [4, 1, 5])


def test_maxmin_duplicates_picked_last_and_whole_pool():
    desc = np.array([_unit(0), _unit(0), _unit(50), _unit(50), _unit(120)])
    sel, _ = O.maxmin_select(np.arange(5), desc, 5)
    assert list(sel[:3]) == [0, 4, 2] and sorted(sel[3:]) == [1, 3]
    sel3, _ = O.maxmin_select(np.arange(5), desc, 3)
    assert len(set(np.round([desc[i][0] for i in sel3], 9))) == 3


def test_maxmin_greedy_property_random():
    rng = np.random.default_rng(7)
    desc = rng.standard_normal((12, 5))
    desc /= np.linalg.norm(desc, axis=1, keepdims=True)
    pool = rng.permutation(12)[:9]
    sel, _ = O.maxmin_select(pool, desc, 6)
    chosen = [sel[0]]
    assert sel[0] == pool[0]
    for s in sel[1:]:
        rest = [u for u in pool if u not in chosen]
        val = {u: min(1 - desc[u] @ desc[c] for c in chosen) for u in rest}
        assert val[s] == max(val.values())
        chosen.append(s)


# ---------------------------------------------------------------------------
# Descriptor (Eq. memory_key)
# ---------------------------------------------------------------------------

def test_descriptor_properties():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((3, 7, 5))
    dsc = O.descriptor(x)
    assert abs(np.linalg.norm(dsc) - 1) < 1e-12
    np.testing.assert_allclose(O.descriptor(x[:, rng.permutation(7), :]), dsc, atol=1e-15)
    c = np.tile(np.arange(1.0, 6.0)[None, None, :], (2, 4, 1))
    want = np.tile(np.arange(1.0, 6.0), 2)
    np.testing.assert_allclose(O.descriptor(c), want / np.linalg.norm(want), atol=1e-15)
    # head-major flatten: KV head 0's mean comes first
    y = np.zeros((2, 1, 3))
    y[0, 0] = [3, 0, 0]
    y[1, 0] = [0, 0, 4]
    np.testing.assert_allclose(O.descriptor(y), [0.6, 0, 0, 0, 0, 0.8])
    np.testing.assert_array_equal(O.descriptor(np.zeros((2, 3, 4))), np.zeros(8))


# ---------------------------------------------------------------------------
# k-means compression
# ---------------------------------------------------------------------------

def test_kmeans_hand_example():
    spec = _load("hand_kmeans.json")
    C, counts, diag = O.kmeans(np.array(spec["tokens"], float), spec["n_centroids"], spec["n_iters"])
    assert diag["order"] == spec["order"]
    np.testing.assert_array_equal(C, spec["centroids"])
    np.testing.assert_array_equal(counts, spec["counts"])


def test_kmeans_fewer_tokens_than_centroids():
    rng = np.random.default_rng(0)
    X = rng.standard_normal((5, 3))
    C, counts, diag = O.kmeans(X, 8, 10)
    assert C.shape == (5, 3)
    np.testing.assert_array_equal(C, X[diag["order"]])
    np.testing.assert_array_equal(counts, np.ones(5))
    assert sorted(diag["order"]) == list(range(5))


def test_kmeans_single_centroid_is_mean():
    X = np.random.default_rng(1).standard_normal((20, 4))
    C, counts, _ = O.kmeans(X, 1, 3)
    np.testing.assert_allclose(C[0], X.mean(axis=0), atol=1e-15)
    assert counts[0] == 20


def test_kmeans_separated_blobs():
    rng = np.random.default_rng(2)
    centres = np.array([[0, 0, 0], [100, 0, 0], [0, 100, 0], [0, 0, 100]], float)
    X = np.concatenate([c + rng.standard_normal((10, 3)) for c in centres])
    C, counts, _ = O.kmeans(X, 4, 10)
    got = sorted(map(tuple, np.round(C, 9)))
    want = sorted(tuple(np.round(X[i * 10:(i + 1) * 10].mean(axis=0), 9)) for i in range(4))
    assert got == want
    assert sorted(counts) == [10, 10, 10, 10]


def test_kmeans_sse_non_increasing_and_farthest_point():
    rng = np.random.default_rng(3)
    X = rng.standard_normal((60, 6))
    C, counts, diag = O.kmeans(X, 8, 10)
    sse = diag["sse"]
    assert all(b <= a + 1e-12 for a, b in zip(sse, sse[1:]))
    order = diag["order"]
    mu = X.mean(axis=0)
    assert order[0] == int(np.argmax(((X - mu) ** 2).sum(1)))
    for i in range(1, len(order)):
        dmin = np.min([((X - X[j]) ** 2).sum(1) for j in order[:i]], axis=0)
        dmin[order[:i]] = -1
        assert order[i] == int(np.argmax(dmin))
    assert counts.sum() == 60


def test_kmeans_matches_brute():
    rng = np.random.default_rng(4)
    X = rng.standard_normal((17, 4))
    C, counts, diag = O.kmeans(X, 5, 6)
    Cb, cb, ob = brute.kmeans(X.tolist(), 5, 6)
    assert diag["order"] == ob
    np.testing.assert_allclose(C, np.array(Cb), atol=1e-12)
    np.testing.assert_array_equal(counts, cb)


def test_compressed_append_rows_and_counts():
    rng = np.random.default_rng(6)
    L, Hk, d, F, T = 2, 2, 8, 3, 12
    keys = [W.bf16_bits(rng.standard_normal((Hk, F * T, d)).astype(np.float32)) for _ in range(L)]
    idx = O.Index(L, 2, Hk, d)
    idx.append(keys, F, T, compress=(4, 5))
    assert idx.row_count == [4, 4, 4] and idx.n_rows == 12
    raw = O.Index(L, 2, Hk, d)
    raw.append(keys, F, T)
    np.testing.assert_array_equal(np.array(idx.desc), np.array(raw.desc))   # raw keys feed the descriptor
    for f in range(F):
        assert idx.counts[f].sum(axis=2).tolist() == [[T] * Hk] * L


# ---------------------------------------------------------------------------
# Oracle vs. brute force, end to end
# ---------------------------------------------------------------------------

def _brute_frames(keys, F, T, L, Hk):
    return [[[[keys[l][g][t * T + p] for p in range(T)] for g in range(Hk)] for l in range(L)] for t in range(F)]


@pytest.mark.parametrize("seed,k,K,pm,nr,Hq,Hk,hm,sm", [
    (0, 4, 3, 4, 0, 4, 2, 0, 0), (1, 9, 2, 1, 0, 4, 4, 0, 0), (2, 200, 4, 4, 0, 2, 1, 0, 0),
    (3, 3, 5, 2, 2, 6, 2, 0, 0), (4, 1, 1, 4, 0, 4, 2, 0, 0), (5, 6, 4, 4, 6, 4, 2, 0, 0),
    (6, 4, 3, 4, 0, 4, 2, 1, 0), (7, 9, 2, 4, 1, 6, 2, 1, 0), (8, 200, 4, 4, 0, 2, 1, 1, 0),
    (9, 4, 3, 4, 0, 4, 2, 0, 1), (10, 3, 5, 2, 2, 6, 2, 0, 1), (11, 4, 3, 4, 0, 4, 2, 1, 1),
    (12, 7, 2, 4, 1, 6, 3, 1, 1), (13, 200, 4, 4, 0, 2, 1, 1, 1)])
def test_oracle_matches_brute(seed, k, K, pm, nr, Hq, Hk, hm, sm):
    rng = np.random.default_rng(seed)
    L, d, F, T, nq = 2, 8, 6, 5, 3
    keys = [W.bf16_bits(rng.standard_normal((Hk, F * T, d)).astype(np.float32)) for _ in range(L)]
    q = [W.bf16_bits(rng.standard_normal((Hq, nq, d)).astype(np.float32)) for _ in range(L)]
    idx = O.Index(L, Hq, Hk, d, nr)
    idx.append(keys, F, T)
    ids, v, m, n, dbg = O.retrieve(idx, q, k, K, pm, head_mode=hm, score_mode=sm, debug=True)
    frames = _brute_frames(keys, F, T, L, Hk)
    qs = [[[q[l][h][j] for j in range(nq)] for h in range(Hq)] for l in range(L)]
    bi, bv, bm, bd = brute.retrieve(frames, qs, Hk, k, K, pm, nr, head_mode=hm, score_mode=sm)
    assert list(ids) == bi and list(v) == bv and n == sum(1 for x in bi if x >= 0)
    np.testing.assert_allclose(m, bm, rtol=1e-12, atol=1e-12)
    assert [list(t) for t in dbg["topk"]] == [[r[2] for r in lst] for lst in bd["lists"]]
    assert list(dbg["votes"]) == bd["votes"]
    assert list(dbg["pool"]) == bd["pool"]
    np.testing.assert_allclose(np.array(idx.desc), np.array(bd["desc"]), atol=1e-14)


def test_no_candidates():
    rng = np.random.default_rng(9)
    idx, _ = _random_index(rng, F=3, n_recent=5)
    q = _random_queries(rng)
    ids, v, m, n = O.retrieve(idx, q, 4, 3)
    assert n == 0 and list(ids) == [-1, -1, -1]


# ---------------------------------------------------------------------------
# Planted evidence
# ---------------------------------------------------------------------------

def _planted_case(cfg):
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec, threads=4)
    idx = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim)
    idx.append(keys, spec.n_frames, cfg.tokens_per_frame)
    return spec, q, idx


def test_planted_c1():
    cfg = W.CONFIGS["C1"]
    spec, q, idx = _planted_case(cfg)
    ids, v, m, n, dbg = O.retrieve(idx, q, cfg.top_k, cfg.n_select, debug=True)
    planted = set(spec.planted)
    ranked = list(O.vote_pool(dbg["votes"], dbg["mass"], idx.n_frames))
    assert set(ranked[:len(planted)]) == planted          # P1
    assert ids[0] in planted                                # P2
    ids1, *_ = O.retrieve(idx, q, cfg.top_k, cfg.n_select, pool_mult=1)
    assert planted <= set(ids1)                             # P3


def test_planted_small_gqa7():
    """A reduced C2 shape (G=7, d=128, 60 frames x 49 tokens, 3 planted)."""
    cfg = W.Config("mini", 2, 14, 2, 128, 49, 16, 64, 4, n_frames=60, n_planted=3)
    spec, q, idx = _planted_case(cfg)
    ids, v, m, n, dbg = O.retrieve(idx, q, cfg.top_k, cfg.n_select, debug=True)
    planted = set(spec.planted)
    ranked = list(O.vote_pool(dbg["votes"], dbg["mass"], idx.n_frames))
    assert set(ranked[:3]) == planted and ids[0] in planted
    ids1, *_ = O.retrieve(idx, q, cfg.top_k, cfg.n_select, pool_mult=1)
    assert planted <= set(ids1)


# ---------------------------------------------------------------------------
# Generator
# ---------------------------------------------------------------------------

def test_generator_deterministic_and_blockwise():
    cfg = W.CONFIGS["C1"]
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec, threads=3)
    q2, keys2 = W.make_stream(cfg, spec, threads=1)
    for a, b in zip(keys, keys2):
        np.testing.assert_array_equal(a, b)
    a = W.frame_block_keys(cfg, spec, q, 0, 20)
    b = W.frame_block_keys(cfg, spec, q, 20, 64)
    T = cfg.tokens_per_frame
    for l in range(cfg.n_layers):
        np.testing.assert_array_equal(np.concatenate([a[l], b[l]], axis=1), keys[l])
    assert keys[0].shape == (2, 64 * 16, 64) and spec.planted == (16, 48)


def test_generator_c5_specs():
    specs = W.stream_specs(W.CONFIGS["C5"])
    assert len(specs) == 16
    assert all(300 <= s.n_frames <= 3600 for s in specs)
    assert all((s.compress is not None) == (s.stream % 2 == 1) for s in specs)
    assert all(s.n_planted == math.ceil(s.n_frames / 150) for s in specs)


# ---------------------------------------------------------------------------
# Evidence assembly (Eq. selected_evidence, deduplication, temporal order)
# ---------------------------------------------------------------------------

def _evidence_cases():
    with open(os.path.join(GOLDEN, "evidence_hand.json")) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("case", _evidence_cases(), ids=lambda c: c["name"])
def test_evidence_hand(case):
    got = O.evidence_units(case["n_frames"], case["selected"], case["n_recent"], case["n_before"],
                           case["n_after"], case["retrieved"])
    assert got.tolist() == case["units"]


def test_evidence_invariants_random():
    """Sorted, repeat-free, holds the recent window and every selected unit,
    every member is recent or within the neighbourhood of a selected unit, and
    the size stays within N_r + |sel| (1 + before + after).  Checked against a
    per-unit membership test written from the definition."""
    rng = np.random.default_rng(5)
    for _ in range(300):
        T = int(rng.integers(0, 60))
        nr, nb, na = (int(x) for x in rng.integers(0, 5, size=3))
        nsel = int(rng.integers(0, 8))
        sel = rng.integers(0, max(T, 1), size=nsel) if T > 0 else np.zeros(0, np.int64)
        sel = np.concatenate([sel, -np.ones(int(rng.integers(0, 3)), np.int64)])
        got = O.evidence_units(T, sel, nr, nb, na, True)
        assert np.all(np.diff(got) > 0)
        want = [u for u in range(T)
                if u >= T - nr or any(0 <= s and s - nb <= u <= s + na for s in sel.tolist())]
        assert got.tolist() == want
        assert set(range(max(0, T - nr), T)) <= set(got.tolist())
        assert {int(s) for s in sel if s >= 0} <= set(got.tolist())
        assert got.size <= nr + int((sel >= 0).sum()) * (1 + nb + na)
        only = O.evidence_units(T, sel, nr, nb, na, False)
        assert only.tolist() == list(range(max(0, T - nr), T))


@pytest.mark.parametrize("case", _load("evidence_hand.json")["cluster_cases"], ids=lambda c: c["name"])
def test_evidence_with_clusters_hand(case):
    ids, kinds = O.evidence_items(case["n_frames"], case["selected"], case["n_recent"], case["n_before"],
                                  case["n_after"], case["retrieved"], case["first_detail"], case["cluster_first"],
                                  case["selected_clusters"])
    assert ids.tolist() == case["ids"] and kinds.tolist() == case["kinds"]


def test_evidence_with_clusters_invariants_random():
    """Against a membership test written from the definition: the detailed part
    is every unit of [first_detail, T) that is recent or a neighbour of a
    selected unit, each retrieved cluster appears once, and the items run in
    the order of their positions (a cluster at its first member unit)."""
    rng = np.random.default_rng(6)
    for _ in range(300):
        T = int(rng.integers(1, 60))
        fd = int(rng.integers(0, T + 1))
        cuts = sorted(set(rng.integers(1, fd + 1, size=int(rng.integers(0, 5))).tolist())) if fd > 0 else []
        firsts = [0] + [c for c in cuts if c < fd] if fd > 0 else []
        nr, nb, na = (int(x) for x in rng.integers(0, 5, size=3))
        sel = rng.integers(fd, T, size=int(rng.integers(0, 6))) if fd < T else np.zeros(0, np.int64)
        sc = rng.integers(-1, len(firsts) + 2, size=int(rng.integers(0, 6)))
        ids, kinds = O.evidence_items(T, sel, nr, nb, na, True, fd, firsts, sc)
        det = [u for u in range(fd, T)
               if u >= T - nr or any(s - nb <= u <= s + na for s in sel.tolist())]
        cl = sorted({int(j) for j in sc if 0 <= j < len(firsts)})
        assert ids[kinds == 0].tolist() == det
        assert sorted(ids[kinds == 1].tolist()) == cl
        pos = [int(i) if k == 0 else firsts[int(i)] for i, k in zip(ids, kinds)]
        assert pos == sorted(pos) and len(set(pos)) == len(pos)
        only_ids, only_kinds = O.evidence_items(T, sel, nr, nb, na, False, fd, firsts, sc)
        assert only_ids.tolist() == list(range(max(fd, T - nr), T)) and not only_kinds.any()


def test_evidence_rejects_bad_input():
    with pytest.raises(ValueError):
        O.evidence_units(5, [7], 2)
    with pytest.raises(ValueError):
        O.evidence_units(5, [1], -1)


# ---------------------------------------------------------------------------
# Pooled shallow Q-K ranker
# ---------------------------------------------------------------------------

def test_pooled_hand():
    spec = _load("hand_retrieval.json")
    pooled = _load("pooled_hand.json")
    idx, q = hand_index(spec)
    np.testing.assert_array_equal(O.pooled_scores(idx, q), np.array(pooled["scores"]))
    for c in pooled["cases"]:
        idx, q = hand_index(spec, c["n_recent"])
        ids, sc, n = O.pooled_retrieve(idx, q, c["n_select"])
        assert ids.tolist() == c["frame_ids"]
        np.testing.assert_array_equal(sc, np.array(c["scores"]))
        assert n == sum(1 for x in c["frame_ids"] if x >= 0)


@pytest.mark.parametrize("seed,Hq,Hk,nr", [(0, 4, 2, 0), (1, 6, 2, 1), (2, 3, 3, 2)])
def test_pooled_matches_brute_and_token_means(seed, Hq, Hk, nr):
    """Against the per-token brute force, and (linearity of the logit) against
    the mean of the unit's token scores over every (layer, head) list."""
    rng = np.random.default_rng(50 + seed)
    L, d, F, T, nq = 2, 8, 6, 5, 3
    keys = [W.bf16_bits(rng.standard_normal((Hk, F * T, d)).astype(np.float32)) for _ in range(L)]
    q = [W.bf16_bits(rng.standard_normal((Hq, nq, d)).astype(np.float32)) for _ in range(L)]
    idx = O.Index(L, Hq, Hk, d, nr)
    idx.append(keys, F, T)
    s = O.pooled_scores(idx, q)
    frames = _brute_frames(keys, F, T, L, Hk)
    qs = [[[q[l][h][j] for j in range(nq)] for h in range(Hq)] for l in range(L)]
    np.testing.assert_allclose(s, brute.pooled_scores(frames, qs, Hk, nr), rtol=1e-12, atol=1e-12)
    lists = O.score_lists(idx, q)
    fr = idx.frame_of_row()[:idx.candidate_rows()]
    mean_tok = np.array([np.mean([lst[fr == t].mean() for lst in lists]) for t in range(F - nr)])
    np.testing.assert_allclose(s, mean_tok, rtol=1e-12, atol=1e-12)
    ids, sc, n = O.pooled_retrieve(idx, q, 4)
    want = sorted(range(F - nr), key=lambda t: (-s[t], t))[:4]
    assert ids[:n].tolist() == want


def test_pooled_invariant_under_token_permutation():
    rng = np.random.default_rng(9)
    L, Hq, Hk, d, F, T = 2, 4, 2, 8, 4, 6
    keys = [W.bf16_bits(rng.standard_normal((Hk, F * T, d)).astype(np.float32)) for _ in range(L)]
    q = [W.bf16_bits(rng.standard_normal((Hq, 2, d)).astype(np.float32)) for _ in range(L)]
    perm = np.concatenate([f * T + rng.permutation(T) for f in range(F)])
    a, b = O.Index(L, Hq, Hk, d), O.Index(L, Hq, Hk, d)
    a.append(keys, F, T)
    b.append([k[:, perm, :] for k in keys], F, T)
    np.testing.assert_allclose(O.pooled_scores(a, q), O.pooled_scores(b, q), rtol=1e-12, atol=1e-12)


def test_pooled_uses_raw_keys_of_compressed_units():
    rng = np.random.default_rng(4)
    L, Hq, Hk, d, F, T = 1, 2, 1, 8, 3, 10
    keys = [W.bf16_bits(rng.standard_normal((Hk, F * T, d)).astype(np.float32))]
    q = [W.bf16_bits(rng.standard_normal((Hq, 1, d)).astype(np.float32))]
    raw, comp = O.Index(L, Hq, Hk, d), O.Index(L, Hq, Hk, d)
    raw.append(keys, F, T)
    comp.append(keys, F, T, (3, 4))
    np.testing.assert_array_equal(O.pooled_scores(raw, q), O.pooled_scores(comp, q))


# ---------------------------------------------------------------------------
# Long-history compression and cluster retrieval
# ---------------------------------------------------------------------------

def _cluster_index(tokens):
    idx = O.Index(1, 1, 1, 2)
    rows = bits(np.array(tokens, dtype=np.float32))[None]        # [H_kv=1][units][2]
    idx.append([rows], len(tokens), 1)
    return idx


@pytest.mark.parametrize("case", [c["name"] for c in _load("clusters_hand.json")["cases"]])
def test_clusters_hand(case):
    spec = _load("clusters_hand.json")
    c = next(c for c in spec["cases"] if c["name"] == case)
    idx = _cluster_index(spec["tokens"])
    cl = O.LongClusters(c["tau"], c["max_clusters"])
    cl.absorb(idx, 6)
    assert idx.first_detail == 6
    assert [[a, b] for a, b in zip(cl.first, cl.last)] == c["members"]
    assert cl.sizes == c["sizes"] and cl.overflow == c["overflow"]
    if "centroids" in c:
        np.testing.assert_allclose(np.array(cl.centroids), np.array(c["centroids"]), atol=5e-6)  # six-digit hand arithmetic
    if "representatives" in c:
        reps = np.array([r[0, 0, 0] for r in cl.rep])
        np.testing.assert_allclose(reps, np.array(c["representatives"]), atol=1e-7)
    for qc in c.get("queries", []):
        q = [bits(np.array([[qc["q"]]], dtype=np.float32))]       # [H_q=1][n_q=1][2]
        np.testing.assert_allclose(O.cluster_scores(idx, cl, q), qc["scores"], atol=5e-6)
        ids, sc, fst, lst, n = O.cluster_retrieve(idx, cl, q, 5)
        assert ids[:n].tolist() == qc["order"] and n == 3
        assert fst[:n].tolist() == [c["members"][i][0] for i in qc["order"]]


def test_clusters_properties_random():
    """Clusters are contiguous runs covering the absorbed units in order; each
    joining unit met tau against the centroid it joined (replayed from scratch);
    representatives are the members' mean rows; absorbing in pieces equals
    absorbing at once; tau below -1 gives one cluster, above 1 one per unit."""
    rng = np.random.default_rng(21)
    L, Hk, d, F, T = 2, 2, 8, 30, 3
    scene = rng.standard_normal((5, Hk, d))           # five scenes of six units each
    keys = []
    for l in range(L):
        base = scene[np.arange(F * T) // (6 * T)].transpose(1, 0, 2)   # [H_kv][F*T][d]
        x = base + rng.standard_normal((Hk, F * T, d)) * 0.3
        keys.append(W.bf16_bits(x.astype(np.float32)))
    mk = lambda: (lambda i: (i.append(keys, F, T), i)[1])(O.Index(L, 4, Hk, d))
    a = mk()
    cl = O.LongClusters(0.8, 100)
    cl.absorb(a, F)
    assert cl.first[0] == 0 and cl.last[-1] == F - 1
    assert all(cl.last[j] + 1 == cl.first[j + 1] for j in range(len(cl.first) - 1))
    assert sum(cl.sizes) == F and 1 < len(cl.sizes) < F
    for j in range(len(cl.first)):
        mem = range(cl.first[j], cl.last[j] + 1)
        rows = [np.stack([O.decode_bf16(a.rows(l)[:, t * T:(t + 1) * T, :]) for l in range(L)]) for t in mem]
        np.testing.assert_allclose(cl.rep[j], np.mean(rows, axis=0), rtol=1e-12, atol=1e-12)
        c = np.array(a.desc[cl.first[j]])
        for t in list(mem)[1:]:
            assert a.desc[t] @ c >= 0.8
            n = t - cl.first[j]
            c = (n * c + a.desc[t]) / (n + 1)
            c = c / np.linalg.norm(c)
        np.testing.assert_allclose(c, cl.centroids[j], rtol=1e-12, atol=1e-12)
    b = mk()
    cl2 = O.LongClusters(0.8, 100)
    for hi in (7, 8, 19, 30):
        cl2.absorb(b, hi)
    assert cl2.sizes == cl.sizes
    np.testing.assert_allclose(np.array(cl2.centroids), np.array(cl.centroids), rtol=1e-12, atol=1e-12)
    one = O.LongClusters(-1.5, 100)
    one.absorb(mk(), F)
    assert one.sizes == [F]
    every = O.LongClusters(1.5, 100)
    every.absorb(mk(), F)
    assert every.sizes == [1] * F
    with pytest.raises(ValueError):
        O.LongClusters(0.8, 100).absorb(mk(), F + 1)


def test_detailed_window_equals_index_of_the_window():
    """Token voting with units folded into clusters equals voting on an index
    that holds only the detailed units (frame ids shifted)."""
    rng = np.random.default_rng(33)
    L, Hq, Hk, d, F, T, f0 = 2, 4, 2, 8, 12, 4, 5
    keys = [W.bf16_bits(rng.standard_normal((Hk, F * T, d)).astype(np.float32)) for _ in range(L)]
    q = [W.bf16_bits(rng.standard_normal((Hq, 2, d)).astype(np.float32)) for _ in range(L)]
    full = O.Index(L, Hq, Hk, d, 2)
    full.append(keys, F, T)
    O.LongClusters(0.5, 10).absorb(full, f0)
    part = O.Index(L, Hq, Hk, d, 2)
    part.append([k[:, f0 * T:, :] for k in keys], F - f0, T)
    a = O.retrieve(full, q, 6, 3)
    b = O.retrieve(part, q, 6, 3)
    assert [x + f0 if x >= 0 else -1 for x in b[0].tolist()] == a[0].tolist()
    assert a[1].tolist() == b[1].tolist() and a[3] == b[3]
    pa = O.pooled_retrieve(full, q, 4)
    pb = O.pooled_retrieve(part, q, 4)
    assert pa[0].tolist() == [x + f0 for x in pb[0].tolist()]


def test_budget_split_hand():
    spec = _load("budget_hand.json")
    sh = spec["shape"]
    assert [O.frame_bytes(r, sh["n_layers"], sh["n_kv_heads"], sh["head_dim"]) for r in spec["rows"]] == \
        spec["frame_bytes"]
    for c in spec["cases"]:
        got = O.budget_split(spec["rows"], c["first_detail"], c["n_recent"], sh["n_layers"], sh["n_kv_heads"],
                             sh["head_dim"], c["budget"])
        assert got == c["frame_hi"], c
