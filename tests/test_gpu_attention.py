"""GPU parity of the attention-probability reading (score_mode 1: per
(layer, head) softmax over the candidate rows, averaged over heads in head mode
1, the attention mass a sum of probabilities) through the C ABI against the
oracle: the hand-worked cases where the two readings disagree, the tiny and
paper-settings workloads staged in full, both fallback paths, ragged batches."""
import json
import math
import os
import sys

import numpy as np
import pytest

import workloads as W
from oracle import oracle as O

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


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


def pair(cfg, keys, n_recent=0):
    import paper_2609_02780_amd as P
    F, T = cfg.n_frames, cfg.tokens_per_frame
    g = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, F, F * T, n_recent)
    g.append([dev(k) for k in keys], F, T)
    o = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, n_recent)
    o.append(keys, F, T)
    return g, o


def run(gs, qs, top_k, n_select, pool_mult, head_mode, score_mode=1):
    import paper_2609_02780_amd as P
    r = P.Retriever(gs, top_k, n_select, pool_mult, head_mode, score_mode)
    return r.debug([[dev(x) for x in q] for q in qs])


def _closed(expr, defs):
    env = {"exp": math.exp, "sqrt": math.sqrt}
    for k, e in defs.items():
        env[k] = eval(e, {"__builtins__": {}}, dict(env))
    return float(eval(expr, {"__builtins__": {}}, env))


def test_hand_attention_cases():
    """The hand-worked index (d = 4 in the fixture) padded to d = 64 with zeros,
    the queries scaled by 4 so that q.k / sqrt(64) equals the fixture's
    q.k / sqrt(4): every list, vote, pool and frame id exactly as worked out by
    hand, in both readings; values and masses against the closed forms."""
    import paper_2609_02780_amd as P
    with open(os.path.join(GOLDEN, "hand_attention.json")) as f:
        spec = json.load(f)
    rows = np.zeros((1, 6, 64), np.float32)
    rows[0, :, :4] = np.array(spec["rows"], np.float32)
    q = np.zeros((2, 1, 64), np.float32)
    q[:, :, :4] = 4.0 * np.array(spec["queries"], np.float32)
    keys, qb = [W.bf16_bits(rows)], [W.bf16_bits(q)]
    cf = lambda e: _closed(e, spec["defs"])
    for c in spec["cases"]:
        g = P.ShallowIndex(1, 2, 1, 64, 3, 6, c["n_recent"])
        g.append([dev(keys[0])], 3, 2)
        out = run([g], [qb], c["top_k"], c["n_select"], c["pool_mult"], c["head_mode"], c["score_mode"])
        k = len(c["topk"][0])
        got_lists = [out["topk_pos"][0, j, :k].tolist() for j in range(len(c["topk"]))]
        log(c["name"], got_lists, out["frame_ids"][0].tolist(), out["list_stats"][0].tolist())
        assert got_lists == c["topk"], c["name"]
        assert out["vote_hist"][0, :3].tolist() == c["votes"], c["name"]
        np.testing.assert_allclose(out["mass_hist"][0, :3], [cf(e) for e in c["mass"]], rtol=2e-5, atol=1e-6)
        pn = int(out["pool_n"][0])
        assert out["pool"][0, :pn].tolist() == c["pool"], c["name"]
        n = int(out["n_out"][0])
        assert n == c["n_out"] and out["frame_ids"][0, :n].tolist() == c["frame_ids"][:n], c["name"]
        assert out["votes"][0, :n].tolist() == c["sel_votes"][:n]
        np.testing.assert_allclose(out["mass"][0, :n], [cf(e) for e in c["sel_mass"][:n]], rtol=2e-5, atol=1e-6)
        if "values" in c:
            for j, (lst, vals) in enumerate(zip(c["topk"], c["values"])):
                want = [cf(vals[p]) for p in lst]
                np.testing.assert_allclose(out["topk_score"][0, j, :k], want, rtol=2e-5, atol=1e-7)


@pytest.mark.parametrize("head_mode", [0, 1])
def test_c1_probabilities_staged(head_mode):
    from parity import staged_check
    cfg = W.CONFIGS["C1"]
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec)
    g, o = pair(cfg, keys)
    k = cfg.top_k if head_mode == 0 else 64
    out = run([g], [q], k, cfg.n_select, 4, head_mode)
    rep = staged_check(o, q, out, 0, k, cfg.n_select, 4, head_mode=head_mode, score_mode=1)
    log("C1 probabilities, head mode", head_mode, rep, "fallbacks", out["list_stats"][0, :, 1].tolist())
    assert out["frame_ids"][0, 0] in set(spec.planted)
    again = run([g], [q], k, cfg.n_select, 4, head_mode)
    for key in ("frame_ids", "votes", "mass", "topk_pos", "topk_score", "mass_hist"):
        assert np.array_equal(out[key].view(np.uint8), again[key].view(np.uint8)), key


def test_sampled_lists_probabilities_staged():
    """Lists long enough to be sampled (2 layers x 2 KV heads, 1,500 frames x
    16 tokens): the head-mode-1 pass with sample estimates of each head's
    normaliser and the proof of its selection, and head mode 0's sums below
    the cut-off, staged against the oracle."""
    from parity import staged_check
    cfg = W.Config("prob-mid", 2, 8, 2, 128, 16, 1, 64, 8, n_frames=1500, n_planted=4, pool_mult=4)
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec)
    g, o = pair(cfg, keys)
    for head_mode in (0, 1):
        out = run([g], [q], cfg.top_k, cfg.n_select, 4, head_mode)
        rep = staged_check(o, q, out, 0, cfg.top_k, cfg.n_select, 4, head_mode=head_mode, score_mode=1)
        log("sampled lists, head mode", head_mode, rep, "candidates", out["list_stats"][0, :, 0].tolist(),
            "fallbacks", out["list_stats"][0, :, 1].tolist())
        assert np.all(out["list_stats"][0, :, 1] == 0)
        assert out["frame_ids"][0, 0] in set(spec.planted)


def test_probability_fallbacks():
    """Zero queries make every logit 0, so every row ties and the candidate
    buffer overflows (fallback 1, both head modes): each list keeps rows
    0..k-1 with probability 1/n each.  Then rows on the sample lattice dominate
    one head, so the sample overestimates that head's normaliser and the
    head-mode-1 selection cannot be proven from the candidates (or there are
    too few): the exact pass must still match the oracle."""
    import paper_2609_02780_amd as P
    from parity import staged_check
    cfg = W.Config("prob-fb", 1, 2, 1, 64, 16, 1, 40, 3, n_frames=512, n_planted=0)
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec)
    g, o = pair(cfg, keys)
    zq = [np.zeros_like(x) for x in q]
    for head_mode in (0, 1):
        out = run([g], [zq], cfg.top_k, cfg.n_select, 4, head_mode)
        assert np.all(out["list_stats"][0, :, 1] == 1)
        for j in range(out["topk_pos"].shape[1]):
            np.testing.assert_array_equal(out["topk_pos"][0, j, :40], np.arange(40))
            np.testing.assert_allclose(out["topk_score"][0, j, :40], 1.0 / 8192, rtol=1e-5)
        rep = staged_check(o, zq, out, 0, cfg.top_k, cfg.n_select, 4, head_mode=head_mode, score_mode=1)
        assert rep["end_to_end_equal"]
    # sample-lattice rows dominate head 0
    L, Hq, Hk, d, T, F, k = 1, 2, 1, 64, 100, 1000, 64
    n = F * T
    m, r, cap, E = P.sample_plan(n, k)
    step = (n << 32) // m
    rows = ((np.arange(m, dtype=np.uint64) * np.uint64(step) + np.uint64(step >> 1)) >> np.uint64(32)).astype(np.int64)
    rng = np.random.default_rng(21)
    x = rng.standard_normal((1, n, d)).astype(np.float32) * 0.5
    x[0, rows, 0] = 6.0 + rng.random(m).astype(np.float32)
    qv = np.zeros((Hq, 1, d), np.float32)
    qv[0, 0, 0] = 8.0
    qv[1, 0, 1:] = rng.standard_normal(d - 1).astype(np.float32)
    keys2, q2 = [W.bf16_bits(x)], [W.bf16_bits(qv)]
    cfg2 = W.Config("prob-lattice", L, Hq, Hk, d, T, 1, k, 4, n_frames=F, n_planted=0)
    g2, o2 = pair(cfg2, keys2)
    out = run([g2], [q2], k, 4, 4, 1)
    log("lattice case: candidates", out["list_stats"][0, :, 0].tolist(), "fallback", out["list_stats"][0, :, 1].tolist())
    assert out["list_stats"][0, 0, 1] in (1, 2)
    rep = staged_check(o2, q2, out, 0, k, 4, 4, head_mode=1, score_mode=1)
    log("lattice case", rep)


def test_probability_ragged_batch():
    """Five streams of different lengths and recent windows in one call, both
    head modes, each staged on its own."""
    from parity import staged_check
    gs, os_, qs = [], [], []
    for s, (F, nr) in enumerate([(30, 0), (240, 2), (90, 5), (400, 0), (17, 1)]):
        cfg = W.Config("prob-rag", 2, 8, 2, 64, 12, 1 + s, 24, 4, n_frames=F, n_planted=2)
        spec = W.stream_specs(cfg)[0]
        q, keys = W.make_stream(cfg, spec, seed=70 + s)
        g, o = pair(cfg, keys, nr)
        gs.append(g)
        os_.append(o)
        qs.append(q)
    for head_mode in (0, 1):
        out = run(gs, qs, 24, 4, 4, head_mode)
        for s in range(5):
            log("ragged batch with probabilities, head mode", head_mode, "stream", s, "fallbacks",
                out["list_stats"][s, :, 1].tolist())
            staged_check(os_[s], qs[s], out, s, 24, 4, 4, head_mode=head_mode, score_mode=1)
    log("ragged batch with probabilities: ok")
