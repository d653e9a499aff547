"""GPU parity over seeded random small batches: each case draws a head shape
(layers, KV heads, group size, head dimension), a ragged batch of one to three
streams (frames, tokens per frame, query tokens, recent window each their
own), the retrieval parameters (k, frame budget, pool multiplier) and both
readings of the scores, and every stream is staged against the oracle."""
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


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


def _case(rng, i):
    L = int(rng.choice([1, 2, 3]))
    Hk = int(rng.choice([1, 2, 4]))
    G = int(rng.choice([1, 2, 3, 4, 7, 8]))
    d = int(rng.choice([64, 128]))
    streams = []
    for s in range(int(rng.integers(1, 4))):
        F = int(rng.integers(3, 250))
        streams.append(dict(F=F, T=int(rng.integers(2, 40)), nq=int(rng.integers(1, 12)),
                            recent=int(rng.integers(0, min(4, F))), seed=1000 * i + s))
    return dict(L=L, Hk=Hk, G=G, d=d, streams=streams, top_k=int(rng.integers(1, 200)),
                n_select=int(rng.integers(1, 12)), pool_mult=int(rng.choice([1, 2, 4])),
                head_mode=int(rng.integers(0, 2)), score_mode=int(rng.integers(0, 2)))


@pytest.mark.parametrize("i", range(24))
def test_random_small_batch_staged(i):
    import paper_2609_02780_amd as P
    from parity import staged_check
    c = _case(np.random.default_rng([2609, i]), i)
    log("case", i, {k: v for k, v in c.items() if k != "streams"}, "streams",
        [(x["F"], x["T"], x["nq"], x["recent"]) for x in c["streams"]])
    gs, os_, qs = [], [], []
    for x in c["streams"]:
        cfg = W.Config(f"rand{i}", c["L"], c["Hk"] * c["G"], c["Hk"], c["d"], x["T"], x["nq"], c["top_k"],
                       c["n_select"], n_frames=x["F"], n_planted=min(2, x["F"] // 4))
        spec = W.stream_specs(cfg)[0]
        q, keys = W.make_stream(cfg, spec, seed=x["seed"])
        g = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, x["F"], x["F"] * x["T"],
                           x["recent"])
        g.append([_dev(k) for k in keys], x["F"], x["T"])
        o = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, x["recent"])
        o.append(keys, x["F"], x["T"])
        gs.append(g)
        os_.append(o)
        qs.append(q)
    r = P.Retriever(gs, c["top_k"], c["n_select"], c["pool_mult"], c["head_mode"], c["score_mode"])
    out = r.debug([[_dev(a) for a in q] for q in qs])
    for s in range(len(gs)):
        rep = staged_check(os_[s], qs[s], out, s, c["top_k"], c["n_select"], c["pool_mult"],
                           head_mode=c["head_mode"], score_mode=c["score_mode"])
        log("  stream", s, "fallbacks", out["list_stats"][s, :, 1].tolist(), rep)


def _medium_case(rng, i):
    G = int(rng.choice([1, 2, 4, 7, 8, 16]))
    Hk = int(rng.choice([1, 2] if G == 16 else [1, 2, 4]))
    c = dict(L=int(rng.choice([1, 2])), Hk=Hk, G=G, d=int(rng.choice([64, 128])), streams=[],
             top_k=int(rng.integers(16, 1025)), n_select=int(rng.integers(1, 33)), pool_mult=int(rng.choice([1, 2, 4])),
             head_mode=int(rng.integers(0, 2)), score_mode=int(rng.integers(0, 2)))
    for s in range(int(rng.integers(1, 5))):
        c["streams"].append(dict(F=int(rng.integers(300, 3001)), T=int(rng.integers(2, 13)),
                                 nq=int(rng.integers(1, 17)), recent=int(rng.integers(0, 6)), seed=50000 + 100 * i + s))
    return c


@pytest.mark.parametrize("i", range(8))
def test_random_medium_batch_staged(i):
    """Longer streams (300 to 3,000 frames, up to four of them), k up to 1,024
    (candidate lists beyond the 4,096 slots the selection holds in registers),
    frame budgets up to 32 and groups up to 16 query heads."""
    import paper_2609_02780_amd as P
    from parity import staged_check
    c = _medium_case(np.random.default_rng([2609, 7, i]), i)
    log("medium case", i, {k: v for k, v in c.items() if k != "streams"}, "streams",
        [(x["F"], x["T"], x["nq"], x["recent"]) for x in c["streams"]])
    gs, os_, qs = [], [], []
    for x in c["streams"]:
        cfg = W.Config(f"randm{i}", c["L"], c["Hk"] * c["G"], c["Hk"], c["d"], x["T"], x["nq"], c["top_k"],
                       c["n_select"], n_frames=x["F"], n_planted=4)
        spec = W.stream_specs(cfg)[0]
        q, keys = W.make_stream(cfg, spec, seed=x["seed"])
        g = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, x["F"], x["F"] * x["T"],
                           x["recent"])
        g.append([_dev(k) for k in keys], x["F"], x["T"])
        o = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, x["recent"])
        o.append(keys, x["F"], x["T"])
        gs.append(g)
        os_.append(o)
        qs.append(q)
    r = P.Retriever(gs, c["top_k"], c["n_select"], c["pool_mult"], c["head_mode"], c["score_mode"])
    out = r.debug([[_dev(a) for a in q] for q in qs])
    for s in range(len(gs)):
        rep = staged_check(os_[s], qs[s], out, s, c["top_k"], c["n_select"], c["pool_mult"],
                           head_mode=c["head_mode"], score_mode=c["score_mode"])
        st = out["list_stats"][s]
        log("  stream", s, "candidates", int(st[:, 0].min()), "..", int(st[:, 0].max()),
            "fallbacks", np.bincount(st[:, 1], minlength=3).tolist(), rep)


@pytest.mark.parametrize("i", range(8))
def test_random_compressed_batch_staged(i):
    """Ragged batches that mix streams appended with per-frame k-means (random
    centroid counts and rounds) and plain streams: retrieval staged against the
    oracle over the stored centroids, with descriptors from the raw keys."""
    import paper_2609_02780_amd as P
    from parity import staged_check
    rng = np.random.default_rng([2609, 11, i])
    c = _case(rng, 2000 + i)
    comp = [bool(rng.integers(0, 2)) for _ in c["streams"]]
    log("compressed case", i, {k: v for k, v in c.items() if k != "streams"}, "streams",
        [(x["F"], x["T"], x["nq"], x["recent"], cp) for x, cp in zip(c["streams"], comp)])
    gs, os_, qs = [], [], []
    for x, cp in zip(c["streams"], comp):
        F, T = x["F"], x["T"]
        cfg = W.Config(f"randc{i}", c["L"], c["Hk"] * c["G"], c["Hk"], c["d"], T, x["nq"], c["top_k"],
                       c["n_select"], n_frames=F, n_planted=min(2, F // 4))
        spec = W.stream_specs(cfg)[0]
        q, keys = W.make_stream(cfg, spec, seed=x["seed"])
        o = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, x["recent"])
        if cp:
            nc = int(rng.integers(1, T + 1))
            compress = (nc, int(rng.integers(1, 6)))
            g = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, F, F * nc, x["recent"])
            g.append([_dev(k) for k in keys], F, T, compress)
            ex = g.export()
            desc = [O.descriptor(O.decode_bf16(keys[-1][:, f * T:(f + 1) * T, :])) for f in range(F)]
            o.append_stored([ex["rows"][l] for l in range(cfg.n_layers)], [nc] * F, desc)
        else:
            g = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, F, F * T, x["recent"])
            g.append([_dev(k) for k in keys], F, T)
            o.append(keys, F, T)
        gs.append(g)
        os_.append(o)
        qs.append(q)
    r = P.Retriever(gs, c["top_k"], c["n_select"], c["pool_mult"], c["head_mode"], c["score_mode"])
    out = r.debug([[_dev(a) for a in q] for q in qs])
    for s in range(len(gs)):
        rep = staged_check(os_[s], qs[s], out, s, c["top_k"], c["n_select"], c["pool_mult"],
                           head_mode=c["head_mode"], score_mode=c["score_mode"])
        log("  stream", s, "fallbacks", out["list_stats"][s, :, 1].tolist(), rep)


@pytest.mark.parametrize("i", range(8))
def test_random_pooled_ranker(i):
    """The pooled Q-K ranker over seeded random ragged batches (the head shapes
    and per-stream lengths, tokens, query tokens and recent windows of the
    cases above; K from 1 to 64), each stream checked as in
    tests/test_gpu_pooled.py."""
    import paper_2609_02780_amd as P
    from test_gpu_pooled import check
    rng = np.random.default_rng([2609, 13, i])
    c = _case(rng, 3000 + i)
    K = int(rng.integers(1, 65))
    log("pooled case", i, {k: v for k, v in c.items() if k != "streams"}, "K", K, "streams",
        [(x["F"], x["T"], x["nq"], x["recent"]) for x in c["streams"]])
    gs, os_, qs = [], [], []
    for x in c["streams"]:
        cfg = W.Config(f"randp{i}", c["L"], c["Hk"] * c["G"], c["Hk"], c["d"], x["T"], x["nq"], c["top_k"],
                       c["n_select"], n_frames=x["F"], n_planted=min(2, x["F"] // 4))
        spec = W.stream_specs(cfg)[0]
        q, keys = W.make_stream(cfg, spec, seed=x["seed"])
        g = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, x["F"], x["F"] * x["T"],
                           x["recent"])
        g.append([_dev(k) for k in keys], x["F"], x["T"])
        o = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, x["recent"])
        o.append(keys, x["F"], x["T"])
        gs.append(g)
        os_.append(o)
        qs.append(q)
    r = P.PooledRanker(gs, K)
    ids, sc, n = r([[_dev(a) for a in q] for q in qs])
    torch.cuda.synchronize()
    ids, sc, n = ids.cpu().numpy(), sc.cpu().numpy(), n.cpu().numpy()
    for s in range(len(gs)):
        near = check(os_[s], qs[s], ids[s], sc[s], int(n[s]), K)
        log("  stream", s, "near ties", near)


@pytest.mark.parametrize("head_mode,score_mode", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_repeat_bitwise_equal_all_modes(head_mode, score_mode):
    """Three calls on the same inputs return bitwise-identical outputs in both
    head modes and both readings: a two-layer, 2,000-frame stream (392,000 rows
    per (layer, KV head), hundreds of streaming blocks), where the integer
    atomics of the candidate counts, the sums below the cut-off and the
    per-frame votes and mass land in a different order on every call."""
    import paper_2609_02780_amd as P
    F, T = 2000, 196
    cfg = W.Config("repeat", 2, 28, 4, 128, T, 8, 256, 16, n_frames=F, n_planted=8)
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec, seed=77)
    g = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, F, F * T, 0)
    g.append([_dev(k) for k in keys], F, T)
    r = P.Retriever([g], cfg.top_k, cfg.n_select, 4, head_mode, score_mode)
    qd = [[_dev(a) for a in q]]
    outs = [r.debug(qd) for _ in range(3)]
    for o in outs[1:]:
        assert set(o) == set(outs[0])
        for k in outs[0]:
            np.testing.assert_array_equal(np.asarray(outs[0][k]), np.asarray(o[k]), err_msg=k)
    log("modes", head_mode, score_mode, "fallbacks", np.bincount(outs[0]["list_stats"][0, :, 1], minlength=3).tolist())
