"""GPU parity of evidence assembly (Eq. selected_evidence, deduplication,
temporal order) through the C ABI against the oracle.  Unit ids are integers:
results must be exactly equal."""
import json
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


def frames_index(T, max_frames=None):
    """An index holding T one-token frames (only its frame count matters here)."""
    import paper_2609_02780_amd as P
    idx = P.ShallowIndex(1, 1, 1, 64, max(1, max_frames or T), max(1, max_frames or T))
    if T > 0:
        keys = torch.zeros((1, T, 64), dtype=torch.int16, device="cuda")
        idx.append([keys], T, 1)
    return idx


def run(idxs, sel, n_recent, n_before, n_after, retrieved):
    import paper_2609_02780_amd as P
    fid = torch.from_numpy(np.asarray(sel, dtype=np.int64)).cuda() if retrieved else None
    units, kinds, n_units = P.assemble_evidence(idxs, fid, n_recent, n_before, n_after, retrieved)
    torch.cuda.synchronize()
    u, n = units.cpu().numpy(), n_units.cpu().numpy()
    out = []
    for s in range(len(idxs)):
        assert np.all(u[s, n[s]:] == -1)
        out.append(u[s, :n[s]])
    return out


def test_evidence_hand_fixture():
    with open(os.path.join(GOLDEN, "evidence_hand.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        log("evidence case", c["name"])
        idx = frames_index(c["n_frames"])
        got = run([idx], [c["selected"]], c["n_recent"], c["n_before"], c["n_after"], c["retrieved"])[0]
        assert got.tolist() == c["units"], c["name"]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_evidence_random_batches(seed):
    """Ragged batches (40 streams, so two launches of up to 32) with padding,
    repeats, ids at both ends and every parameter mix, against the oracle."""
    rng = np.random.default_rng(100 + seed)
    S = 40
    Ts = [int(x) for x in rng.integers(0, 300, size=S)]
    Ts[0], Ts[1] = 0, 1
    idxs = [frames_index(T, max_frames=300) for T in Ts]
    for nr, nb, na, retrieved in ((6, 1, 0, True), (2, 1, 0, False), (0, 2, 3, True), (9, 0, 0, True)):
        K = int(rng.integers(1, 65))
        sel = np.full((S, K), -1, dtype=np.int64)
        for s, T in enumerate(Ts):
            if T == 0:
                continue
            n = int(rng.integers(0, K + 1))
            pick = rng.integers(0, T, size=n)
            pick[: min(n, 2)] = [0, T - 1][: min(n, 2)]
            sel[s, :n] = pick
        log("evidence batch", seed, nr, nb, na, retrieved, K)
        got = run(idxs, sel, nr, nb, na, retrieved)
        for s, T in enumerate(Ts):
            want = O.evidence_units(T, sel[s], nr, nb, na, retrieved)
            assert got[s].tolist() == want.tolist(), (s, T)


def test_evidence_after_retrieval_c1():
    """End to end on C1 with the paper's settings (6 recent units, one
    preceding unit): the GPU's selection, assembled on the GPU, equals the
    oracle's assembly of the oracle's selection."""
    import paper_2609_02780_amd as P
    cfg = W.CONFIGS["C1"]
    spec = W.stream_specs(cfg)[0]
    q, keys = W.make_stream(cfg, spec)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()
    idx = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, spec.n_frames,
                         spec.n_frames * cfg.tokens_per_frame, 6)
    idx.append([dev(k) for k in keys], spec.n_frames, cfg.tokens_per_frame)
    r = P.Retriever([idx], cfg.top_k, cfg.n_select)
    ids, _, _, _ = r([[dev(x) for x in q]])
    units, kinds, n_units = P.assemble_evidence([idx], ids, 6, 1, 0, True)
    torch.cuda.synchronize()
    oi = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, 6)
    oi.append(keys, spec.n_frames, cfg.tokens_per_frame)
    sel = O.retrieve(oi, q, cfg.top_k, cfg.n_select)[0]
    want = O.evidence_units(spec.n_frames, sel, 6, 1, 0, True)
    n = int(n_units.cpu()[0])
    assert units.cpu().numpy()[0, :n].tolist() == want.tolist()


def _scene_frames_index(groups, T, tau, n_leave):
    """T one-token frames whose keys point along basis vector groups[f] (64-d),
    the first n_leave folded into long-term clusters with threshold tau, on the
    GPU and in the oracle."""
    import paper_2609_02780_amd as P
    x = np.zeros((1, T, 64), np.float32)
    for f in range(T):
        x[0, f, groups[f]] = 1.0
    bits = W.bf16_bits(x)
    idx = P.ShallowIndex(1, 1, 1, 64, T, T)
    idx.append([torch.from_numpy(bits.view(np.int16)).cuda()], T, 1)
    cl = P.LongClusters(idx, 1, 16, tau)
    cl.absorb(n_leave, n_leave)
    o = O.Index(1, 1, 1, 64)
    o.append([bits], T, 1)
    ocl = O.LongClusters(tau, 16)
    ocl.absorb(o, n_leave)
    return idx, cl, ocl


def test_evidence_with_clusters_hand_fixture():
    """The hand-worked cases of detailed evidence united with retrieved
    clusters: 20 frames, frames 0..7 folded into three clusters (0..2, 3..5,
    6..7: three directions, threshold 0.5), ids and kinds exactly."""
    with open(os.path.join(GOLDEN, "evidence_hand.json")) as f:
        cases = json.load(f)["cluster_cases"]
    groups = [0, 0, 0, 1, 1, 1, 2, 2] + [3 + (f % 5) for f in range(12)]
    idx, cl, ocl = _scene_frames_index(groups, 20, 0.5, 8)
    ex = cl.export()
    assert ocl.first == [0, 3, 6] and ocl.last == [2, 5, 7]
    assert ex["span"].tolist() == [[0, 2], [3, 5], [6, 7]]
    import paper_2609_02780_amd as P
    for c in cases:
        assert c["cluster_first"] == ocl.first and c["first_detail"] == 8
        fid = torch.tensor([c["selected"]], dtype=torch.int64, device="cuda")
        cid = torch.tensor([c["selected_clusters"]], dtype=torch.int64, device="cuda")
        units, kinds, n_units = P.assemble_evidence([idx], fid, c["n_recent"], c["n_before"], c["n_after"],
                                                    c["retrieved"], clusters=[cl], cluster_ids=cid)
        torch.cuda.synchronize()
        n = int(n_units.cpu()[0])
        u, k = units.cpu().numpy()[0], kinds.cpu().numpy()[0]
        log("evidence with clusters", c["name"], u[:n].tolist(), k[:n].tolist())
        assert u[:n].tolist() == c["ids"] and k[:n].tolist() == c["kinds"], c["name"]
        assert np.all(u[n:] == -1) and np.all(k[n:] == -1)


def test_evidence_with_clusters_random_batches():
    """Ragged batches with and without long-term clusters per stream (some
    entries None), random detailed windows, padded and invalid cluster ids,
    against the oracle's assembly with the oracle's own cluster spans."""
    import paper_2609_02780_amd as P
    rng = np.random.default_rng(77)
    S = 12
    idxs, cls, ocls, Ts, fds = [], [], [], [], []
    for s in range(S):
        T = int(rng.integers(5, 80))
        fd = int(rng.integers(0, T - 2)) if s % 3 else 0
        groups = [int(g) for g in np.cumsum(rng.random(T) < 0.3)]
        groups = [g % 60 for g in groups]
        idx, cl, ocl = _scene_frames_index(groups, T, 0.5, fd)
        idxs.append(idx)
        cls.append(cl if s % 4 != 3 else None)
        ocls.append(ocl if s % 4 != 3 else None)
        Ts.append(T)
        fds.append(fd)
    for nr, nb, na, retrieved, K, KC in ((6, 1, 0, True, 8, 5), (2, 1, 0, False, 8, 5), (0, 2, 1, True, 3, 16)):
        sel = np.full((S, K), -1, dtype=np.int64)
        csel = np.full((S, KC), -1, dtype=np.int64)
        for s in range(S):
            n = int(rng.integers(0, K + 1))
            sel[s, :n] = rng.integers(fds[s], Ts[s], size=n)
            nc = len(ocls[s].first) if ocls[s] is not None else 0
            m = int(rng.integers(0, KC + 1))
            csel[s, :m] = rng.integers(-1, nc + 2, size=m)
        units, kinds, n_units = P.assemble_evidence(
            idxs, torch.from_numpy(sel).cuda(), nr, nb, na, retrieved, clusters=cls,
            cluster_ids=torch.from_numpy(csel).cuda())
        torch.cuda.synchronize()
        u, k, n = units.cpu().numpy(), kinds.cpu().numpy(), n_units.cpu().numpy()
        for s in range(S):
            firsts = ocls[s].first if ocls[s] is not None else []
            wi, wk = O.evidence_items(Ts[s], sel[s], nr, nb, na, retrieved, fds[s], firsts,
                                      csel[s] if ocls[s] is not None else [])
            assert u[s, :n[s]].tolist() == wi.tolist() and k[s, :n[s]].tolist() == wk.tolist(), s
    log("evidence with clusters: random batches ok")
