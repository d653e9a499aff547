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
    units, n_units = P.assemble_evidence(idxs, fid, n_recent, n_before, n_after, retrieved)
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
    units, n_units = P.assemble_evidence([idx], ids, 6, 1, 0, True)
    torch.cuda.synchronize()
    oi = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, 6)
    oi.append(keys, spec.n_frames, cfg.tokens_per_frame)
    sel = O.retrieve(oi, q, cfg.top_k, cfg.n_select)[0]
    want = O.evidence_units(spec.n_frames, sel, 6, 1, 0, True)
    n = int(n_units.cpu()[0])
    assert units.cpu().numpy()[0, :n].tolist() == want.tolist()
