"""Host-side tests of the C ABI: the library loads, exports every declared
symbol, and rejects invalid calls before touching the device.  No GPU: every
call here fails validation (or is a pure host query) and enqueues nothing."""
import ctypes as C
import math
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "shallowstream.h")


@pytest.fixture(scope="module")
def L():
    from paper_2609_02780_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2609_02780_amd.build import build_library
        build_library()
    return _lib


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ss_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert len(names) >= 15
    lib = L.lib()
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing
    assert set(names) == set(L._SIGS), "binding signatures and header disagree"


def desc(L, **kw):
    d = dict(n_layers=4, n_q_heads=28, n_kv_heads=4, head_dim=128, max_frames=100, max_rows=19600, n_recent=0)
    d.update(kw)
    return L.IndexDesc(**d)


FAKE = 0x7F0000000000     # 256-byte aligned stand-in address, never dereferenced here


def test_required_bytes_and_layout(L):
    lib = L.lib()
    d = desc(L)
    # one (layer, KV head) of keys must stay below 2 GiB: 2^23 - 1 rows at d = 128
    assert lib.ss_index_required_bytes(C.byref(desc(L, max_rows=2 ** 23 - 1))) > 0
    n = lib.ss_index_required_bytes(C.byref(d))
    keys = 4 * 4 * 19600 * 128 * 2
    counts = 4 * 4 * 19600 * 4
    assert n >= keys + counts + 100 * 512 * 4 + 101 * 4
    assert n % 256 == 0
    for bad in (dict(head_dim=96), dict(n_q_heads=27), dict(n_q_heads=68, n_kv_heads=4),
                dict(max_rows=0), dict(max_frames=0), dict(n_layers=0), dict(n_layers=33),
                dict(n_kv_heads=16, n_q_heads=16), dict(n_recent=-1), dict(max_rows=2 ** 31),
                dict(max_rows=2 ** 23)):
        assert lib.ss_index_required_bytes(C.byref(desc(L, **bad))) == 0, bad


def create(L, **kw):
    lib = L.lib()
    d = desc(L, **kw)
    h = C.c_void_p()
    st = lib.ss_index_create(C.byref(d), FAKE, lib.ss_index_required_bytes(C.byref(d)), C.byref(h))
    assert st == 0, lib.ss_last_error()
    return h


def test_create_errors(L):
    lib = L.lib()
    d = desc(L)
    n = lib.ss_index_required_bytes(C.byref(d))
    h = C.c_void_p()
    assert lib.ss_index_create(C.byref(d), None, n, C.byref(h)) == L.SS_ERR_INVALID_ARGUMENT
    assert lib.ss_index_create(C.byref(d), FAKE + 8, n, C.byref(h)) == L.SS_ERR_INVALID_ARGUMENT
    assert b"aligned" in lib.ss_last_error()
    assert lib.ss_index_create(C.byref(d), FAKE, n - 1, C.byref(h)) == L.SS_ERR_CAPACITY
    bad = desc(L, head_dim=80)
    assert lib.ss_index_create(C.byref(bad), FAKE, n, C.byref(h)) == L.SS_ERR_UNSUPPORTED
    assert lib.ss_index_create(C.byref(d), FAKE, n, None) == L.SS_ERR_INVALID_ARGUMENT


def test_append_validation_leaves_index_unchanged(L):
    lib = L.lib()
    h = create(L, max_frames=4, max_rows=4 * 196)
    ptrs = L.ptr_array([FAKE] * 4)
    first = C.c_int64(-5)
    # too many frames / rows
    assert lib.ss_index_append(h, ptrs, 5, 196, None, None, C.byref(first)) == L.SS_ERR_CAPACITY
    assert lib.ss_index_append(h, ptrs, 4, 197, None, None, C.byref(first)) == L.SS_ERR_CAPACITY
    # misaligned and missing pointers
    bad = L.ptr_array([FAKE, FAKE + 2, FAKE, FAKE])
    assert lib.ss_index_append(h, bad, 1, 196, None, None, C.byref(first)) == L.SS_ERR_INVALID_ARGUMENT
    assert b"layer_keys[1]" in lib.ss_last_error()
    nul = L.ptr_array([FAKE, FAKE, None, FAKE])
    assert lib.ss_index_append(h, nul, 1, 196, None, None, C.byref(first)) == L.SS_ERR_INVALID_ARGUMENT
    assert lib.ss_index_append(h, ptrs, 0, 196, None, None, C.byref(first)) == L.SS_ERR_INVALID_ARGUMENT
    # compression limits
    comp = L.Compress(65, 10)
    assert lib.ss_index_append(h, ptrs, 1, 196, C.byref(comp), None, C.byref(first)) == L.SS_ERR_UNSUPPORTED
    comp = L.Compress(32, 101)
    assert lib.ss_index_append(h, ptrs, 1, 196, C.byref(comp), None, C.byref(first)) == L.SS_ERR_INVALID_ARGUMENT
    comp = L.Compress(32, 10)
    assert lib.ss_index_append(h, ptrs, 1, 300, C.byref(comp), None, C.byref(first)) == L.SS_ERR_UNSUPPORTED
    f, r = C.c_int64(-1), C.c_int64(-1)
    assert lib.ss_index_info(h, C.byref(f), C.byref(r)) == 0
    assert (f.value, r.value) == (0, 0) and first.value == -5
    assert lib.ss_index_destroy(h) == 0


def test_retrieve_validation(L):
    lib = L.lib()
    h1 = create(L)
    h2 = create(L, n_q_heads=16, n_kv_heads=2)
    idx = L.ptr_array([h1.value])
    nq = (C.c_int32 * 1)(32)
    prm = L.RetrieveParams(256, 16, 4, 0)
    ws = lib.ss_retrieve_workspace_bytes(idx, 1, nq, C.byref(prm))
    assert ws > 0 and ws % 256 == 0
    q = L.ptr_array([FAKE] * 4)
    outs = [FAKE] * 4

    def call(idx_=idx, n=1, q_=q, nq_=nq, prm_=prm, w=FAKE, wb=ws):
        return lib.ss_retrieve(idx_, n, q_, nq_, C.byref(prm_), w, wb, None, *outs)

    assert call(w=None) == L.SS_ERR_WORKSPACE
    assert call(wb=ws - 1) == L.SS_ERR_WORKSPACE
    assert call(w=FAKE + 64) == L.SS_ERR_WORKSPACE
    assert call(prm_=L.RetrieveParams(0, 16, 4, 0)) == L.SS_ERR_UNSUPPORTED
    assert call(prm_=L.RetrieveParams(4096, 16, 4, 0)) == L.SS_ERR_UNSUPPORTED
    assert call(prm_=L.RetrieveParams(256, 0, 4, 0)) == L.SS_ERR_UNSUPPORTED
    assert call(prm_=L.RetrieveParams(256, 16, 0, 0)) == L.SS_ERR_INVALID_ARGUMENT
    assert call(prm_=L.RetrieveParams(256, 64, 8, 0)) == L.SS_ERR_UNSUPPORTED
    assert call(prm_=L.RetrieveParams(256, 16, 4, 2)) == L.SS_ERR_INVALID_ARGUMENT
    assert call(prm_=L.RetrieveParams(256, 16, 4, 0, 2)) == L.SS_ERR_INVALID_ARGUMENT   # score_mode
    assert b"score_mode" in lib.ss_last_error()
    # head mode 1 with probabilities keeps every KV head's B tiles in registers
    h8 = create(L, n_q_heads=32, n_kv_heads=8)
    idx8 = L.ptr_array([h8.value])
    assert lib.ss_retrieve(idx8, 1, q, nq, C.byref(L.RetrieveParams(256, 16, 4, 1, 1)), FAKE, ws, None,
                           *outs) == L.SS_ERR_UNSUPPORTED
    assert lib.ss_retrieve_workspace_bytes(idx8, 1, nq, C.byref(L.RetrieveParams(256, 16, 4, 1, 0))) > 0
    assert lib.ss_retrieve_workspace_bytes(idx, 1, nq, C.byref(L.RetrieveParams(256, 16, 4, 1, 1))) > 0
    lib.ss_index_destroy(h8)
    assert call(nq_=(C.c_int32 * 1)(0)) == L.SS_ERR_INVALID_ARGUMENT
    assert call(q_=L.ptr_array([FAKE, FAKE, FAKE + 4, FAKE])) == L.SS_ERR_INVALID_ARGUMENT
    assert call(n=0) == L.SS_ERR_INVALID_ARGUMENT
    both = L.ptr_array([h1.value, h2.value])
    nq2 = (C.c_int32 * 2)(32, 32)
    assert lib.ss_retrieve_workspace_bytes(both, 2, nq2, C.byref(prm)) == 0
    assert b"shape" in lib.ss_last_error()
    assert lib.ss_retrieve(idx, 1, q, nq, C.byref(prm), FAKE, ws, None, None, FAKE, FAKE, FAKE) == \
        L.SS_ERR_INVALID_ARGUMENT
    for h in (h1, h2):
        lib.ss_index_destroy(h)


def test_debug_scores_and_misc_validation(L):
    lib = L.lib()
    h = create(L)
    q = L.ptr_array([FAKE] * 4)
    wsb = lib.ss_debug_scores_workspace_bytes(h)
    assert wsb == 4 * 4 * 2 * 4 * 64 * 16
    # no rows stored yet: any non-empty range is out of bounds
    assert lib.ss_debug_scores(h, q, 8, 0, 0, 0, 0, 1, FAKE, FAKE, wsb, None) == L.SS_ERR_INVALID_ARGUMENT
    assert lib.ss_debug_scores(h, q, 8, 4, 0, 0, 0, 0, FAKE, FAKE, wsb, None) == L.SS_ERR_INVALID_ARGUMENT
    assert lib.ss_debug_scores(h, q, 8, 0, 28, 0, 0, 0, FAKE, FAKE, wsb, None) == L.SS_ERR_INVALID_ARGUMENT
    assert lib.ss_debug_scores(h, q, 8, 0, 0, 0, 0, 0, FAKE, FAKE, wsb - 1, None) == L.SS_ERR_WORKSPACE
    assert lib.ss_set_profile_events(FAKE, None) == L.SS_ERR_INVALID_ARGUMENT
    assert lib.ss_set_profile_events(None, None) == 0
    assert lib.ss_status_string(0) == b"ok" and lib.ss_status_string(4) == b"workspace too small"
    assert lib.ss_version() >= 1
    assert lib.ss_index_destroy(None) == L.SS_ERR_INVALID_ARGUMENT
    lib.ss_index_destroy(h)


def test_workspace_grows_with_batch(L):
    lib = L.lib()
    hs = [create(L) for _ in range(3)]
    prm = L.RetrieveParams(256, 16, 4, 0)
    one = lib.ss_retrieve_workspace_bytes(L.ptr_array([hs[0].value]), 1, (C.c_int32 * 1)(8), C.byref(prm))
    three = lib.ss_retrieve_workspace_bytes(L.ptr_array([h.value for h in hs]), 3, (C.c_int32 * 3)(8, 8, 8),
                                            C.byref(prm))
    assert three > one > 0
    for h in hs:
        lib.ss_index_destroy(h)


def test_evidence_validation(L):
    """Host-side checks of ss_assemble_evidence; nothing is launched."""
    lib = L.lib()
    h = create(L, max_frames=4, max_rows=4 * 196)
    idx = (C.c_void_p * 1)(h.value)
    P = L.EvidenceParams
    assert lib.ss_evidence_max_units(C.byref(P(6, 1, 0, 1)), 8, 0) == 6 + 8 * 2
    assert lib.ss_evidence_max_units(C.byref(P(6, 1, 0, 1)), 8, 5) == 6 + 8 * 2 + 5
    assert lib.ss_evidence_max_units(C.byref(P(2, 1, 0, 0)), 8, 5) == 2          # no retrieval, no clusters
    assert lib.ss_evidence_max_units(C.byref(P(0, 0, 0, 0)), 0, 0) == 1       # room for nothing, still >= 1
    assert lib.ss_evidence_max_units(C.byref(P(-1, 1, 0, 1)), 8, 0) == 0
    assert lib.ss_evidence_max_units(C.byref(P(6, 1, 0, 2)), 8, 0) == 0
    assert lib.ss_evidence_max_units(C.byref(P(6, 1, 0, 1)), 65, 0) == 0
    assert lib.ss_evidence_max_units(C.byref(P(6, 1, 0, 1)), 8, 65) == 0
    assert lib.ss_evidence_max_units(C.byref(P(4000, 10, 10, 1)), 64, 0) == 0   # beyond 4096 candidates
    ok = P(6, 1, 0, 1)
    F = FAKE
    ev = lambda n, fid, ns, cl, prm, units, kinds, nu, mx: lib.ss_assemble_evidence(  # noqa: E731
        idx, n, fid, ns, cl, prm, None, units, kinds, nu, mx)
    assert ev(1, F, 8, None, C.byref(ok), F, F, F, 10) == L.SS_ERR_INVALID_ARGUMENT
    assert b"max_units" in lib.ss_last_error()
    assert ev(1, None, 8, None, C.byref(ok), F, F, F, 22) == L.SS_ERR_INVALID_ARGUMENT
    assert ev(1, F, 8, None, C.byref(ok), None, F, F, 22) == L.SS_ERR_INVALID_ARGUMENT
    assert ev(1, F + 4, 8, None, C.byref(ok), F, F, F, 22) == L.SS_ERR_INVALID_ARGUMENT
    assert ev(0, F, 8, None, C.byref(ok), F, F, F, 22) == L.SS_ERR_INVALID_ARGUMENT
    assert ev(1, F, 8, None, None, F, F, F, 22) == L.SS_ERR_INVALID_ARGUMENT
    big = P(4000, 10, 10, 1)
    assert ev(1, F, 64, None, C.byref(big), F, F, F, 4096) == L.SS_ERR_UNSUPPORTED
    # with clusters: k_clusters range, the cluster ids and the kinds output are required
    sets = (C.c_void_p * 1)(None)
    EC = L.EvidenceClusters
    assert ev(1, F, 8, C.byref(EC(C.cast(sets, C.c_void_p), F, 0)), C.byref(ok), F, F, F, 22) == L.SS_ERR_UNSUPPORTED
    assert ev(1, F, 8, C.byref(EC(C.cast(sets, C.c_void_p), F, 4)), C.byref(ok), F, F, F, 22) == \
        L.SS_ERR_INVALID_ARGUMENT                                                 # 26 items need max_units 26
    assert ev(1, F, 8, C.byref(EC(C.cast(sets, C.c_void_p), None, 4)), C.byref(ok), F, F, F, 26) == \
        L.SS_ERR_INVALID_ARGUMENT
    assert ev(1, F, 8, C.byref(EC(C.cast(sets, C.c_void_p), F, 4)), C.byref(ok), F, None, F, 26) == \
        L.SS_ERR_INVALID_ARGUMENT
    assert ev(1, F, 8, C.byref(EC(None, F, 4)), C.byref(ok), F, F, F, 26) == L.SS_ERR_INVALID_ARGUMENT
    assert lib.ss_index_destroy(h) == 0


def test_pooled_validation(L):
    lib = L.lib()
    h = create(L, max_frames=4, max_rows=4 * 196)
    idx = (C.c_void_p * 1)(h.value)
    nq = (C.c_int32 * 1)(8)
    assert lib.ss_pooled_workspace_bytes(idx, 1, nq, 8) > 0
    assert lib.ss_pooled_workspace_bytes(idx, 1, nq, 0) == 0
    assert lib.ss_pooled_workspace_bytes(idx, 1, nq, 65) == 0
    bad = (C.c_int32 * 1)(0)
    assert lib.ss_pooled_workspace_bytes(idx, 1, bad, 8) == 0
    F = FAKE
    qs = (C.c_void_p * 4)(F, F, F, F)
    ws = lib.ss_pooled_workspace_bytes(idx, 1, nq, 8)
    assert lib.ss_retrieve_pooled(idx, 1, qs, nq, 8, F, ws - 1, None, F, F, F) == L.SS_ERR_WORKSPACE
    assert lib.ss_retrieve_pooled(idx, 1, qs, nq, 8, F, ws, None, None, F, F) == L.SS_ERR_INVALID_ARGUMENT
    qs_bad = (C.c_void_p * 4)(F, F + 2, F, F)
    assert lib.ss_retrieve_pooled(idx, 1, qs_bad, nq, 8, F, ws, None, F, F, F) == L.SS_ERR_INVALID_ARGUMENT
    assert b"queries[1]" in lib.ss_last_error()
    assert lib.ss_index_destroy(h) == 0


def test_clusters_validation(L):
    lib = L.lib()
    D = L.ClusterDesc
    ok = D(4, 4, 128, 196, 100, 0.9)
    n = lib.ss_clusters_required_bytes(C.byref(ok))
    assert n >= 100 * (512 * 4 + 4 + 16 + 4 * 4 * 196 * 128 * 4)
    for bad in (D(0, 4, 128, 196, 100, 0.9), D(4, 4, 96, 196, 100, 0.9), D(4, 4, 128, 0, 100, 0.9),
                D(4, 4, 128, 196, 0, 0.9), D(4, 4, 128, 196, 100, float("nan")), D(4, 16, 128, 196, 100, 0.9)):
        assert lib.ss_clusters_required_bytes(C.byref(bad)) == 0
    h = C.c_void_p()
    assert lib.ss_clusters_create(C.byref(ok), FAKE, n - 1, None, C.byref(h)) == L.SS_ERR_CAPACITY
    assert lib.ss_clusters_create(C.byref(ok), FAKE + 8, n, None, C.byref(h)) == L.SS_ERR_INVALID_ARGUMENT
    assert lib.ss_clusters_absorb_workspace_bytes(10) >= 80
    assert lib.ss_clusters_absorb_workspace_bytes(-1) == 0


def _poisson_tail(lam, r):
    """P(X >= r) for X ~ Poisson(lam), summed from the terms upward."""
    if lam <= 0:
        return 1.0 if r <= 0 else 0.0
    term = math.exp(-lam + r * math.log(lam) - math.lgamma(r + 1))
    tot, i = 0.0, r
    while term > 1e-300 and i < r + 4000:
        tot += term
        term *= lam / (i + 1)
        i += 1
    return tot


def _poisson_cdf(lam, r):
    """P(X <= r) for X ~ Poisson(lam)."""
    return sum(math.exp(-lam + i * math.log(lam) - math.lgamma(i + 1)) for i in range(r + 1)) if r >= 0 else 0.0


def test_sample_plan(L):
    """The streaming cut-off's sample plan (a host query, no GPU): small lists
    are sampled whole with r = k; otherwise the plan keeps both ways into the
    exact fallback (too few candidates, more than the capacity) at odds of at
    most 2e-7 per list, with the smallest rank that does so."""
    lib = L.lib()
    out = (C.c_int32 * 4)()
    assert lib.ss_debug_sample_plan(100, 8, None) == L.SS_ERR_INVALID_ARGUMENT
    assert lib.ss_debug_sample_plan(-1, 8, out) == L.SS_ERR_INVALID_ARGUMENT
    assert lib.ss_debug_sample_plan(100, 0, out) == L.SS_ERR_UNSUPPORTED
    assert lib.ss_debug_sample_plan(100, 2049, out) == L.SS_ERR_UNSUPPORTED
    for n, k in [(0, 8), (1, 8), (1000, 32), (4096, 512), (4096, 5000 // 3)]:
        assert lib.ss_debug_sample_plan(n, k, out) == 0
        m, r, cap, E = out
        assert m == n and r == min(k, n) and cap >= 4096
    for n, k in [(117600, 256), (705600, 512), (705600, 64), (19200, 64), (24000, 2048), (8388606, 2048),
                 (5000, 1), (200000, 1)]:
        assert lib.ss_debug_sample_plan(n, k, out) == 0
        m, r, cap, E = out
        kk = min(k, n)
        if m == n:
            assert r == kk
            continue
        assert 1 <= r <= min(kk, 32) and r <= m < n
        assert m == max(r, -(-n * r // E)) and E >= 6 * kk and cap >= 3 * E
        assert m <= 16384
        if r < min(kk, 32):
            assert _poisson_tail(r * kk / E, r) <= 2e-7 * (1 + 1e-9)
            assert _poisson_cdf(3.0 * r, r - 1) <= 2e-7 * (1 + 1e-9)
        if r > 1:
            worse = _poisson_tail((r - 1) * kk / E, r - 1) > 2e-7 or _poisson_cdf(3.0 * (r - 1), r - 2) > 2e-7
            assert worse, (n, k, r)
    lib.ss_debug_sample_plan(705600, 512, out)
    assert tuple(out)[:2] == (3216, 14)       # the 1-hour index: 3,216 sampled rows, rank 14


def test_window_compact_budget_on_empty_index(L):
    """Host paths of the compaction calls: an empty index stores nothing, has
    nothing to compact (no work is enqueued) and fits any budget."""
    lib = L.lib()
    h = create(L, max_frames=8, max_rows=8 * 196)
    a, b, fh = C.c_int64(-1), C.c_int64(-1), C.c_int64(-1)
    assert lib.ss_index_window(h, C.byref(a), C.byref(b)) == 0 and (a.value, b.value) == (0, 0)
    assert lib.ss_index_window(None, C.byref(a), C.byref(b)) == L.SS_ERR_INVALID_ARGUMENT
    assert lib.ss_index_compact(h, None) == 0
    assert lib.ss_index_compact(None, None) == L.SS_ERR_INVALID_ARGUMENT
    assert lib.ss_index_budget_split(h, 0, C.byref(fh)) == 0 and fh.value == 0
    assert lib.ss_index_budget_split(h, 0, None) == L.SS_ERR_INVALID_ARGUMENT
    assert lib.ss_index_destroy(h) == 0
