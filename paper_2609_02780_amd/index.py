"""Python binding over the C ABI.  PyTorch supplies device memory and streams only.

Tensors passed in must live on the current HIP device.  bfloat16 data may be
given as ``torch.bfloat16`` or as raw ``int16``/``uint16`` bit patterns.
"""
from __future__ import annotations

import ctypes as C

import torch

from . import _lib as L

_BF16_OK = (torch.bfloat16, torch.int16, torch.uint16)


def _stream_handle(stream) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _used_on(stream, *tensors) -> None:
    """Tell torch's caching allocator that work enqueued on a caller-given
    stream reads or writes these buffers, so that their memory is not handed
    out again before that work is done (buffers used on the current stream
    need nothing)."""
    if stream is None:
        return
    for t in tensors:
        if t is not None:
            t.record_stream(stream)


def sample_plan(n_rows: int, top_k: int) -> tuple[int, int, int, int]:
    """The library's sample plan of one list: ``(m, r, capacity, expected)``
    (see ``ss_debug_sample_plan``)."""
    out = (C.c_int32 * 4)()
    L.check(L.lib().ss_debug_sample_plan(n_rows, top_k, out))
    return tuple(out)


def _check_bf16(t: torch.Tensor, shape, what: str) -> int:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{what} must be a device tensor")
    if t.dtype not in _BF16_OK:
        raise ValueError(f"{what} must hold bfloat16 values (got {t.dtype})")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{what} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    return t.data_ptr()


class ShallowIndex:
    """One stream's shallow-layer key index in a device arena owned by this object."""

    def __init__(self, n_layers: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                 max_frames: int, max_rows: int, n_recent: int = 0, device=None):
        self.desc = L.IndexDesc(n_layers, n_q_heads, n_kv_heads, head_dim, max_frames, max_rows, n_recent)
        nbytes = L.lib().ss_index_required_bytes(C.byref(self.desc))
        if nbytes == 0:
            h = C.c_void_p()
            L.check(L.lib().ss_index_create(C.byref(self.desc), None, 0, C.byref(h)))
        dev = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
        self.arena = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        self._h = C.c_void_p()
        L.check(L.lib().ss_index_create(C.byref(self.desc), self.arena.data_ptr(), nbytes, C.byref(self._h)))
        self.n_layers, self.n_q_heads, self.n_kv_heads, self.head_dim = n_layers, n_q_heads, n_kv_heads, head_dim

    @property
    def handle(self) -> C.c_void_p:
        if self._h is None:
            raise RuntimeError("index closed")
        return self._h

    def close(self) -> None:
        if getattr(self, "_h", None) is not None:
            L.check(L.lib().ss_index_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def info(self) -> tuple[int, int]:
        f, r = C.c_int64(), C.c_int64()
        L.check(L.lib().ss_index_info(self.handle, C.byref(f), C.byref(r)))
        return f.value, r.value

    def window(self) -> tuple[int, int]:
        """``(first_stored, first_detail)``: the first frame the arena still
        stores, and the first frame of the detailed window."""
        a, b = C.c_int64(), C.c_int64()
        L.check(L.lib().ss_index_window(self.handle, C.byref(a), C.byref(b)))
        return a.value, b.value

    def compact(self, stream=None) -> None:
        """Drop the frames that left the detailed window from the arena (their
        space is reused by later appends)."""
        L.check(L.lib().ss_index_compact(self.handle, _stream_handle(stream)))

    def budget_split(self, budget_bytes: int) -> int:
        """The frame where the detailed window must start to fit ``budget_bytes``
        (pass it to :meth:`LongClusters.absorb`, then :meth:`compact`)."""
        h = C.c_int64()
        L.check(L.lib().ss_index_budget_split(self.handle, budget_bytes, C.byref(h)))
        return h.value

    @property
    def n_frames(self) -> int:
        return self.info()[0]

    @property
    def n_rows(self) -> int:
        return self.info()[1]

    def append(self, layer_keys, n_frames: int, n_tokens: int, compress=None, stream=None) -> int:
        """Append frames; ``layer_keys[l]`` is ``[H_kv][n_frames*n_tokens][d]`` bfloat16.
        ``compress`` is ``None`` or ``(n_centroids, n_iters)``.  Returns the first frame id."""
        shape = (self.n_kv_heads, n_frames * n_tokens, self.head_dim)
        ptrs = [_check_bf16(t, shape, f"layer_keys[{l}]") for l, t in enumerate(layer_keys)]
        if len(ptrs) != self.n_layers:
            raise ValueError(f"expected {self.n_layers} key tensors, got {len(ptrs)}")
        comp = L.Compress(*compress) if compress is not None else None
        first = C.c_int64()
        L.check(L.lib().ss_index_append(self.handle, L.ptr_array(ptrs), n_frames, n_tokens,
                                        C.byref(comp) if comp is not None else None,
                                        _stream_handle(stream), C.byref(first)))
        return first.value

    def export(self, stream=None) -> dict:
        """Stored rows, member counts, descriptors and frame offsets of the frames
        the arena stores (synchronises)."""
        f, r = self.info()
        f -= self.window()[0]          # stored frames
        dev = self.arena.device
        rows = torch.empty((self.n_layers, self.n_kv_heads, r, self.head_dim), dtype=torch.int16, device=dev)
        counts = torch.empty((self.n_layers, self.n_kv_heads, r), dtype=torch.int32, device=dev)
        desc = torch.empty((f, self.n_kv_heads * self.head_dim), dtype=torch.float32, device=dev)
        offs = (C.c_int64 * (f + 1))()
        L.check(L.lib().ss_index_export(self.handle, rows.data_ptr(), counts.data_ptr(), desc.data_ptr(),
                                        offs, _stream_handle(stream)))
        torch.cuda.synchronize(dev)
        return {"rows": rows.cpu().numpy().view("uint16"), "counts": counts.cpu().numpy(),
                "desc": desc.cpu().numpy(), "frame_offsets": list(offs)}

    def debug_scores(self, queries, layer: int, q_head: int, head_mode: int = 0, row0: int = 0,
                     n_rows: int | None = None, stream=None) -> torch.Tensor:
        """fp32 scores of one list over rows ``[row0, row0 + n_rows)`` (parity checks)."""
        n_q = queries[0].shape[1]
        qshape = (self.n_q_heads, n_q, self.head_dim)
        qp = [_check_bf16(q, qshape, f"queries[{l}]") for l, q in enumerate(queries)]
        if n_rows is None:
            n_rows = self.n_rows - row0
        out = torch.empty(max(n_rows, 1), dtype=torch.float32, device=self.arena.device)
        wsb = L.lib().ss_debug_scores_workspace_bytes(self.handle)
        ws = torch.empty(wsb, dtype=torch.uint8, device=self.arena.device)
        L.check(L.lib().ss_debug_scores(self.handle, L.ptr_array(qp), n_q, layer, q_head, head_mode,
                                        row0, n_rows, out.data_ptr(), ws.data_ptr(), wsb,
                                        _stream_handle(stream)))
        _used_on(stream, ws, out)
        return out[:n_rows]


class Retriever:
    """Evidence retrieval over a batch of indices with identical shapes.

    Holds the device workspace and output buffers, grown on demand, so repeated
    calls allocate nothing once sizes are stable.
    """

    def __init__(self, indices, top_k: int, n_select: int, pool_mult: int = 4, head_mode: int = 0,
                 score_mode: int = 0):
        self.indices = list(indices)
        self.params = L.RetrieveParams(top_k, n_select, pool_mult, head_mode, score_mode)
        self._ws = None
        dev = self.indices[0].arena.device
        S = len(self.indices)
        self.frame_ids = torch.empty((S, n_select), dtype=torch.int64, device=dev)
        self.votes = torch.empty((S, n_select), dtype=torch.int32, device=dev)
        self.mass = torch.empty((S, n_select), dtype=torch.float32, device=dev)
        self.n_out = torch.empty(S, dtype=torch.int32, device=dev)
        self._handles = L.ptr_array([x.handle.value for x in self.indices])

    def workspace_bytes(self, n_q) -> int:
        nq = (C.c_int32 * len(self.indices))(*n_q)
        need = L.lib().ss_retrieve_workspace_bytes(self._handles, len(self.indices), nq, C.byref(self.params))
        if need == 0:
            raise L.SSError(L.SS_ERR_INVALID_ARGUMENT, L.lib().ss_last_error().decode())
        return need

    def _marshal(self, queries):
        S = len(self.indices)
        if len(queries) != S:
            raise ValueError(f"expected queries for {S} streams, got {len(queries)}")
        ptrs, n_q = [], []
        for s, (x, qs) in enumerate(zip(self.indices, queries)):
            if len(qs) != x.n_layers:
                raise ValueError(f"stream {s}: expected {x.n_layers} query tensors")
            nq = qs[0].shape[1]
            n_q.append(nq)
            for l, q in enumerate(qs):
                ptrs.append(_check_bf16(q, (x.n_q_heads, nq, x.head_dim), f"queries[{s}][{l}]"))
        need = self.workspace_bytes(n_q)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(need, dtype=torch.uint8, device=self.frame_ids.device)
        return L.ptr_array(ptrs), (C.c_int32 * S)(*n_q)

    def __call__(self, queries, stream=None):
        """``queries[s][l]``: ``[H_q][n_q][d]`` bfloat16.  Returns device tensors
        ``(frame_ids, votes, mass, n_out)`` (views of reused buffers)."""
        qp, nq = self._marshal(queries)
        L.check(L.lib().ss_retrieve(self._handles, len(self.indices), qp, nq, C.byref(self.params),
                                    self._ws.data_ptr(), self._ws.numel(), _stream_handle(stream),
                                    self.frame_ids.data_ptr(), self.votes.data_ptr(), self.mass.data_ptr(),
                                    self.n_out.data_ptr()))
        _used_on(stream, self._ws)
        return self.frame_ids, self.votes, self.mass, self.n_out

    def noalloc(self, queries, stream=None):
        """The same retrieval through ``ss_retrieve_noalloc``: the library's own
        device workspace instead of this object's (no device allocation by the
        library or here).  Returns the same reused output buffers."""
        S = len(self.indices)
        if len(queries) != S:
            raise ValueError(f"expected queries for {S} streams, got {len(queries)}")
        ptrs, n_q = [], []
        for s, (x, qs) in enumerate(zip(self.indices, queries)):
            if len(qs) != x.n_layers:
                raise ValueError(f"stream {s}: expected {x.n_layers} query tensors")
            nq = qs[0].shape[1]
            n_q.append(nq)
            for l, q in enumerate(qs):
                ptrs.append(_check_bf16(q, (x.n_q_heads, nq, x.head_dim), f"queries[{s}][{l}]"))
        L.check(L.lib().ss_retrieve_noalloc(self._handles, S, L.ptr_array(ptrs), (C.c_int32 * S)(*n_q),
                                            C.byref(self.params), _stream_handle(stream),
                                            self.frame_ids.data_ptr(), self.votes.data_ptr(),
                                            self.mass.data_ptr(), self.n_out.data_ptr()))
        return self.frame_ids, self.votes, self.mass, self.n_out

    def debug(self, queries, stream=None) -> dict:
        """One retrieval with every intermediate (synchronises; parity checks only)."""
        qp, nq = self._marshal(queries)
        S = len(self.indices)
        dev = self.frame_ids.device
        p = self.params
        NL = self.indices[0].n_layers * (self.indices[0].n_q_heads if p.head_mode == 0 else 1)
        hist = max(x.desc.max_frames for x in self.indices)
        pool = p.pool_mult * p.n_select
        t = {
            "topk_pos": torch.empty((S, NL, p.top_k), dtype=torch.int32, device=dev),
            "topk_score": torch.empty((S, NL, p.top_k), dtype=torch.float32, device=dev),
            "vote_hist": torch.empty((S, hist), dtype=torch.int32, device=dev),
            "mass_hist": torch.empty((S, hist), dtype=torch.float32, device=dev),
            "pool": torch.empty((S, pool), dtype=torch.int32, device=dev),
            "pool_n": torch.empty(S, dtype=torch.int32, device=dev),
            "list_stats": torch.empty((S, NL, 2), dtype=torch.int32, device=dev),
        }
        dbg = L.DebugOut(*(t[k].data_ptr() for k in ("topk_pos", "topk_score", "vote_hist", "mass_hist",
                                                      "pool", "pool_n", "list_stats")))
        L.check(L.lib().ss_retrieve_debug(self._handles, S, qp, nq, C.byref(p), self._ws.data_ptr(),
                                          self._ws.numel(), _stream_handle(stream), self.frame_ids.data_ptr(),
                                          self.votes.data_ptr(), self.mass.data_ptr(), self.n_out.data_ptr(),
                                          C.byref(dbg)))
        _used_on(stream, self._ws)
        torch.cuda.synchronize(dev)
        out = {k: v.cpu().numpy() for k, v in t.items()}
        out.update(frame_ids=self.frame_ids.cpu().numpy(), votes=self.votes.cpu().numpy(),
                   mass=self.mass.cpu().numpy(), n_out=self.n_out.cpu().numpy())
        return out


class PooledRanker:
    """Pooled shallow Q-K ranking over a batch of indices with identical shapes
    (unit-mean keys against the question's mean query; no diversity)."""

    def __init__(self, indices, n_select: int):
        self.indices = list(indices)
        self.n_select = n_select
        self._ws = None
        dev = self.indices[0].arena.device
        S = len(self.indices)
        self.frame_ids = torch.empty((S, n_select), dtype=torch.int64, device=dev)
        self.scores = torch.empty((S, n_select), dtype=torch.float32, device=dev)
        self.n_out = torch.empty(S, dtype=torch.int32, device=dev)
        self._handles = L.ptr_array([x.handle.value for x in self.indices])

    def __call__(self, queries, stream=None):
        """``queries[s][l]``: ``[H_q][n_q][d]`` bfloat16.  Returns device tensors
        ``(frame_ids, scores, n_out)`` (views of reused buffers)."""
        S = len(self.indices)
        if len(queries) != S:
            raise ValueError(f"expected queries for {S} streams, got {len(queries)}")
        ptrs, n_q = [], []
        for s, (x, qs) in enumerate(zip(self.indices, queries)):
            if len(qs) != x.n_layers:
                raise ValueError(f"stream {s}: expected {x.n_layers} query tensors")
            nq = qs[0].shape[1]
            n_q.append(nq)
            for l, q in enumerate(qs):
                ptrs.append(_check_bf16(q, (x.n_q_heads, nq, x.head_dim), f"queries[{s}][{l}]"))
        nqa = (C.c_int32 * S)(*n_q)
        need = L.lib().ss_pooled_workspace_bytes(self._handles, S, nqa, self.n_select)
        if need == 0:
            raise L.SSError(L.SS_ERR_INVALID_ARGUMENT, L.lib().ss_last_error().decode())
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(need, dtype=torch.uint8, device=self.frame_ids.device)
        L.check(L.lib().ss_retrieve_pooled(self._handles, S, L.ptr_array(ptrs), nqa, self.n_select,
                                           self._ws.data_ptr(), self._ws.numel(), _stream_handle(stream),
                                           self.frame_ids.data_ptr(), self.scores.data_ptr(),
                                           self.n_out.data_ptr()))
        _used_on(stream, self._ws)
        return self.frame_ids, self.scores, self.n_out


class LongClusters:
    """Long-term clusters of the frames that left an index's detailed window
    (the paper's optional long-history compression), in a device arena owned by
    this object."""

    def __init__(self, index: ShallowIndex, rows_per_unit: int, max_clusters: int, tau: float, stream=None):
        self.index = index
        self.desc = L.ClusterDesc(index.n_layers, index.n_kv_heads, index.head_dim, rows_per_unit,
                                  max_clusters, tau)
        nbytes = L.lib().ss_clusters_required_bytes(C.byref(self.desc))
        if nbytes == 0:
            raise L.SSError(L.SS_ERR_INVALID_ARGUMENT, "invalid cluster description")
        self.arena = torch.empty(nbytes, dtype=torch.uint8, device=index.arena.device)
        self._h = C.c_void_p()
        L.check(L.lib().ss_clusters_create(C.byref(self.desc), self.arena.data_ptr(), nbytes,
                                           _stream_handle(stream), C.byref(self._h)))
        self._ws = None
        self._qws = None

    def close(self) -> None:
        if getattr(self, "_h", None) is not None:
            L.check(L.lib().ss_clusters_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def absorb(self, frame_hi: int, n_frames: int, stream=None) -> None:
        """Frames up to ``frame_hi`` (exclusive) leave the detailed window;
        ``n_frames`` is how many leave in this call (sizes the workspace)."""
        need = L.lib().ss_clusters_absorb_workspace_bytes(n_frames)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(need, dtype=torch.uint8, device=self.arena.device)
        L.check(L.lib().ss_clusters_absorb(self._h, self.index.handle, frame_hi, self._ws.data_ptr(),
                                           self._ws.numel(), _stream_handle(stream)))
        _used_on(stream, self._ws)

    def retrieve(self, queries, k_clusters: int, stream=None):
        """``queries[l]``: ``[H_q][n_q][d]`` bfloat16 (only the last layer is
        read).  Returns device tensors ``(cluster_ids, scores, first_frame,
        last_frame, n_out)``."""
        x = self.index
        if len(queries) != x.n_layers:
            raise ValueError(f"expected {x.n_layers} query tensors")
        nq = queries[0].shape[1]
        ptrs = [_check_bf16(q, (x.n_q_heads, nq, x.head_dim), f"queries[{l}]") for l, q in enumerate(queries)]
        need = L.lib().ss_clusters_retrieve_workspace_bytes(self._h)
        if self._qws is None or self._qws.numel() < need:
            self._qws = torch.empty(need, dtype=torch.uint8, device=self.arena.device)
        dev = self.arena.device
        ids = torch.empty(k_clusters, dtype=torch.int64, device=dev)
        sc = torch.empty(k_clusters, dtype=torch.float32, device=dev)
        first = torch.empty(k_clusters, dtype=torch.int64, device=dev)
        last = torch.empty(k_clusters, dtype=torch.int64, device=dev)
        n_out = torch.empty(1, dtype=torch.int32, device=dev)
        L.check(L.lib().ss_clusters_retrieve(self._h, x.handle, L.ptr_array(ptrs), nq, k_clusters,
                                             self._qws.data_ptr(), self._qws.numel(), _stream_handle(stream),
                                             ids.data_ptr(), sc.data_ptr(), first.data_ptr(), last.data_ptr(),
                                             n_out.data_ptr()))
        _used_on(stream, self._qws, ids, sc, first, last, n_out)
        return ids, sc, first, last, n_out

    def export(self, stream=None) -> dict:
        """The cluster state on the host (synchronises; parity checks only)."""
        d = self.desc
        M, dim = d.max_clusters, d.n_kv_heads * d.head_dim
        dev = self.arena.device
        t = {"state": torch.empty(2, dtype=torch.int32, device=dev),
             "centroids": torch.empty((M, dim), dtype=torch.float32, device=dev),
             "sizes": torch.empty(M, dtype=torch.int32, device=dev),
             "span": torch.empty((M, 2), dtype=torch.int64, device=dev),
             "reps": torch.empty((M, d.n_layers, d.n_kv_heads, d.rows_per_unit, d.head_dim), dtype=torch.float32,
                                 device=dev)}
        L.check(L.lib().ss_clusters_export(self._h, *(t[k].data_ptr() for k in ("state", "centroids", "sizes",
                                                                                  "span", "reps")),
                                           _stream_handle(stream)))
        torch.cuda.synchronize(dev)
        out = {k: v.cpu().numpy() for k, v in t.items()}
        n = int(out["state"][0])
        return {"n_clusters": n, "overflow": bool(out["state"][1]), "centroids": out["centroids"][:n],
                "sizes": out["sizes"][:n], "span": out["span"][:n], "reps": out["reps"][:n]}


def assemble_evidence(indices, frame_ids, n_recent: int, n_before: int = 1, n_after: int = 0,
                      retrieved: bool = True, clusters=None, cluster_ids=None, stream=None):
    """The evidence handed to answering for each stream (Eq. selected_evidence,
    united with the retrieved long-term clusters of Eq.
    selected_cluster_evidence when ``clusters`` is given; deduplicated, in
    temporal order).  ``frame_ids``: device int64 ``[n_streams][n_select]`` as
    returned by :class:`Retriever` (ignored when ``retrieved`` is false).
    ``clusters``: a list of :class:`LongClusters` (or None) per stream, with
    ``cluster_ids`` device int64 ``[n_streams][k_clusters]``.  Returns device
    tensors ``(units, kinds, n_units)``: ``units`` int64 and ``kinds`` int32
    ``[n_streams][max_units]`` (kind 0 a frame id, 1 a cluster id; -1 padded)."""
    indices = list(indices)
    S = len(indices)
    n_select = frame_ids.shape[1] if (retrieved and frame_ids is not None) else 0
    prm = L.EvidenceParams(n_recent, n_before, n_after, 1 if retrieved else 0)
    dev = indices[0].arena.device
    ec = None
    k_clusters = 0
    keep = []
    if clusters is not None:
        if len(clusters) != S:
            raise ValueError(f"expected {S} cluster sets (or None entries)")
        if cluster_ids is None or cluster_ids.dtype != torch.int64 or not cluster_ids.is_cuda \
                or cluster_ids.dim() != 2 or cluster_ids.shape[0] != S or not cluster_ids.is_contiguous():
            raise ValueError("cluster_ids must be a contiguous device int64 tensor [n_streams][k_clusters]")
        k_clusters = cluster_ids.shape[1]
        sets = L.ptr_array([c._h.value if c is not None else None for c in clusters])
        keep.append(sets)
        ec = L.EvidenceClusters(C.cast(sets, C.c_void_p), cluster_ids.data_ptr(), k_clusters)
    max_units = L.lib().ss_evidence_max_units(C.byref(prm), n_select, k_clusters)
    if max_units == 0:
        raise L.SSError(L.SS_ERR_INVALID_ARGUMENT, "invalid evidence parameters")
    fid = 0
    if retrieved:
        if frame_ids.dtype != torch.int64 or not frame_ids.is_cuda or tuple(frame_ids.shape) != (S, n_select) \
                or not frame_ids.is_contiguous():
            raise ValueError("frame_ids must be a contiguous device int64 tensor [n_streams][n_select]")
        fid = frame_ids.data_ptr()
    units = torch.empty((S, max_units), dtype=torch.int64, device=dev)
    kinds = torch.empty((S, max_units), dtype=torch.int32, device=dev)
    n_units = torch.empty(S, dtype=torch.int32, device=dev)
    handles = L.ptr_array([x.handle.value for x in indices])
    L.check(L.lib().ss_assemble_evidence(handles, S, fid, n_select, C.byref(ec) if ec is not None else None,
                                         C.byref(prm), _stream_handle(stream), units.data_ptr(), kinds.data_ptr(),
                                         n_units.data_ptr(), max_units))
    _used_on(stream, units, kinds, n_units)
    return units, kinds, n_units


def set_profile_events(start, stop) -> None:
    """Record ``start``/``stop`` (torch.cuda.Event) around the streaming scoring
    kernel of later retrievals on this thread; ``None, None`` turns it off."""
    a = start.cuda_event if start is not None else None
    b = stop.cuda_event if stop is not None else None
    L.check(L.lib().ss_set_profile_events(a, b))
