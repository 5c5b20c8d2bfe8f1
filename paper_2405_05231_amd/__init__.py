"""MI355X (gfx950) offline-sampling hot path after DiskGNN (arXiv 2405.05231):
group sampling, batched packing and batch assembly, run by the HIP kernels of
libdg.so.

This module only marshals torch tensors (device memory + the current HIP
stream) into the C ABI declared in include/dg.h; every step of the path runs
in the library's kernels.  Importing it fails if libdg.so is missing.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass

import numpy as np
import torch

from . import _lib
from ._lib import (DG_ECAPACITY, DG_MAX_BATCHES, DG_OK, DGError, Csr, Sizes, Timing, check,
                   load)

__all__ = ["sample_bounds", "member_lines_bytes", "sample_group", "pack_group", "assemble_batch",
           "assemble_batches", "cache_by_frequency",
           "gather_rows", "pack_individual", "minhash_order", "DGError", "SampleResult",
           "PackResult", "version"]

_L = load()


def version() -> str:
    return _L.dg_version().decode()


def _ptr(t: torch.Tensor | None):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _need(t: torch.Tensor, name: str, dtype=None, device=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if device is not None and t.device != device:
        raise ValueError(f"{name}: expected device {device}, got {t.device}")
    if t.device.type != "cuda":
        raise ValueError(f"{name}: must live in GPU memory")


def _workspace(nbytes: int, device, ws: torch.Tensor | None):
    if ws is not None and ws.numel() * ws.element_size() >= nbytes:
        return ws
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


def member_lines_bytes(num_nodes: int) -> int:
    """Bytes of a member-lines map (dg_member_lines_bytes)."""
    return int(_L.dg_member_lines_bytes(num_nodes))


def sample_bounds(num_nodes: int, num_edges: int, S: int, fanouts,
                  layered: bool = False) -> tuple[int, int]:
    fo = (ctypes.c_int32 * max(len(fanouts), 1))(*fanouts)
    nc, ec = ctypes.c_int64(), ctypes.c_int64()
    check(_L.dg_sample_bounds(num_nodes, num_edges, S, fo, len(fanouts),
                              _lib.DG_SAMPLE_LAYERED if layered else 0, ctypes.byref(nc),
                              ctypes.byref(ec)))
    return nc.value, ec.value


@dataclass
class SampleResult:
    nodes: torch.Tensor      # int32 [B, node_cap]
    hop_ptr: np.ndarray      # int64 [B, K+2]
    edge_src: torch.Tensor   # int32 [B, edge_cap] local
    edge_dst: torch.Tensor   # int32 [B, edge_cap] local
    edge_ptr: np.ndarray     # int64 [B, K+1]
    sizes: dict
    timing: dict | None

    @property
    def node_count(self) -> np.ndarray:
        return np.ascontiguousarray(self.hop_ptr[:, -1])

    def batch_nodes(self, b: int) -> torch.Tensor:
        return self.nodes[b, :int(self.hop_ptr[b, -1])]

    def batch_edges(self, b: int):
        e = int(self.edge_ptr[b, -1])
        return self.edge_src[b, :e], self.edge_dst[b, :e]


def sample_flags(layered: bool = False, direct: bool = False, entry_clear: bool = False,
                 exit_clear: bool = False) -> int:
    """dg_sample_group flag word."""
    return ((_lib.DG_SAMPLE_LAYERED if layered else 0) | (_lib.DG_SAMPLE_DIRECT if direct else 0)
            | (_lib.DG_SAMPLE_ENTRY_CLEAR if entry_clear else 0)
            | (_lib.DG_SAMPLE_EXIT_CLEAR if exit_clear else 0))


def sample_group(offsets: torch.Tensor, indices: torch.Tensor, seeds: torch.Tensor, fanouts,
                 rng_seed: int, batch_base: int = 0, node_cap: int | None = None,
                 edge_cap: int | None = None, out: SampleResult | None = None,
                 workspace: torch.Tensor | None = None, stream=None, timing: bool = False,
                 membership: torch.Tensor | None = None, layered: bool = False,
                 direct: bool = False, entry_clear: bool = False,
                 exit_clear: bool = False, member_lines: torch.Tensor | None = None,
                 cache_slot: torch.Tensor | None = None, loc: torch.Tensor | None = None
                 ) -> SampleResult:
    """Group sampling (dg_sample_group).  seeds: int32 [B, S] on the GPU.
    membership: optional int64 [N] tensor that receives the (node, batch)
    membership mask (bit b of word u = u is in batch b).  layered: every node
    of the mini-batch so far samples at each hop (DGL-style layer blocks).
    direct: relabel through a direct [N][B] table (4*N*B workspace bytes).
    exit_clear / entry_clear: DG_SAMPLE_EXIT_CLEAR / DG_SAMPLE_ENTRY_CLEAR (a
    loop over groups that reuses `workspace` and `membership`, packing each
    group with clear_membership=True, skips two mask clears per group).
    member_lines: optional uint8 tensor of member_lines_bytes(N) bytes that
    receives a byte per 8 nodes, non-zero iff one of them is in some list.
    cache_slot, loc: int32 [N] and int32 [B, node_cap] (both or neither): loc
    receives the address-table entries of cached nodes, DG_LOC_PENDING for the
    others, for pack_group(..., loc_pending=True) to complete."""
    dev = offsets.device
    _need(offsets, "offsets", torch.int64)
    _need(indices, "indices", torch.int32, dev)
    _need(seeds, "seeds", torch.int32, dev)
    if membership is not None:
        _need(membership, "membership", torch.int64, dev)
        if membership.numel() != offsets.numel() - 1:
            raise ValueError("membership must hold one word per node")
    if seeds.dim() != 2:
        raise ValueError("seeds must be [B, S]")
    if member_lines is not None:
        _need(member_lines, "member_lines", torch.uint8, dev)
        if member_lines.numel() < member_lines_bytes(offsets.numel() - 1):
            raise ValueError("member_lines holds fewer than member_lines_bytes(N) bytes")
    if (cache_slot is None) != (loc is None):
        raise ValueError("cache_slot and loc go together")
    if cache_slot is not None:
        _need(cache_slot, "cache_slot", torch.int32, dev)
        _need(loc, "loc", torch.int32, dev)
        if cache_slot.numel() != offsets.numel() - 1:
            raise ValueError("cache_slot must hold one entry per node")
    B, S = seeds.shape
    N = offsets.numel() - 1
    E = indices.numel()
    fanouts = [int(f) for f in fanouts]
    K = len(fanouts)
    if out is not None:
        node_cap, edge_cap = out.nodes.shape[1], out.edge_src.shape[1]
    else:
        bn, be = sample_bounds(N, E, S, fanouts, layered)
        node_cap = bn if node_cap is None else node_cap
        edge_cap = be if edge_cap is None else edge_cap
        out = SampleResult(
            nodes=torch.empty((B, node_cap), dtype=torch.int32, device=dev),
            hop_ptr=np.zeros((B, K + 2), dtype=np.int64),
            edge_src=torch.empty((B, max(edge_cap, 1)), dtype=torch.int32, device=dev),
            edge_dst=torch.empty((B, max(edge_cap, 1)), dtype=torch.int32, device=dev),
            edge_ptr=np.zeros((B, K + 1), dtype=np.int64), sizes={}, timing=None)
    if loc is not None and (loc.dim() != 2 or tuple(loc.shape) != (B, node_cap)):
        raise ValueError("loc must be [B, node_cap], laid out as the node lists")
    flags = sample_flags(layered, direct, entry_clear, exit_clear)
    ws_bytes = _L.dg_sample_workspace_bytes(N, B, node_cap, edge_cap, flags)
    ws = _workspace(ws_bytes, dev, workspace)
    g = Csr(N, E, offsets.data_ptr(), indices.data_ptr())
    fo = (ctypes.c_int32 * max(K, 1))(*fanouts)
    sz, tm = Sizes(), Timing()
    st = _L.dg_sample_group(
        ctypes.byref(g), _ptr(seeds), B, S, batch_base, fo, K, rng_seed & (2**64 - 1),
        flags, node_cap, _ptr(out.nodes), out.hop_ptr.ctypes.data_as(_lib.I64P), edge_cap,
        _ptr(out.edge_src), _ptr(out.edge_dst), out.edge_ptr.ctypes.data_as(_lib.I64P),
        _ptr(membership), _ptr(member_lines), _ptr(cache_slot), _ptr(loc), _ptr(ws),
        ws.numel(), _stream(stream),
        ctypes.byref(sz),
        ctypes.byref(tm) if timing else None)
    out.sizes = sz.as_dict()
    check(st)
    out.timing = tm.as_dict() if timing else None
    return out


@dataclass
class PackResult:
    packed: torch.Tensor          # uint8 [packed_rows, row_bytes] (or the caller's buffer)
    packed_ids: torch.Tensor      # int32 [packed_rows]
    packed_ptr: torch.Tensor      # int64 [B+1] on the GPU
    packed_ptr_host: np.ndarray   # int64 [B+1]
    loc: torch.Tensor             # int32 [B, node_stride]
    unique: torch.Tensor | None   # int32 [|U|]
    sizes: dict
    timing: dict | None
    row_bytes: int

    def chunk(self, b: int) -> torch.Tensor:
        """Packed rows of batch b (a view)."""
        return self.packed[int(self.packed_ptr_host[b]):int(self.packed_ptr_host[b + 1])]


def _row_bytes(feats: torch.Tensor) -> int:
    return feats[0].numel() * feats.element_size() if feats.shape[0] else 0


def pack_group(feats: torch.Tensor, cache_slot: torch.Tensor, nodes: torch.Tensor, node_count,
               with_unique: bool = False, out: PackResult | None = None,
               workspace: torch.Tensor | None = None, stream=None, timing: bool = False,
               membership: torch.Tensor | None = None, tables_only: bool = False,
               clear_membership: bool = False, rows_stream=None,
               member_lines: torch.Tensor | None = None, no_alloc: bool = False,
               loc_pending: bool = False, cache_nodes: torch.Tensor | None = None,
               cache_table: torch.Tensor | None = None) -> PackResult:
    """Batched packing (dg_pack_group).  nodes: int32 [B, node_stride];
    node_count: the B list lengths (host).  membership: optional int64 [N]
    mask from sample_group (skips rebuilding it).  tables_only: build the
    packed order and address tables without copying rows (packed = None).
    clear_membership: DG_PACK_CLEAR_MEMBERSHIP (membership is all-zero after
    the call).  rows_stream: DG_PACK_ROWS_STREAM, the row copy is left queued on
    that stream (the call returns once the tables are done; keep `workspace`,
    `feats` and the packed buffer untouched until the copy has run).
    member_lines: the map sample_group wrote (with membership): only the
    words of marked lines are read.  no_alloc: call dg_pack_group_noalloc
    (scratch inside the library, no workspace; no timing or rows_stream);
    pass `out` as well for a call that allocates nothing at all.
    loc_pending: DG_PACK_LOC_PENDING, out.loc already holds what sample_group
    wrote into it for these lists and this cache_slot (`out` required).
    cache_nodes, cache_table: int32 [C] and a [C, row_bytes]-byte buffer: the
    row copy also fills cache row s with the features of cache_nodes[s] (the
    cache as one more mini-batch of the same gather)."""
    dev = feats.device
    _need(feats, "feats", None)
    _need(cache_slot, "cache_slot", torch.int32, dev)
    _need(nodes, "nodes", torch.int32, dev)
    N = feats.shape[0]
    R = _row_bytes(feats)
    B, stride = nodes.shape
    if membership is not None:
        _need(membership, "membership", torch.int64, dev)
        if membership.numel() != N:
            raise ValueError("membership must hold one word per node")
    if member_lines is not None:
        _need(member_lines, "member_lines", torch.uint8, dev)
        if member_lines.numel() < member_lines_bytes(N):
            raise ValueError("member_lines holds fewer than member_lines_bytes(N) bytes")
    counts = np.ascontiguousarray(np.asarray(node_count, dtype=np.int64).reshape(-1))
    if counts.shape[0] != B:
        raise ValueError("node_count must have one entry per batch")
    total = int(counts.sum())
    n_cache = 0
    if (cache_nodes is None) != (cache_table is None):
        raise ValueError("cache_nodes and cache_table go together")
    if cache_nodes is not None:
        _need(cache_nodes, "cache_nodes", torch.int32, dev)
        _need(cache_table, "cache_table", None, dev)
        n_cache = cache_nodes.numel()
        if cache_table.numel() * cache_table.element_size() < n_cache * R:
            raise ValueError("cache_table holds fewer than len(cache_nodes) rows")
    if loc_pending and (out is None or tuple(out.loc.shape) != (B, stride)):
        raise ValueError("loc_pending needs `out` whose loc is laid out as the node lists")
    if no_alloc:
        if timing or rows_stream is not None:
            raise ValueError("no_alloc takes neither timing nor rows_stream")
        ws = None
    else:
        ws = _workspace(_L.dg_pack_workspace_bytes(N, B, total), dev, workspace)

    def call(cap, packed, packed_ids, ptr, ptr_host, loc, unique, unique_cap, flags, sz, tm,
             fill_cache=True):
        fill = fill_cache and cache_nodes is not None
        head = (_ptr(feats), N, R, _ptr(cache_slot), B, _ptr(nodes), stride,
                counts.ctypes.data_as(_lib.I64P), cap, packed, packed_ids, ptr,
                ptr_host.ctypes.data_as(_lib.I64P), loc, unique, unique_cap,
                _ptr(membership), _ptr(member_lines), _ptr(cache_nodes) if fill else None,
                n_cache if fill else 0, _ptr(cache_table) if fill else None, flags)
        if no_alloc:
            return _L.dg_pack_group_noalloc(*head, _stream(stream), ctypes.byref(sz))
        return _L.dg_pack_group(*head, _ptr(ws), ws.numel(), _stream(stream),
                                _stream(rows_stream) if rows_stream is not None else None,
                                ctypes.byref(sz), ctypes.byref(tm) if tm is not None else None)

    ptr_host = np.zeros(B + 1, dtype=np.int64)
    sz, tm = Sizes(), Timing()
    if out is None and tables_only:
        out = PackResult(packed=None, packed_ids=torch.empty(max(total, 1), dtype=torch.int32,
                                                             device=dev),
                         packed_ptr=torch.empty(B + 1, dtype=torch.int64, device=dev),
                         packed_ptr_host=ptr_host, loc=torch.empty((B, stride), dtype=torch.int32,
                                                                   device=dev),
                         unique=torch.empty(max(total, 1), dtype=torch.int32, device=dev)
                         if with_unique else None, sizes={}, timing=None, row_bytes=R)
    if out is None:
        loc = torch.empty((B, stride), dtype=torch.int32, device=dev)
        ptr = torch.empty(B + 1, dtype=torch.int64, device=dev)
        # size query: a zero packed capacity returns the exact sizes needed
        st = call(0, None, None, _ptr(ptr), ptr_host, _ptr(loc), None, 0, 0, sz, None,
                  fill_cache=False)
        if st not in (DG_OK, DG_ECAPACITY):
            check(st)
        rows, nu = sz.packed_rows, sz.unique_nodes
        out = PackResult(
            packed=torch.empty((max(rows, 1), R), dtype=torch.uint8, device=dev),
            packed_ids=torch.empty(max(rows, 1), dtype=torch.int32, device=dev),
            packed_ptr=ptr, packed_ptr_host=ptr_host, loc=loc,
            unique=torch.empty(max(nu, 1), dtype=torch.int32, device=dev) if with_unique else None,
            sizes={}, timing=None, row_bytes=R)
    cap = out.packed_ids.numel()
    if out.packed is not None and out.packed.numel() < cap * R:
        raise ValueError("packed buffer smaller than packed_ids")
    st = call(cap, _ptr(out.packed), _ptr(out.packed_ids), _ptr(out.packed_ptr),
              out.packed_ptr_host, _ptr(out.loc), _ptr(out.unique),
              out.unique.numel() if out.unique is not None else 0,
              (_lib.DG_PACK_CLEAR_MEMBERSHIP if clear_membership else 0)
              | (_lib.DG_PACK_ROWS_STREAM if rows_stream is not None else 0)
              | (_lib.DG_PACK_LOC_PENDING if loc_pending else 0),
              sz, tm if timing else None)
    out.sizes = sz.as_dict()
    check(st)
    out.timing = tm.as_dict() if timing else None
    return out


def sample_pack_group(offsets: torch.Tensor, indices: torch.Tensor, seeds: torch.Tensor,
                      fanouts, rng_seed: int, feats: torch.Tensor, cache_slot: torch.Tensor,
                      batch_base: int = 0, node_cap: int | None = None,
                      edge_cap: int | None = None, out: SampleResult | None = None,
                      pack_out: PackResult | None = None, with_unique: bool = False,
                      tables_only: bool = False, workspace: torch.Tensor | None = None,
                      pack_workspace: torch.Tensor | None = None, stream=None,
                      rows_stream=None, timing: bool = False,
                      membership: torch.Tensor | None = None, layered: bool = False,
                      direct: bool = True, entry_clear: bool = False,
                      exit_clear: bool = False) -> tuple[SampleResult, PackResult]:
    """Group sampling and batched packing in one call (dg_sample_pack_group):
    the results of sample_group(..., cache_slot=cache_slot, loc=...) followed by
    pack_group(..., membership, clear_membership=True, loc_pending=True), with
    the membership words consumed (all-zero afterwards).  With direct=True the
    last hop's compaction also does packing's pass.  pack_out: buffers for the
    packing outputs (loc [B, node_cap], packed_ids, packed, packed_ptr,
    unique); without it the call first runs once with no packed capacity to
    learn the sizes (so the group is sampled twice).  rows_stream: leave the
    row copy queued there (DG_PACK_ROWS_STREAM; keep pack_workspace, feats and
    the packed buffer untouched until it has run)."""
    dev = offsets.device
    _need(offsets, "offsets", torch.int64)
    _need(indices, "indices", torch.int32, dev)
    _need(seeds, "seeds", torch.int32, dev)
    _need(feats, "feats", None, dev)
    _need(cache_slot, "cache_slot", torch.int32, dev)
    if seeds.dim() != 2:
        raise ValueError("seeds must be [B, S]")
    N = offsets.numel() - 1
    E = indices.numel()
    if feats.shape[0] != N or cache_slot.numel() != N:
        raise ValueError("feats and cache_slot must hold one row / entry per node")
    if membership is not None:
        _need(membership, "membership", torch.int64, dev)
        if membership.numel() != N:
            raise ValueError("membership must hold one word per node")
    B, S = seeds.shape
    R = _row_bytes(feats)
    fanouts = [int(f) for f in fanouts]
    K = len(fanouts)
    if out is not None:
        node_cap, edge_cap = out.nodes.shape[1], out.edge_src.shape[1]
    else:
        bn, be = sample_bounds(N, E, S, fanouts, layered)
        node_cap = bn if node_cap is None else node_cap
        edge_cap = be if edge_cap is None else edge_cap
        out = SampleResult(
            nodes=torch.empty((B, node_cap), dtype=torch.int32, device=dev),
            hop_ptr=np.zeros((B, K + 2), dtype=np.int64),
            edge_src=torch.empty((B, max(edge_cap, 1)), dtype=torch.int32, device=dev),
            edge_dst=torch.empty((B, max(edge_cap, 1)), dtype=torch.int32, device=dev),
            edge_ptr=np.zeros((B, K + 1), dtype=np.int64), sizes={}, timing=None)
    flags = sample_flags(layered, direct, entry_clear, exit_clear)
    ws = _workspace(_L.dg_sample_workspace_bytes(N, B, node_cap, edge_cap, flags), dev,
                    workspace)
    pws = _workspace(_L.dg_sample_pack_workspace_bytes(N, B, node_cap), dev, pack_workspace)
    g = Csr(N, E, offsets.data_ptr(), indices.data_ptr())
    fo = (ctypes.c_int32 * max(K, 1))(*fanouts)

    def call(po, cap, flags_, sz, tm):
        return _L.dg_sample_pack_group(
            ctypes.byref(g), _ptr(seeds), B, S, batch_base, fo, K, rng_seed & (2**64 - 1),
            flags_, node_cap, _ptr(out.nodes), out.hop_ptr.ctypes.data_as(_lib.I64P), edge_cap,
            _ptr(out.edge_src), _ptr(out.edge_dst), out.edge_ptr.ctypes.data_as(_lib.I64P),
            _ptr(membership), _ptr(cache_slot), _ptr(po.loc), _ptr(feats), R, cap,
            _ptr(po.packed) if cap > 0 else None, _ptr(po.packed_ids) if cap > 0 else None,
            _ptr(po.packed_ptr), po.packed_ptr_host.ctypes.data_as(_lib.I64P),
            _ptr(po.unique), po.unique.numel() if po.unique is not None else 0,
            _lib.DG_PACK_ROWS_STREAM if (rows_stream is not None and cap > 0) else 0,
            _ptr(ws), ws.numel(), _ptr(pws), pws.numel(), _stream(stream),
            _stream(rows_stream) if rows_stream is not None else None, ctypes.byref(sz),
            ctypes.byref(tm) if tm is not None else None)

    sz, tm = Sizes(), Timing()
    if pack_out is None:
        loc = torch.empty((B, node_cap), dtype=torch.int32, device=dev)
        ptr = torch.empty(B + 1, dtype=torch.int64, device=dev)
        probe = PackResult(packed=None, packed_ids=None, packed_ptr=ptr,
                           packed_ptr_host=np.zeros(B + 1, dtype=np.int64), loc=loc,
                           unique=None, sizes={}, timing=None, row_bytes=R)
        # size query: no packed capacity; the membership words are left in an
        # unspecified state, so the real call clears them on entry
        st = call(probe, 0, flags & ~_lib.DG_SAMPLE_ENTRY_CLEAR, sz, None)
        if st not in (DG_OK, DG_ECAPACITY):
            check(st)
        if st == DG_ECAPACITY and sz.packed_rows <= 0 and sz.unique_nodes <= 0:
            check(st)  # sampling itself ran out of room
        rows, nu = max(sz.packed_rows, 0), max(sz.unique_nodes, 0)
        pack_out = PackResult(
            packed=None if tables_only else torch.empty((max(rows, 1), R), dtype=torch.uint8,
                                                        device=dev),
            packed_ids=torch.empty(max(rows, 1), dtype=torch.int32, device=dev),
            packed_ptr=ptr, packed_ptr_host=probe.packed_ptr_host, loc=loc,
            unique=torch.empty(max(nu, 1), dtype=torch.int32, device=dev) if with_unique else None,
            sizes={}, timing=None, row_bytes=R)
        flags &= ~_lib.DG_SAMPLE_ENTRY_CLEAR
        sz = Sizes()
    if tuple(pack_out.loc.shape) != (B, node_cap):
        raise ValueError("pack_out.loc must be [B, node_cap], laid out as the node lists")
    cap = pack_out.packed_ids.numel()
    if pack_out.packed is not None and pack_out.packed.numel() < cap * R:
        raise ValueError("packed buffer smaller than packed_ids")
    st = call(pack_out, cap, flags, sz, tm if timing else None)
    out.sizes = sz.as_dict()
    pack_out.sizes = sz.as_dict()
    check(st)
    out.timing = pack_out.timing = tm.as_dict() if timing else None
    return out, pack_out


def assemble_batch(cache: torch.Tensor | None, packed_b: torch.Tensor, loc_b: torch.Tensor,
                   row_bytes: int, out: torch.Tensor | None = None,
                   status: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Feature assembling for one batch (dg_assemble_batch), asynchronous on the
    stream.  Returns `out` viewed as uint8 [n_b, row_bytes]."""
    _need(loc_b, "loc_b", torch.int32)
    dev = loc_b.device
    n = loc_b.numel()
    if out is None:
        out = torch.empty((n, row_bytes), dtype=torch.uint8, device=dev)
    _need(out, "out", None, dev)
    cache_rows = 0
    if cache is not None and cache.numel():
        _need(cache, "cache", None, dev)
        cache_rows = cache.numel() * cache.element_size() // row_bytes
    pr = 0
    if packed_b is not None and packed_b.numel():
        _need(packed_b, "packed_b", None, dev)
        pr = packed_b.numel() * packed_b.element_size() // row_bytes
    if out.numel() * out.element_size() < n * row_bytes:
        raise ValueError("out is too small")
    check(_L.dg_assemble_batch(_ptr(cache) if cache_rows else None, cache_rows,
                               _ptr(packed_b) if pr else None, pr, _ptr(loc_b), n, row_bytes,
                               _ptr(out), _ptr(status), _stream(stream)))
    return out


def assemble_batches(cache: torch.Tensor | None, pr: PackResult, node_count, outs,
                     status: torch.Tensor | None = None, stream=None) -> None:
    """dg_assemble_batches: dg_assemble_batch for every batch of a packing
    result, asynchronous, issued by one library call.  Batch b goes to
    outs[b % len(outs)] (uint8 [>= n_b, row_bytes] buffers, in order on one
    stream)."""
    R = pr.row_bytes
    counts = np.ascontiguousarray(np.asarray(node_count, dtype=np.int64).reshape(-1))
    B = pr.loc.shape[0]
    if counts.shape[0] != B:
        raise ValueError("node_count must have one entry per batch")
    _need(pr.loc, "loc", torch.int32)
    dev = pr.loc.device
    if not len(outs):
        raise ValueError("at least one output buffer is needed")
    nmax = int(counts.max()) if B else 0
    for o in outs:
        _need(o, "out", None, dev)
        if o.numel() * o.element_size() < nmax * R:
            raise ValueError("an output buffer is too small")
    cache_rows = 0
    if cache is not None and cache.numel():
        _need(cache, "cache", None, dev)
        cache_rows = cache.numel() * cache.element_size() // R
    packed = None
    if pr.packed is not None and pr.packed.numel():
        _need(pr.packed, "packed", None, dev)
        packed = pr.packed
    ptr = np.ascontiguousarray(pr.packed_ptr_host, dtype=np.int64)
    optr = (ctypes.c_void_p * len(outs))(*[o.data_ptr() for o in outs])
    check(_L.dg_assemble_batches(_ptr(cache) if cache_rows else None, cache_rows, _ptr(packed),
                                 ptr.ctypes.data_as(_lib.I64P), _ptr(pr.loc), pr.loc.shape[1],
                                 counts.ctypes.data_as(_lib.I64P), B, R, optr, len(outs),
                                 _ptr(status), _stream(stream)))


def cache_by_frequency(membership: torch.Tensor, B: int, cache_rows: int,
                       workspace: torch.Tensor | None = None, stream=None):
    """Access-frequency cache (dg_cache_by_frequency).  Returns (cache_slot
    int32 [N], cache_nodes int32 [cache_rows], cached count)."""
    _need(membership, "membership", torch.int64)
    dev = membership.device
    N = membership.numel()
    slot = torch.empty(N, dtype=torch.int32, device=dev)
    nodes = torch.empty(max(cache_rows, 1), dtype=torch.int32, device=dev)
    ws = _workspace(_L.dg_cache_workspace_bytes(N), dev, workspace)
    cached = ctypes.c_int64()
    check(_L.dg_cache_by_frequency(_ptr(membership), N, B, cache_rows, _ptr(slot), _ptr(nodes),
                                   ctypes.byref(cached), _ptr(ws), ws.numel(), _stream(stream)))
    return slot, nodes[:cache_rows], cached.value


def gather_rows(feats: torch.Tensor, ids: torch.Tensor, out: torch.Tensor | None = None,
                status: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """out[i] = feats[ids[i]] as bytes (dg_gather_rows), asynchronous.  Returns
    out viewed as uint8 [n, row_bytes]."""
    _need(feats, "feats", None)
    _need(ids, "ids", torch.int32, feats.device)
    R = _row_bytes(feats)
    n = ids.numel()
    if out is None:
        out = torch.empty((n, R), dtype=torch.uint8, device=feats.device)
    _need(out, "out", None, feats.device)
    if out.numel() * out.element_size() < n * R:
        raise ValueError("out is too small")
    check(_L.dg_gather_rows(_ptr(feats), feats.shape[0], R, _ptr(ids), n, _ptr(out),
                            _ptr(status), _stream(stream)))
    return out


def pack_individual(feats: torch.Tensor, packed_ids: torch.Tensor, packed_ptr_host,
                    packed: torch.Tensor, stream=None) -> torch.Tensor:
    """Individual packing (the paper's naive scheme, Fig. 6a): one row gather
    per mini-batch over its packed IDs, reading a row once per mini-batch that
    needs it.  Fills the same packed buffer dg_pack_group would."""
    R = _row_bytes(feats)
    for b in range(len(packed_ptr_host) - 1):
        lo, hi = int(packed_ptr_host[b]), int(packed_ptr_host[b + 1])
        if hi > lo:
            gather_rows(feats, packed_ids[lo:hi], out=packed[lo:hi], stream=stream)
    return packed


def minhash_order(membership: torch.Tensor, B: int, entries: torch.Tensor, perms: torch.Tensor,
                  workspace: torch.Tensor | None = None, stream=None):
    """Disk-cache reordering by MinHash (dg_minhash_order).  perms: int32
    [k, B] on the GPU, each row a permutation of 0..B-1.  Returns (order
    int32 [m], signature int32 [m], -1 = in no sample)."""
    _need(membership, "membership", torch.int64)
    dev = membership.device
    _need(entries, "entries", torch.int32, dev)
    _need(perms, "perms", torch.int32, dev)
    if perms.dim() != 2 or perms.shape[1] != B:
        raise ValueError("perms must be [k, B]")
    m = entries.numel()
    order = torch.empty(max(m, 1), dtype=torch.int32, device=dev)
    sig = torch.empty(max(m, 1), dtype=torch.int32, device=dev)
    ws = _workspace(_L.dg_minhash_workspace_bytes(m), dev, workspace)
    check(_L.dg_minhash_order(_ptr(membership), membership.numel(), B, _ptr(entries), m,
                              _ptr(perms), perms.shape[0], _ptr(order), _ptr(sig), _ptr(ws),
                              ws.numel(), _stream(stream)))
    return order[:m], sig[:m]
