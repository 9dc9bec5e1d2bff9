"""Python binding of libmsparse (vertical-slash sparse attention on MI355X).

Argument marshalling only: every step of the hot path runs in the library's
HIP kernels.  PyTorch provides device memory and the current stream.  The
functions keep the C names without the ``msparse_`` prefix and raise
MsparseError on a non-zero status.  Nothing here falls back to another
implementation: if libmsparse.so is missing the first call raises.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
# MSPARSE_LIBRARY selects another build of the same library (the host
# AddressSanitizer build of build.build_asan, for the host-side tests)
LIB_PATH = os.environ.get("MSPARSE_LIBRARY") or os.path.join(HERE, "libmsparse.so")

STRIPED = 0
ZIGZAG = 1
_LAYOUTS = {"striped": STRIPED, "zigzag": ZIGZAG}

c_i32, c_i64, c_f32, c_vp, c_sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t


class Dims(ctypes.Structure):
    _fields_ = [("batch", c_i32), ("seq_q", c_i32), ("seq_k", c_i32), ("heads_q", c_i32), ("heads_kv", c_i32),
                ("head_dim", c_i32), ("block", c_i32), ("causal", c_i32), ("scale", c_f32)]


class Ring(ctypes.Structure):
    _fields_ = [("world", c_i32), ("rank", c_i32), ("step", c_i32), ("layout", c_i32), ("inner", c_i32)]


class IndexStruct(ctypes.Structure):
    _fields_ = [("blk_ptr", c_vp), ("blk_idx", c_vp), ("blk_cap", c_i64),
                ("col_ptr", c_vp), ("col_idx", c_vp), ("col_cap", c_i64),
                ("kblk_ptr", c_vp), ("kblk_idx", c_vp),
                ("vcol_ptr", c_vp), ("vcol_idx", c_vp), ("vcol_cap", c_i64),
                ("diag_bits", c_vp), ("q_blk_global", c_vp), ("k_blk_global", c_vp), ("overflow", c_vp),
                ("world", c_i32)]


class TraceEntry(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", c_i32), ("total_ms", ctypes.c_double)]


_P = ctypes.POINTER
_SIGS = {
    "msparse_trace_enable": (None, [c_i32]),
    "msparse_trace_read": (c_i32, [_P(TraceEntry), c_i32]),
    "msparse_strerror": (ctypes.c_char_p, [c_i32]),
    "msparse_last_error": (ctypes.c_char_p, []),
    "msparse_estimate_workspace": (c_sz, [_P(Dims), c_i32, c_i32, c_i32]),
    "msparse_estimate": (c_i32, [_P(Dims), c_vp, c_vp, c_i32, c_i32, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, c_sz, c_vp]),
    "msparse_estimate_topp_workspace": (c_sz, [_P(Dims), c_i32, c_i32, c_i32]),
    "msparse_ring_shard": (c_i32, [c_i32, c_i32, c_i32, c_i32]),
    "msparse_mfma_peak_probe": (c_i32, [c_i32, c_i32, c_i32, c_vp, c_vp]),
    "msparse_ring_work": (c_i32, [_P(Dims), c_vp, c_i32, c_vp, c_i32, c_i32, c_i32, c_vp, c_vp, c_vp, c_sz, c_vp]),
    "msparse_estimate_topp": (c_i32, [_P(Dims), c_vp, c_vp, c_i32, ctypes.c_double, ctypes.c_double, c_i32, c_i32,
                                      c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_sz, c_vp]),
    "msparse_index_workspace": (c_sz, [_P(Dims), c_i32, c_i32, _P(Ring)]),
    "msparse_index_count": (c_i32, [_P(Dims), c_vp, c_i32, c_vp, c_i32, _P(Ring), _P(c_i64), _P(c_i64), _P(c_i64),
                                    c_vp, c_sz, c_vp]),
    "msparse_build_index": (c_i32, [_P(Dims), c_vp, c_i32, c_vp, c_i32, _P(Ring), _P(IndexStruct), c_vp, c_sz, c_vp]),
    "msparse_build_index_noalloc": (c_i32, [_P(Dims), c_vp, c_i32, c_vp, c_i32, _P(Ring), _P(IndexStruct), c_vp]),
    "msparse_index_count_build": (c_i32, [_P(Dims), c_vp, c_i32, c_vp, c_i32, _P(Ring), _P(IndexStruct), _P(c_i64),
                                          _P(c_i64), _P(c_i64), c_vp, c_sz, c_vp]),
    "msparse_attn_fwd_workspace": (c_sz, [_P(Dims)]),
    "msparse_attn_fwd": (c_i32, [_P(Dims), c_vp, c_vp, c_vp, _P(IndexStruct), c_vp, c_vp, c_vp, c_vp, c_sz, c_vp]),
    "msparse_attn_fwd_merge": (c_i32, [_P(Dims), c_vp, c_vp, c_vp, _P(IndexStruct), c_vp, c_vp, c_vp, c_i32, c_vp,
                                       c_sz, c_vp]),
    "msparse_merge_out_lse": (c_i32, [_P(Dims), c_vp, c_vp, c_vp, c_vp, c_vp, c_i32, c_vp]),
    "msparse_attn_bwd_workspace": (c_sz, [_P(Dims), c_i64]),
    "msparse_attn_bwd": (c_i32, [_P(Dims), c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, _P(IndexStruct), c_vp, c_vp,
                                 c_vp, c_i32, c_vp, c_sz, c_vp]),
}

_lib = None


class MsparseError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(msg)
        self.status = status


def lib() -> ctypes.CDLL:
    """Load libmsparse.so (built in-tree by build.py); raise if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run paper_2510_18830_amd.build.build()")
        so = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(so, name)
            fn.restype = res
            fn.argtypes = args
        _lib = so
    return _lib


def _check(status: int):
    if status != 0:
        L = lib()
        raise MsparseError(status, f"{L.msparse_strerror(status).decode()}: {L.msparse_last_error().decode()}")


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def make_dims(batch, seq_q, heads_q, heads_kv, head_dim, seq_k=None, scale=0.0) -> Dims:
    return Dims(batch, seq_q, seq_q if seq_k is None else seq_k, heads_q, heads_kv, head_dim, 64, 1, scale)


def make_ring(world=1, rank=0, step=0, layout="striped", inner=0):
    """A ring step descriptor; inner > 1 selects the hierarchical step order (cards per node)."""
    if world == 1 and rank == 0 and step == 0:
        return None
    return Ring(world, rank, step, _LAYOUTS[layout] if isinstance(layout, str) else layout, inner)


def ring_shard(world, inner, rank, step) -> int:
    """msparse_ring_shard: the worker whose KV shard `rank` holds at `step` (-1 if invalid)."""
    return int(lib().msparse_ring_shard(world, inner, rank, step))


def ring_work(dims, v_idx, s_idx, world, layout="striped", workspace=None, stream=None):
    """msparse_ring_work: (tiles, cols) int64 [world, world] on the device, query worker x KV shard."""
    k_v, k_s = v_idx.shape[-1], s_idx.shape[-1]
    if workspace is None:
        workspace = _workspace(index_workspace_bytes(dims, k_v, k_s), v_idx.device)
    tiles = torch.empty((world, world), dtype=torch.int64, device=v_idx.device)
    cols = torch.empty_like(tiles)
    _check(lib().msparse_ring_work(ctypes.byref(dims), _p(v_idx), k_v, _p(s_idx), k_s, world,
                                   _LAYOUTS[layout] if isinstance(layout, str) else layout, _p(tiles), _p(cols),
                                   _p(workspace), workspace.numel(), _stream(stream)))
    return tiles, cols


def _ring_ptr(ring):
    return ctypes.byref(ring) if ring is not None else None


def _workspace(nbytes, device):
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


# ------------------------------------------------------------------ estimate
def estimate(dims: Dims, q, k, last_q, k_v, k_s, v_idx=None, s_idx=None, v_score=None, s_score=None,
             workspace=None, stream=None):
    """msparse_estimate: returns (v_idx, s_idx) int32 [B, Hq, k]."""
    BH = (dims.batch, dims.heads_q)
    v_idx = torch.empty(BH + (k_v,), dtype=torch.int32, device=q.device) if v_idx is None else v_idx
    s_idx = torch.empty(BH + (k_s,), dtype=torch.int32, device=q.device) if s_idx is None else s_idx
    if workspace is None:
        workspace = _workspace(lib().msparse_estimate_workspace(ctypes.byref(dims), last_q, k_v, k_s), q.device)
    _check(lib().msparse_estimate(ctypes.byref(dims), _p(q), _p(k), last_q, k_v, k_s, _p(v_idx), _p(s_idx),
                                  _p(v_score), _p(s_score), _p(workspace), workspace.numel(), _stream(stream)))
    return v_idx, s_idx


def estimate_topp(dims: Dims, q, k, last_q, p_v, p_s, kmax_v, kmax_s, v_score=None, s_score=None, workspace=None,
                  stream=None):
    """msparse_estimate_topp: returns (v_idx [B, Hq, kmax_v], s_idx [B, Hq, kmax_s], v_cnt, s_cnt [B, Hq]), int32;
    unused slots of the index lists hold -1."""
    BH = (dims.batch, dims.heads_q)
    v_idx = torch.empty(BH + (kmax_v,), dtype=torch.int32, device=q.device)
    s_idx = torch.empty(BH + (kmax_s,), dtype=torch.int32, device=q.device)
    v_cnt = torch.empty(BH, dtype=torch.int32, device=q.device)
    s_cnt = torch.empty(BH, dtype=torch.int32, device=q.device)
    if workspace is None:
        workspace = _workspace(lib().msparse_estimate_topp_workspace(ctypes.byref(dims), last_q, kmax_v, kmax_s),
                               q.device)
    _check(lib().msparse_estimate_topp(ctypes.byref(dims), _p(q), _p(k), last_q, float(p_v), float(p_s), kmax_v,
                                       kmax_s, _p(v_idx), _p(s_idx), _p(v_cnt), _p(s_cnt), _p(v_score), _p(s_score),
                                       _p(workspace), workspace.numel(), _stream(stream)))
    return v_idx, s_idx, v_cnt, s_cnt


# ------------------------------------------------------------------ index
@dataclass
class SparseIndex:
    """Device arrays of one msparse_index plus the C struct that points at them."""
    tensors: dict
    struct: IndexStruct
    nqb: int
    nkb: int

    def __getitem__(self, key):
        return self.tensors[key]


def index_workspace_bytes(dims, k_v, k_s, ring=None):
    return int(lib().msparse_index_workspace(ctypes.byref(dims), k_v, k_s, _ring_ptr(ring)))


def index_count(dims, v_idx, s_idx, ring=None, workspace=None, stream=None):
    """msparse_index_count (waits for the GPU): (blk_nnz, col_nnz, vcol_nnz)."""
    k_v, k_s = v_idx.shape[-1], s_idx.shape[-1]
    if workspace is None:
        workspace = _workspace(index_workspace_bytes(dims, k_v, k_s, ring), v_idx.device)
    out = [c_i64(0), c_i64(0), c_i64(0)]
    _check(lib().msparse_index_count(ctypes.byref(dims), _p(v_idx), k_v, _p(s_idx), k_s, _ring_ptr(ring),
                                     *[ctypes.byref(x) for x in out], _p(workspace), workspace.numel(),
                                     _stream(stream)))
    return tuple(int(x.value) for x in out)


def alloc_index(dims, blk_cap, col_cap, vcol_cap, device, world=1) -> SparseIndex:
    BH = dims.batch * dims.heads_q
    nqb, nkb = dims.seq_q // 64, dims.seq_k // 64
    nb = nqb * world
    i64, i32 = torch.int64, torch.int32
    t = {
        "blk_ptr": torch.empty(BH * nqb + 1, dtype=i64, device=device),
        "blk_idx": torch.empty(max(blk_cap, 1), dtype=i32, device=device),
        "col_ptr": torch.empty(BH * nqb + 1, dtype=i64, device=device),
        "col_idx": torch.empty(max(col_cap, 1), dtype=i32, device=device),
        "kblk_ptr": torch.empty(BH * nkb + 1, dtype=i64, device=device),
        "kblk_idx": torch.empty(max(blk_cap, 1), dtype=i32, device=device),
        "vcol_ptr": torch.empty(BH + 1, dtype=i64, device=device),
        "vcol_idx": torch.empty(max(vcol_cap, 1), dtype=i32, device=device),
        "diag_bits": torch.empty(BH * ((nb + 31) // 32), dtype=i32, device=device),
        "q_blk_global": torch.empty(nqb, dtype=i32, device=device),
        "k_blk_global": torch.empty(nkb, dtype=i32, device=device),
        "overflow": torch.zeros(1, dtype=i32, device=device),
    }
    s = IndexStruct(_p(t["blk_ptr"]), _p(t["blk_idx"]), blk_cap, _p(t["col_ptr"]), _p(t["col_idx"]), col_cap,
                    _p(t["kblk_ptr"]), _p(t["kblk_idx"]), _p(t["vcol_ptr"]), _p(t["vcol_idx"]), vcol_cap,
                    _p(t["diag_bits"]), _p(t["q_blk_global"]), _p(t["k_blk_global"]), _p(t["overflow"]), world)
    return SparseIndex(t, s, nqb, nkb)


def build_index(dims, v_idx, s_idx, index: SparseIndex, ring=None, workspace=None, stream=None):
    """msparse_build_index into a preallocated SparseIndex."""
    k_v, k_s = v_idx.shape[-1], s_idx.shape[-1]
    if workspace is None:
        workspace = _workspace(index_workspace_bytes(dims, k_v, k_s, ring), v_idx.device)
    _check(lib().msparse_build_index(ctypes.byref(dims), _p(v_idx), k_v, _p(s_idx), k_s, _ring_ptr(ring),
                                     ctypes.byref(index.struct), _p(workspace), workspace.numel(), _stream(stream)))
    return index


def index_count_build(dims, v_idx, s_idx, index: SparseIndex, ring=None, workspace=None, stream=None):
    """msparse_index_count_build (waits for the GPU once): returns (built, (blk_nnz, col_nnz, vcol_nnz));
    built is False when a capacity of `index` was too small (nothing filled, its overflow flag set)."""
    k_v, k_s = v_idx.shape[-1], s_idx.shape[-1]
    if workspace is None:
        workspace = _workspace(index_workspace_bytes(dims, k_v, k_s, ring), v_idx.device)
    out = [c_i64(0), c_i64(0), c_i64(0)]
    st = lib().msparse_index_count_build(ctypes.byref(dims), _p(v_idx), k_v, _p(s_idx), k_s, _ring_ptr(ring),
                                         ctypes.byref(index.struct), *[ctypes.byref(x) for x in out],
                                         _p(workspace), workspace.numel(), _stream(stream))
    if st == -3:
        return False, tuple(int(x.value) for x in out)
    _check(st)
    return True, tuple(int(x.value) for x in out)


def build_index_noalloc(dims, v_idx, s_idx, index: SparseIndex, ring=None, stream=None):
    """msparse_build_index_noalloc: the index build with the library's fixed scratch (no workspace)."""
    k_v, k_s = v_idx.shape[-1], s_idx.shape[-1]
    _check(lib().msparse_build_index_noalloc(ctypes.byref(dims), _p(v_idx), k_v, _p(s_idx), k_s, _ring_ptr(ring),
                                             ctypes.byref(index.struct), _stream(stream)))
    return index


def make_index(dims, v_idx, s_idx, ring=None, stream=None) -> SparseIndex:
    """Count (one GPU wait), allocate exactly, then build."""
    k_v, k_s = v_idx.shape[-1], s_idx.shape[-1]
    ws = _workspace(index_workspace_bytes(dims, k_v, k_s, ring), v_idx.device)
    blk, col, vcol = index_count(dims, v_idx, s_idx, ring, ws, stream)
    idx = alloc_index(dims, blk, col, vcol, v_idx.device, ring.world if ring is not None else 1)
    return build_index(dims, v_idx, s_idx, idx, ring, ws, stream)


# ------------------------------------------------------------------ attention
def attn_fwd_workspace_bytes(dims):
    return int(lib().msparse_attn_fwd_workspace(ctypes.byref(dims)))


def attn_fwd(dims, q, k, v, index: SparseIndex, out=None, lse=None, out_f32=None, stream=None, bf16_out=True,
             workspace=None):
    """msparse_attn_fwd: returns (out bf16 [B,Hq,Nq,d] or None, lse fp32 [B,Hq,Nq]); out_f32 is optional."""
    if out is None and bf16_out:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty(q.shape[:-1], dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = _workspace(attn_fwd_workspace_bytes(dims), q.device)
    _check(lib().msparse_attn_fwd(ctypes.byref(dims), _p(q), _p(k), _p(v), ctypes.byref(index.struct), _p(out),
                                  _p(lse), _p(out_f32), _p(workspace), workspace.numel(), _stream(stream)))
    return out, lse


def attn_fwd_merge(dims, q, k, v, index: SparseIndex, o_acc, lse_acc, out_bf16=None, first=False, workspace=None,
                   stream=None):
    """msparse_attn_fwd_merge: one ring step's forward merged into the running (o_acc, lse_acc)."""
    if workspace is None:
        workspace = _workspace(attn_fwd_workspace_bytes(dims), q.device)
    _check(lib().msparse_attn_fwd_merge(ctypes.byref(dims), _p(q), _p(k), _p(v), ctypes.byref(index.struct),
                                        _p(o_acc), _p(lse_acc), _p(out_bf16), int(bool(first)), _p(workspace),
                                        workspace.numel(), _stream(stream)))


def merge_out_lse(dims, o_part, lse_part, o_acc, lse_acc, out_bf16=None, first=False, stream=None):
    _check(lib().msparse_merge_out_lse(ctypes.byref(dims), _p(o_part), _p(lse_part), _p(o_acc), _p(lse_acc),
                                       _p(out_bf16), int(bool(first)), _stream(stream)))


def attn_bwd_workspace_bytes(dims, vcol_cap):
    return int(lib().msparse_attn_bwd_workspace(ctypes.byref(dims), vcol_cap))


def attn_bwd(dims, q, k, v, out, dout, lse, index: SparseIndex, dq=None, dk=None, dv=None, dq_accumulate=False,
             out_f32=None, workspace=None, stream=None, reuse_qrows=False):
    """msparse_attn_bwd: returns (dq, dk, dv) fp32.  reuse_qrows: the workspace still holds the query-side
    data of the previous call of the same ring worker (MSPARSE_BWD_REUSE_QROWS)."""
    f32 = torch.float32
    dq = torch.empty(q.shape, dtype=f32, device=q.device) if dq is None else dq
    dk = torch.empty(k.shape, dtype=f32, device=q.device) if dk is None else dk
    dv = torch.empty(v.shape, dtype=f32, device=q.device) if dv is None else dv
    if workspace is None:
        workspace = _workspace(attn_bwd_workspace_bytes(dims, index.struct.vcol_cap), q.device)
    _check(lib().msparse_attn_bwd(ctypes.byref(dims), _p(q), _p(k), _p(v), _p(out), _p(out_f32), _p(dout), _p(lse),
                                  ctypes.byref(index.struct), _p(dq), _p(dk), _p(dv),
                                  int(bool(dq_accumulate)) | (2 if reuse_qrows else 0),
                                  _p(workspace), workspace.numel(), _stream(stream)))
    return dq, dk, dv


def default_scale(head_dim: int) -> float:
    return 1.0 / math.sqrt(head_dim)


# ------------------------------------------------------------------ tracing
def mfma_peak_tflops(waves_per_simd: int = 4, iters: int = 20000, device=None, random: bool = False) -> float:
    """Achievable dense fp16 MFMA rate in TFLOP/s (msparse_mfma_peak_probe, timed with HIP events);
    random=True cycles random operands (real data's switching) instead of one constant pair."""
    device = device or torch.device("cuda", torch.cuda.current_device())
    cus = torch.cuda.get_device_properties(device).multi_processor_count
    out = torch.empty(cus * waves_per_simd * 256, dtype=torch.float32, device=device)
    iters = (iters + 7) // 8 * 8
    _check(lib().msparse_mfma_peak_probe(waves_per_simd, 104, int(random), _p(out), _stream(None)))
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    _check(lib().msparse_mfma_peak_probe(waves_per_simd, iters, int(random), _p(out), _stream(None)))
    b.record()
    torch.cuda.synchronize()
    flops = cus * waves_per_simd * 4 * iters * 4 * 32768.0
    return flops / (a.elapsed_time(b) * 1e-3) / 1e12


def trace_enable(on: bool = True):
    """Bracket every library kernel launch with HIP events (for measurement)."""
    lib().msparse_trace_enable(int(bool(on)))


def trace_read() -> dict:
    """{kernel name: (launches, total ms)} since the last read (waits for the events)."""
    cap = 64
    buf = (TraceEntry * cap)()
    n = lib().msparse_trace_read(buf, cap)
    return {buf[i].name.decode(): (int(buf[i].launches), float(buf[i].total_ms)) for i in range(min(n, cap))}
