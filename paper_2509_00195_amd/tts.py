"""Python binding of libtts (argument marshalling only).

Every function forwards to the C ABI of ``include/tts.h`` with the same
name; all computation happens in the HIP library. Device buffers are passed
as torch tensors (their ``data_ptr()``) or raw integer addresses; host arrays
as numpy int32 arrays. The library is loaded from this package's directory;
if it has not been built, loading raises instead of falling back to
anything else.
"""

from __future__ import annotations

import ctypes as C
import os
from typing import Optional

import numpy as np

# TTS_LIBRARY names another build of the same library (the sanitized CPU-test
# build); by default the one built in this package's directory.
LIB_PATH = os.environ.get("TTS_LIBRARY") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtts.so")

TTS_OK = 0
TTS_ERR_INVALID_ARG = -1
TTS_ERR_UNSUPPORTED = -2
TTS_ERR_OUT_OF_RANGE = -3
TTS_ERR_WORKSPACE = -4
TTS_ERR_HIP = -5
TTS_ERR_NOMEM = -6
STATUS_NAMES = {0: "TTS_OK", -1: "TTS_ERR_INVALID_ARG", -2: "TTS_ERR_UNSUPPORTED", -3: "TTS_ERR_OUT_OF_RANGE",
                -4: "TTS_ERR_WORKSPACE", -5: "TTS_ERR_HIP", -6: "TTS_ERR_NOMEM"}

TTS_F32, TTS_BF16, TTS_FP8_E4M3 = 0, 1, 2
DTYPES = {"f32": TTS_F32, "bf16": TTS_BF16, "fp8": TTS_FP8_E4M3}

EXPORTED = [
    "tts_build_prefix_meta", "tts_prefix_meta_destroy", "tts_prefix_meta_export", "tts_prefix_meta_coverage",
    "tts_prefix_meta_stats", "tts_plan_units_host", "tts_paged_decode_workspace_size", "tts_paged_decode_attn",
    "tts_prefix_decode_workspace_size", "tts_prefix_decode_attn", "tts_prefix_decode_attn_noalloc",
    "tts_prefix_decode_partials",
    "tts_prefix_decode_merge", "tts_append_kv", "tts_copy_blocks", "tts_fork_tables", "tts_kv_alloc_time",
    "tts_kv_alloc_search", "tts_prefix_schedule", "tts_build_verify_meta", "tts_prefix_verify_attn",
    "tts_last_error", "tts_fork_prefix_meta", "tts_truncated_lengths",
]


class TTSError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class tts_attn_desc(C.Structure):
    _fields_ = [("num_q_heads", C.c_int32), ("num_kv_heads", C.c_int32), ("head_dim", C.c_int32),
                ("block_size", C.c_int32), ("q_dtype", C.c_int), ("kv_dtype", C.c_int), ("out_dtype", C.c_int),
                ("scale", C.c_float)]


class tts_model_cost(C.Structure):
    _fields_ = [("params", C.c_double), ("weight_bytes", C.c_double), ("kv_bytes_per_token", C.c_double),
                ("num_layers", C.c_int32), ("attn_dim", C.c_int32)]


class tts_alloc_problem(C.Structure):
    _fields_ = [("verifier", tts_model_cost), ("generator", tts_model_cost), ("num_requests", C.c_int64),
                ("verify_len", C.c_int64), ("decode_len", C.c_int64), ("mem_bytes", C.c_double),
                ("peak_flops", C.c_double), ("peak_bw", C.c_double)]


class tts_alloc_result(C.Structure):
    _fields_ = [("b_pre", C.c_int64), ("b_dec", C.c_int64), ("t_tot", C.c_double), ("t_pre", C.c_double),
                ("t_dec", C.c_double)]


class tts_prefix_meta_view(C.Structure):
    _fields_ = [("num_seqs", C.c_int32), ("num_segs", C.c_int32), ("perm", C.POINTER(C.c_int32)),
                ("seg_req", C.POINTER(C.c_int32)), ("seg_parent", C.POINTER(C.c_int32)),
                ("seg_lblock_begin", C.POINTER(C.c_int32)), ("seg_nblocks", C.POINTER(C.c_int32)),
                ("seg_beam_begin", C.POINTER(C.c_int32)), ("seg_beam_end", C.POINTER(C.c_int32)),
                ("tail_lblock", C.POINTER(C.c_int32)), ("unique_blocks", C.c_int64),
                ("unique_tokens", C.c_int64)]


_lib = None


def load() -> C.CDLL:
    """Load libtts.so (raises if it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} not built: run __graft_entry__.build() or python -m paper_2509_00195_amd.build")
    # Bind to the HIP runtime PyTorch already uses (same soname): the caller's
    # device memory and streams come from it.
    try:
        import torch  # noqa: F401
    except ImportError:  # pragma: no cover - C callers without torch
        pass
    lib = C.CDLL(LIB_PATH)
    P, I32, I64, VP = C.POINTER, C.c_int32, C.c_int64, C.c_void_p
    pi32 = P(C.c_int32)
    lib.tts_last_error.restype = C.c_char_p
    lib.tts_last_error.argtypes = []
    lib.tts_build_prefix_meta.restype = C.c_int
    lib.tts_build_prefix_meta.argtypes = [I32, pi32, I32, pi32, I32, pi32, I32, I32, P(tts_attn_desc), VP, P(VP)]
    lib.tts_build_verify_meta.restype = C.c_int
    lib.tts_build_verify_meta.argtypes = [I32, pi32, I32, pi32, I32, pi32, I32, I32, I32, P(tts_attn_desc), VP,
                                          P(VP)]
    lib.tts_fork_prefix_meta.restype = C.c_int
    lib.tts_fork_prefix_meta.argtypes = [VP, I32, pi32, I32, pi32, I32, pi32, I32, I32, VP, P(VP)]
    lib.tts_truncated_lengths.restype = C.c_int
    lib.tts_truncated_lengths.argtypes = [I32, pi32, pi32, pi32, I32, C.c_double, C.c_double, P(C.c_double), pi32]
    lib.tts_prefix_meta_destroy.restype = None
    lib.tts_prefix_meta_destroy.argtypes = [VP]
    lib.tts_prefix_meta_export.restype = C.c_int
    lib.tts_prefix_meta_export.argtypes = [VP, P(tts_prefix_meta_view)]
    lib.tts_prefix_meta_coverage.restype = C.c_int
    lib.tts_prefix_meta_coverage.argtypes = [VP, pi32, pi32, I64, P(I64)]
    lib.tts_prefix_meta_stats.restype = C.c_int
    lib.tts_prefix_meta_stats.argtypes = [VP, P(I64), P(I64)]
    lib.tts_plan_units_host.restype = C.c_int
    lib.tts_plan_units_host.argtypes = [I32, pi32, I32, pi32, I32, pi32, I32, I32, P(tts_attn_desc), I32, pi32, I64,
                                        P(I64), P(I64)]
    lib.tts_paged_decode_workspace_size.restype = C.c_size_t
    lib.tts_paged_decode_workspace_size.argtypes = [P(tts_attn_desc), I32, I32]
    lib.tts_paged_decode_attn.restype = C.c_int
    lib.tts_paged_decode_attn.argtypes = [P(tts_attn_desc), I32, VP, VP, VP, VP, VP, VP, I32, VP, I32, I32, VP, VP,
                                          C.c_size_t, VP]
    lib.tts_prefix_decode_workspace_size.restype = C.c_size_t
    lib.tts_prefix_decode_workspace_size.argtypes = [P(tts_attn_desc), VP]
    lib.tts_prefix_decode_attn.restype = C.c_int
    lib.tts_prefix_decode_attn.argtypes = [P(tts_attn_desc), VP, VP, VP, VP, VP, VP, VP, I32, VP, I32, VP, VP,
                                           C.c_size_t, VP]
    lib.tts_prefix_verify_attn.restype = C.c_int
    lib.tts_prefix_verify_attn.argtypes = lib.tts_prefix_decode_attn.argtypes
    lib.tts_prefix_decode_attn_noalloc.restype = C.c_int
    lib.tts_prefix_decode_attn_noalloc.argtypes = [P(tts_attn_desc), VP, VP, VP, VP, VP, VP, VP, I32, VP, I32, VP,
                                                   VP]
    lib.tts_prefix_decode_partials.restype = C.c_int
    lib.tts_prefix_decode_partials.argtypes = lib.tts_prefix_decode_attn.argtypes
    lib.tts_prefix_decode_merge.restype = C.c_int
    lib.tts_prefix_decode_merge.argtypes = [P(tts_attn_desc), VP, VP, VP, VP, C.c_size_t, VP]
    lib.tts_append_kv.restype = C.c_int
    lib.tts_append_kv.argtypes = [P(tts_attn_desc), I32, VP, VP, VP, I32, VP, I32, VP, VP, VP, VP, VP]
    lib.tts_copy_blocks.restype = C.c_int
    lib.tts_copy_blocks.argtypes = [P(tts_attn_desc), I32, VP, I32, VP, VP, VP, VP, VP]
    lib.tts_kv_alloc_time.restype = C.c_int
    lib.tts_kv_alloc_time.argtypes = [P(tts_alloc_problem), I64, I64, P(tts_alloc_result)]
    lib.tts_kv_alloc_search.restype = C.c_int
    lib.tts_kv_alloc_search.argtypes = [P(tts_alloc_problem), P(tts_alloc_result)]
    lib.tts_prefix_schedule.restype = C.c_int
    lib.tts_prefix_schedule.argtypes = [I32, pi32, pi32, I32, P(C.c_int64), I64, pi32, pi32, pi32, P(I64), P(I64)]
    lib.tts_fork_tables.restype = C.c_int
    lib.tts_fork_tables.argtypes = [I32, pi32, I32, pi32, I32, I32, pi32, pi32, pi32, I32, pi32, pi32, pi32, pi32]
    _lib = lib
    return lib


def _check(status: int):
    if status != TTS_OK:
        raise TTSError(status, load().tts_last_error().decode())


def make_desc(num_q_heads, num_kv_heads, head_dim, block_size=16, q_dtype="bf16", kv_dtype="bf16",
              out_dtype="f32", scale=0.0) -> tts_attn_desc:
    dt = lambda x: DTYPES[x] if isinstance(x, str) else int(x)  # noqa: E731
    return tts_attn_desc(num_q_heads, num_kv_heads, head_dim, block_size, dt(q_dtype), dt(kv_dtype), dt(out_dtype),
                         float(scale))


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        if not x.is_contiguous():
            raise ValueError("device tensors must be contiguous")
        return x.data_ptr()
    raise TypeError(f"cannot pass {type(x)} as a device pointer")


def _stream(stream) -> Optional[int]:
    if stream is None:
        try:
            import torch

            if torch.cuda.is_available():
                return torch.cuda.current_stream().cuda_stream
        except Exception:  # pragma: no cover - torch missing
            pass
        return None
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _host_i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _as_i32p(a: np.ndarray):
    return a.ctypes.data_as(C.POINTER(C.c_int32))


class PrefixMeta:
    """Owning wrapper of a ``tts_prefix_meta*`` handle."""

    def __init__(self, handle: int, desc: Optional[tts_attn_desc]):
        self.handle = handle
        self.desc = desc

    def __del__(self):
        self.destroy()

    def destroy(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.tts_prefix_meta_destroy(self.handle)
            self.handle = None

    def export(self) -> dict:
        return tts_prefix_meta_export(self)

    def coverage(self, seq_lens_host=None) -> np.ndarray:
        return tts_prefix_meta_coverage(self, seq_lens_host)

    def stats(self):
        return tts_prefix_meta_stats(self)


def tts_build_prefix_meta(req_seq_offsets, block_tables, seq_lens, block_size: int, num_blocks: int,
                          desc: Optional[tts_attn_desc] = None, stream=None) -> PrefixMeta:
    lib = load()
    offs = _host_i32(req_seq_offsets)
    tables = _host_i32(block_tables)
    lens = _host_i32(seq_lens)
    s = lens.shape[0]
    maxb = tables.shape[1] if tables.ndim == 2 else 0
    h = C.c_void_p()
    _check(lib.tts_build_prefix_meta(offs.shape[0] - 1, _as_i32p(offs), s, _as_i32p(tables), maxb, _as_i32p(lens),
                                     block_size, num_blocks, C.byref(desc) if desc is not None else None,
                                     _stream(stream) if desc is not None else None, C.byref(h)))
    return PrefixMeta(h.value, desc)


def tts_fork_prefix_meta(prev: PrefixMeta, req_seq_offsets, block_tables, seq_lens, block_size: int, num_blocks: int,
                         stream=None) -> PrefixMeta:
    lib = load()
    offs = _host_i32(req_seq_offsets)
    tables = _host_i32(block_tables)
    lens = _host_i32(seq_lens)
    s = lens.shape[0]
    maxb = tables.shape[1] if tables.ndim == 2 else 0
    h = C.c_void_p()
    _check(lib.tts_fork_prefix_meta(prev.handle, offs.shape[0] - 1, _as_i32p(offs), s, _as_i32p(tables), maxb,
                                    _as_i32p(lens), block_size, num_blocks, _stream(stream), C.byref(h)))
    return PrefixMeta(h.value, prev.desc)


def tts_truncated_lengths(child_parent, parent_lens, parent_spec, ratio: float, sigma: float, z) -> np.ndarray:
    """Lengths of the children of a duplication step (originals whole, duplicates truncated)."""
    lib = load()
    cp = _host_i32(child_parent)
    pl = _host_i32(parent_lens)
    ps = _host_i32(parent_spec)
    zz = np.ascontiguousarray(z, dtype=np.float64)
    n = cp.shape[0]
    if zz.shape[0] != n or ps.shape[0] != pl.shape[0]:
        raise ValueError("z needs one draw per child and parent_spec one entry per parent")
    out = np.zeros(n, np.int32)
    _check(lib.tts_truncated_lengths(n, _as_i32p(cp), _as_i32p(pl), _as_i32p(ps), pl.shape[0], float(ratio),
                                     float(sigma), zz.ctypes.data_as(C.POINTER(C.c_double)), _as_i32p(out)))
    return out


def tts_build_verify_meta(req_seq_offsets, block_tables, seq_lens, q_len: int, block_size: int, num_blocks: int,
                          desc: Optional[tts_attn_desc] = None, stream=None) -> PrefixMeta:
    lib = load()
    offs = _host_i32(req_seq_offsets)
    tables = _host_i32(block_tables)
    lens = _host_i32(seq_lens)
    s = lens.shape[0]
    maxb = tables.shape[1] if tables.ndim == 2 else 0
    h = C.c_void_p()
    _check(lib.tts_build_verify_meta(offs.shape[0] - 1, _as_i32p(offs), s, _as_i32p(tables), maxb, _as_i32p(lens),
                                     q_len, block_size, num_blocks, C.byref(desc) if desc is not None else None,
                                     _stream(stream) if desc is not None else None, C.byref(h)))
    return PrefixMeta(h.value, desc)


def tts_prefix_meta_destroy(meta: PrefixMeta):
    load().tts_prefix_meta_destroy(meta.handle)


def tts_prefix_meta_export(meta: PrefixMeta) -> dict:
    v = tts_prefix_meta_view()
    _check(load().tts_prefix_meta_export(meta.handle, C.byref(v)))
    arr = lambda p, n: np.ctypeslib.as_array(p, shape=(n,)).copy() if n else np.zeros(0, np.int32)  # noqa: E731
    s, g = v.num_seqs, v.num_segs
    return {
        "num_seqs": s, "num_segs": g, "perm": arr(v.perm, s), "seg_req": arr(v.seg_req, g),
        "seg_parent": arr(v.seg_parent, g), "seg_lblock_begin": arr(v.seg_lblock_begin, g),
        "seg_nblocks": arr(v.seg_nblocks, g), "seg_beam_begin": arr(v.seg_beam_begin, g),
        "seg_beam_end": arr(v.seg_beam_end, g), "tail_lblock": arr(v.tail_lblock, s),
        "unique_blocks": int(v.unique_blocks), "unique_tokens": int(v.unique_tokens),
    }


def tts_prefix_meta_coverage(meta: PrefixMeta, seq_lens_host=None) -> np.ndarray:
    lib = load()
    lens = None if seq_lens_host is None else _host_i32(seq_lens_host)
    lp = _as_i32p(lens) if lens is not None else None
    n = C.c_int64(0)
    st = lib.tts_prefix_meta_coverage(meta.handle, lp, None, 0, C.byref(n))
    if st not in (TTS_OK, TTS_ERR_WORKSPACE):
        _check(st)
    rows = np.zeros((max(1, n.value), 5), np.int32)
    _check(lib.tts_prefix_meta_coverage(meta.handle, lp, _as_i32p(rows), rows.shape[0], C.byref(n)))
    return rows[: n.value]


def tts_prefix_meta_stats(meta: PrefixMeta):
    u, s = C.c_int64(0), C.c_int64(0)
    _check(load().tts_prefix_meta_stats(meta.handle, C.byref(u), C.byref(s)))
    return u.value, s.value


# Columns of tts_plan_units_host rows, and its flags.
PLAN_COLUMNS = ("unit", "entry", "kv_head", "beam", "block", "valid", "flags")
PLAN_LIVE, PLAN_EXT, PLAN_SECOND, PLAN_WIDE = 1, 2, 4, 8


def tts_plan_units_host(req_seq_offsets, block_tables, seq_lens, block_size: int, num_blocks: int,
                        desc: tts_attn_desc, num_workgroups: int):
    """Host-only work plan listing: (rows [n][7] int32, number of units)."""
    lib = load()
    offs = _host_i32(req_seq_offsets)
    tables = _host_i32(block_tables)
    lens = _host_i32(seq_lens)
    s = lens.shape[0]
    maxb = tables.shape[1] if tables.ndim == 2 else 0
    n, units = C.c_int64(0), C.c_int64(0)
    args = (offs.shape[0] - 1, _as_i32p(offs), s, _as_i32p(tables), maxb, _as_i32p(lens), block_size, num_blocks,
            C.byref(desc), num_workgroups)
    st = lib.tts_plan_units_host(*args, None, 0, C.byref(n), C.byref(units))
    if st not in (TTS_OK, TTS_ERR_WORKSPACE):
        _check(st)
    rows = np.zeros((max(1, n.value), 7), np.int32)
    _check(lib.tts_plan_units_host(*args, _as_i32p(rows), rows.shape[0], C.byref(n), C.byref(units)))
    return rows[: n.value], units.value


def tts_paged_decode_workspace_size(desc: tts_attn_desc, num_seqs: int, max_seq_len: int) -> int:
    return int(load().tts_paged_decode_workspace_size(C.byref(desc), num_seqs, max_seq_len))


def tts_prefix_decode_workspace_size(desc: tts_attn_desc, meta: PrefixMeta) -> int:
    return int(load().tts_prefix_decode_workspace_size(C.byref(desc), meta.handle))


def tts_paged_decode_attn(desc: tts_attn_desc, num_seqs: int, q, k_cache, v_cache, k_scale, v_scale, block_tables,
                          max_blocks_per_seq: int, seq_lens, max_seq_len: int, num_blocks: int, out, workspace,
                          workspace_bytes: int, stream=None):
    _check(load().tts_paged_decode_attn(
        C.byref(desc), num_seqs, _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(k_scale), _ptr(v_scale),
        _ptr(block_tables), max_blocks_per_seq, _ptr(seq_lens), max_seq_len, num_blocks, _ptr(out), _ptr(workspace),
        workspace_bytes, _stream(stream)))


def tts_prefix_decode_attn(desc: tts_attn_desc, meta: PrefixMeta, q, k_cache, v_cache, k_scale, v_scale,
                           block_tables, max_blocks_per_seq: int, seq_lens, num_blocks: int, out, workspace,
                           workspace_bytes: int, stream=None):
    _check(load().tts_prefix_decode_attn(
        C.byref(desc), meta.handle, _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(k_scale), _ptr(v_scale),
        _ptr(block_tables), max_blocks_per_seq, _ptr(seq_lens), num_blocks, _ptr(out), _ptr(workspace),
        workspace_bytes, _stream(stream)))



def tts_prefix_decode_attn_noalloc(desc: tts_attn_desc, meta: PrefixMeta, q, k_cache, v_cache, k_scale, v_scale,
                                   block_tables, max_blocks_per_seq: int, seq_lens, num_blocks: int, out,
                                   stream=None):
    _check(load().tts_prefix_decode_attn_noalloc(
        C.byref(desc), meta.handle, _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(k_scale), _ptr(v_scale),
        _ptr(block_tables), max_blocks_per_seq, _ptr(seq_lens), num_blocks, _ptr(out), _stream(stream)))


def tts_prefix_decode_partials(desc: tts_attn_desc, meta: PrefixMeta, q, k_cache, v_cache, k_scale, v_scale,
                               block_tables, max_blocks_per_seq: int, seq_lens, num_blocks: int, out, workspace,
                               workspace_bytes: int, stream=None):
    _check(load().tts_prefix_decode_partials(
        C.byref(desc), meta.handle, _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(k_scale), _ptr(v_scale),
        _ptr(block_tables), max_blocks_per_seq, _ptr(seq_lens), num_blocks, _ptr(out), _ptr(workspace),
        workspace_bytes, _stream(stream)))


def tts_prefix_decode_merge(desc: tts_attn_desc, meta: PrefixMeta, seq_lens, out, workspace, workspace_bytes: int,
                            stream=None):
    _check(load().tts_prefix_decode_merge(C.byref(desc), meta.handle, _ptr(seq_lens), _ptr(out), _ptr(workspace),
                                          workspace_bytes, _stream(stream)))


def tts_append_kv(desc: tts_attn_desc, num_seqs: int, k_new, v_new, block_tables, max_blocks_per_seq: int, seq_lens,
                  num_blocks: int, k_cache, v_cache, k_scale=None, v_scale=None, stream=None):
    _check(load().tts_append_kv(
        C.byref(desc), num_seqs, _ptr(k_new), _ptr(v_new), _ptr(block_tables), max_blocks_per_seq, _ptr(seq_lens),
        num_blocks, _ptr(k_cache), _ptr(v_cache), _ptr(k_scale), _ptr(v_scale), _stream(stream)))


def tts_copy_blocks(desc: tts_attn_desc, num_pairs: int, pairs, num_blocks: int, k_cache, v_cache, k_scale=None,
                    v_scale=None, stream=None):
    _check(load().tts_copy_blocks(C.byref(desc), num_pairs, _ptr(pairs), num_blocks, _ptr(k_cache), _ptr(v_cache),
                                  _ptr(k_scale), _ptr(v_scale), _stream(stream)))


def tts_fork_tables(parent_tables, parent_lens, block_size: int, child_parent, child_lens, free_ids):
    """Host call; returns (child_tables [C][max_blocks], copies [n][2], number of free ids used)."""
    lib = load()
    pt = _host_i32(parent_tables)
    if pt.ndim != 2:
        pt = pt.reshape(-1, 0) if pt.size == 0 else pt.reshape(1, -1)
    pl, cp, cl, fr = _host_i32(parent_lens), _host_i32(child_parent), _host_i32(child_lens), _host_i32(free_ids)
    nc, mb = cp.shape[0], pt.shape[1]
    ct = np.zeros((max(nc, 1), max(mb, 1)), np.int32)
    cps = np.zeros((max(nc, 1), 2), np.int32)
    ncp, nfu = C.c_int32(0), C.c_int32(0)
    _check(lib.tts_fork_tables(pt.shape[0], _as_i32p(pt), mb, _as_i32p(pl), block_size, nc, _as_i32p(cp),
                               _as_i32p(cl), _as_i32p(fr), fr.shape[0], _as_i32p(ct), _as_i32p(cps),
                               C.byref(ncp), C.byref(nfu)))
    return ct[:nc, :mb], cps[: ncp.value], nfu.value


def tts_kv_alloc_time(problem: tts_alloc_problem, b_pre: int, b_dec: int) -> tts_alloc_result:
    r = tts_alloc_result()
    _check(load().tts_kv_alloc_time(C.byref(problem), b_pre, b_dec, C.byref(r)))
    return r


def tts_kv_alloc_search(problem: tts_alloc_problem) -> tts_alloc_result:
    r = tts_alloc_result()
    _check(load().tts_kv_alloc_search(C.byref(problem), C.byref(r)))
    return r


def tts_prefix_schedule(cots, num_nodes: int, budget: int, node_weight=None):
    """Host call. cots: list of node-id paths. Returns (order, batch list of order slices, score, cost)."""
    lib = load()
    lens = [len(c) for c in cots]
    offs = _host_i32(np.concatenate([[0], np.cumsum(lens)]) if cots else [0])
    nodes = _host_i32(np.concatenate([np.asarray(c, np.int32) for c in cots]) if sum(lens) else np.zeros(0))
    n = len(cots)
    order = np.zeros(max(n, 1), np.int32)
    boff = np.zeros(n + 1, np.int32)
    nb, sc, co = C.c_int32(0), C.c_int64(0), C.c_int64(0)
    wp = None
    if node_weight is not None:
        w = np.ascontiguousarray(np.asarray(node_weight, np.int64))
        wp = w.ctypes.data_as(C.POINTER(C.c_int64))
    _check(lib.tts_prefix_schedule(n, _as_i32p(offs), _as_i32p(nodes) if nodes.size else None, num_nodes, wp,
                                   int(budget), _as_i32p(order), _as_i32p(boff), C.byref(nb), C.byref(sc),
                                   C.byref(co)))
    order = order[:n]
    batches = [order[boff[i]:boff[i + 1]].tolist() for i in range(nb.value)]
    return order, batches, sc.value, co.value


def tts_prefix_verify_attn(desc: tts_attn_desc, meta: PrefixMeta, q, k_cache, v_cache, k_scale, v_scale,
                           block_tables, max_blocks_per_seq: int, seq_lens, num_blocks: int, out, workspace,
                           workspace_bytes: int, stream=None):
    _check(load().tts_prefix_verify_attn(
        C.byref(desc), meta.handle, _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(k_scale), _ptr(v_scale),
        _ptr(block_tables), max_blocks_per_seq, _ptr(seq_lens), num_blocks, _ptr(out), _ptr(workspace),
        workspace_bytes, _stream(stream)))
