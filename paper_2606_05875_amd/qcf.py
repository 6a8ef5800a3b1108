"""Python binding of libqcf (ctypes).  Argument marshalling only.

Each function has the name of the C entry point it calls, takes torch tensors
on the GPU, checks their device, dtype, layout and shape, and passes raw
pointers plus the current HIP stream.  All work runs in the library's
kernels.  If ``libqcf.so`` has not been built the first call raises: there is
no fallback.
"""
from __future__ import annotations

import ctypes
import os
import threading

import torch

__all__ = [
    "QcfError", "lib", "lib_path", "qcf_version", "qcf_status_string", "qcf_recommended_row_stride",
    "qcf_rerope",
    "qcf_assemble", "qcf_gather_rows", "qcf_scatter_kv", "qcf_probe_scores", "qcf_probe_scores_workspace_size",
    "qcf_rope_table", "qcf_probe_scores_pic",
    "qcf_select_topk", "qcf_probe_scores_select", "qcf_probe_scores_select_noalloc",
    "qcf_sparse_prefill_attn", "qcf_sparse_prefill_attn_rope", "rope_position_table", "qcf_sparse_prefill_attn_workspace_size",
    "qcf_mfma_loop",
    "EXPORTS", "Prepared", "prepare",
]

QCF_F32, QCF_BF16 = 0, 1
_DT = {torch.float32: QCF_F32, torch.bfloat16: QCF_BF16}
_LIB = None
_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I = ctypes.c_int
_SZ = ctypes.c_size_t

# name -> (restype, argtypes); mirrors include/qcf.h
EXPORTS = {
    "qcf_version": (_I, []),
    "qcf_status_string": (ctypes.c_char_p, [_I]),
    "qcf_recommended_row_stride": (_I64, [_I, _I]),
    "qcf_rerope": (_I, [_P, _P, _P, _P, _I, _I64, _I64, _I, _I, _I64, _I64, _I, _P, _P, _P, _P, _I,
                        ctypes.c_double, _P]),
    "qcf_assemble": (_I, [_P, _P, _I64, _I64, _P, _P, _I64, _I64, _I, _P, _P, _P, _P, _I, _P, _P, _P,
                          _I64, _I64, _P, _P, _P, _P, _P, _P, _P, _I64, _I64, _P, _P, _I, _I, _I, _I,
                          ctypes.c_double, _P]),
    "qcf_gather_rows": (_I, [_P, _P, _P, _I64, _I64, _I64, _I64, _I64, _P]),
    "qcf_scatter_kv": (_I, [_P, _P, _I64, _I64, _P, _P, _P, _P, _I64, _P, _I, _I64, _P, _P, _I, _I,
                            _I, ctypes.c_double, _P]),
    "qcf_probe_scores_workspace_size": (_SZ, [_I, _I, _I, _I, _I, _I]),
    "qcf_probe_scores": (_I, [_P, _I, _P, _I64, _P, _I64, _I64, _I, _I, _P, _P, _P, _I, _I, _I, _I,
                              _I, ctypes.c_float, _P, _SZ, _P]),
    "qcf_rope_table": (_I, [_P, _P, _I64, _I, ctypes.c_double, _P]),
    "qcf_probe_scores_pic": (_I, [_P, _I, _P, _I64, _P, _I64, _I64, _P, _P, _I64, _I, _I, _P, _P, _P,
                                  _I, _I, _I, _I, _I, ctypes.c_float, _P, _SZ, _P]),
    "qcf_select_topk": (_I, [_P, _P, _I64, _P, _I64, _I, _P, _P, _P, _P, _P, _I, _P]),
    "qcf_probe_scores_select": (_I, [_P, _I, _P, _I64, _P, _I64, _I64, _I, _I, _P, _P, _P, _I, _I, _I,
                                     _I, _I, ctypes.c_float, _P, _P, _I64, _I, _P, _P, _P, _P, _P,
                                     _I, _P, _SZ, _P]),
    "qcf_probe_scores_select_noalloc": (_I, [_P, _I, _P, _I64, _P, _I64, _I64, _I, _I, _P, _P, _P, _I,
                                             _I, _I, _I, _I, ctypes.c_float, _P, _P, _I64, _I, _P, _P,
                                             _P, _P, _P, _I, _P]),
    "qcf_sparse_prefill_attn_workspace_size": (_SZ, [_I, _I, _I, _I, _I, _I, _I]),
    "qcf_sparse_prefill_attn_rope": (_I, [_P, _P, _P, _P, _I64, _P, _I64, _P, _P, _P, _I64, _I64, _P,
                                          _P, _I64, _I, _I, _I, _I, _I, _I, _I, ctypes.c_float, _P,
                                          _SZ, _P]),
    "qcf_sparse_prefill_attn": (_I, [_P, _P, _P, _P, _I64, _P, _P, _P, _I64, _I64, _P, _P, _I, _I,
                                     _I, _I, _I, _I, _I, ctypes.c_float, _P, _SZ, _P]),
    "qcf_mfma_loop": (_I, [_P, _I64, _P, _I64, _P, _I, _I, _P]),
}


class QcfError(RuntimeError):
    pass


def lib_path() -> str:
    return os.path.join(os.path.dirname(os.path.abspath(__file__)), "libqcf.so")


def lib():
    """Load libqcf.so once; raise if it is missing (no fallback path exists)."""
    global _LIB
    if _LIB is None:
        path = lib_path()
        if not os.path.exists(path):
            raise QcfError(f"{path} is missing: build it with `python -m paper_2606_05875_amd.build`")
        h = ctypes.CDLL(path)
        for name, (res, args) in EXPORTS.items():
            fn = getattr(h, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = h
    return _LIB


def _check(status: int, name: str):
    if status != 0:
        msg = lib().qcf_status_string(status).decode()
        raise QcfError(f"{name} failed with status {status}: {msg}")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


class Prepared:
    """One validated, marshalled libqcf call.  Calling it enqueues the same launch
    again -- on `stream` (a raw HIP stream handle) or torch's current stream --
    without repeating the argument checks and conversions; it keeps the tensors
    of the call alive.  Buffers must not be reallocated while it is in use."""

    __slots__ = ("name", "fn", "args", "keep")

    def __init__(self, name, fn, args, keep):
        self.name, self.fn, self.args, self.keep = name, fn, args, keep

    def __call__(self, stream=None):
        st = self.fn(*self.args, _stream() if stream is None else stream)
        if st:
            _check(st, self.name)


class _Recorder(threading.local):
    on = False
    out = None
    keep = None


_REC = _Recorder()


def _invoke(name, *args, keep=None):
    fn = getattr(lib(), name)
    if _REC.on:
        _REC.out = Prepared(name, fn, args, (_REC.keep, keep))
        return
    _check(fn(*args, _stream()), name)


def prepare(call, *args, **kwargs) -> Prepared:
    """Validate and marshal ``call(*args, **kwargs)`` (a binding of this module) once and
    return it as a Prepared call; a call with nothing to launch gives a no-op."""
    _REC.on, _REC.out, _REC.keep = True, None, (args, kwargs)
    try:
        call(*args, **kwargs)
    finally:
        _REC.on, _REC.keep = False, None
    out, _REC.out = _REC.out, None
    return out if out is not None else Prepared(getattr(call, "__name__", "noop"), lambda *a: 0, (), None)


def _dev(t, name, dtype=None):
    if t is None:
        return
    if not t.is_cuda:
        raise QcfError(f"{name} must be a GPU tensor")
    if dtype is not None and t.dtype != dtype:
        raise QcfError(f"{name} must be {dtype}, got {t.dtype}")


def _rows(t, name):
    """Token-major tensor [rows, heads, d] (or [rows, cols]) with a dense row; returns row stride."""
    if t.dim() < 2 or (t.shape[0] > 0 and not t[0].is_contiguous()):
        raise QcfError(f"{name} must have dense rows")
    return t.stride(0)


def _dtype(t):
    if t.dtype not in _DT:
        raise QcfError(f"unsupported dtype {t.dtype}")
    return _DT[t.dtype]


def _i32(t, name):
    _dev(t, name, torch.int32)
    if t is not None and not t.is_contiguous():
        raise QcfError(f"{name} must be contiguous")


def qcf_version() -> int:
    return lib().qcf_version()


def qcf_status_string(status: int) -> str:
    return lib().qcf_status_string(status).decode()


def qcf_recommended_row_stride(n_kv_heads, head_dim):
    """Row stride (elements) for a K/V cache read by the attention and score kernels; host call."""
    r = int(lib().qcf_recommended_row_stride(int(n_kv_heads), int(head_dim)))
    if r <= 0:
        raise QcfError(f"no row stride for n_kv_heads={n_kv_heads}, head_dim={head_dim}")
    return r


def qcf_rerope(k_out, k_in, seg_start, seg_len, seg_delta, max_seg_len, rope_theta, v_out=None,
               v_in=None, src_start=None):
    """Remap each segment's keys by its offset (and stitch its values); shapes [T, H_kv, d]."""
    _dev(k_out, "k_out", k_in.dtype)
    _dev(k_in, "k_in")
    _dev(v_out, "v_out", k_in.dtype)
    _dev(v_in, "v_in", k_in.dtype)
    for n, t in (("seg_start", seg_start), ("seg_len", seg_len), ("seg_delta", seg_delta),
                 ("src_start", src_start)):
        _i32(t, n)
    if k_out.shape[1:] != k_in.shape[1:]:
        raise QcfError("k_out and k_in must have the same row shape")
    if (v_out is None) != (v_in is None):
        raise QcfError("v_out and v_in go together")
    if v_out is not None and (v_out.shape != k_out.shape or v_in.shape != k_in.shape
                              or v_out.stride(0) != k_out.stride(0) or v_in.stride(0) != k_in.stride(0)):
        raise QcfError("v_out/v_in must match k_out/k_in in shape and row stride")
    T_in, H, d = k_in.shape
    _invoke("qcf_rerope", _ptr(k_out), _ptr(k_in), _ptr(v_out), _ptr(v_in), _dtype(k_in),
                          k_out.shape[0], T_in, H, d, _rows(k_out, "k_out"), _rows(k_in, "k_in"),
                          seg_start.numel(),
                          _ptr(seg_start), _ptr(seg_len), _ptr(seg_delta), _ptr(src_start),
                          int(max_seg_len), float(rope_theta))


def qcf_assemble(k_cache, v_cache, k_pic, v_pic, seg_start, seg_len, seg_delta, max_seg_len,
                 q_new, k_new, v_new, query_row, query_pos, q_u, probe_k, probe_v, probe_src,
                 probe_delta, rope_theta, src_start=None, query_src=None, query_slot=None):
    """One launch: chunk remap + stitch into the cache, query rows rotated into the cache and
    q_u (and probe slots), anchor rows remapped from the stored chunks into the probe buffer."""
    dt = k_pic.dtype
    for n, t in (("k_cache", k_cache), ("v_cache", v_cache), ("k_pic", k_pic), ("v_pic", v_pic),
                 ("q_new", q_new), ("k_new", k_new), ("v_new", v_new), ("q_u", q_u),
                 ("probe_k", probe_k), ("probe_v", probe_v)):
        _dev(t, n, dt)
    for n, t in (("seg_start", seg_start), ("seg_len", seg_len), ("seg_delta", seg_delta),
                 ("src_start", src_start), ("query_row", query_row), ("query_pos", query_pos),
                 ("query_src", query_src), ("query_slot", query_slot), ("probe_src", probe_src),
                 ("probe_delta", probe_delta)):
        _i32(t, n)
    T, hkv, d = k_cache.shape
    rs = _rows(k_cache, "k_cache")
    prs = _rows(k_pic, "k_pic")
    qrs = _rows(probe_k, "probe_k")
    if (v_cache.shape != k_cache.shape or v_cache.stride(0) != rs or k_pic.shape[1:] != (hkv, d)
            or v_pic.shape != k_pic.shape or v_pic.stride(0) != prs or probe_v.stride(0) != qrs):
        raise QcfError("k_cache/v_cache, k_pic/v_pic and probe_k/probe_v pairs must match in row "
                       "shape and row stride")
    for n, t in (("q_new", q_new), ("k_new", k_new), ("v_new", v_new), ("q_u", q_u)):
        if not t.is_contiguous():
            raise QcfError(f"{n} must be dense")
    hq = q_new.shape[1]
    nq = query_row.numel()
    if (k_new.shape[1:] != (hkv, d) or v_new.shape != k_new.shape or q_new.shape[0] != k_new.shape[0]
            or q_new.shape[2] != d or q_u.shape != (nq, hq, d) or query_pos.numel() != nq
            or (query_src is not None and query_src.numel() != nq)
            or (query_slot is not None and query_slot.numel() != nq)):
        raise QcfError("query tensors: q_new [S, H_q, d], k_new/v_new [S, H_kv, d], q_u [n_query, H_q, d]")
    npb = probe_src.numel()
    if (probe_k.shape != (npb, hkv, d) or probe_v.shape != probe_k.shape
            or probe_delta.numel() != npb):
        raise QcfError("probe_k/probe_v must be [len(probe_src), H_kv, d]")
    _invoke("qcf_assemble", _ptr(k_cache), _ptr(v_cache), T, rs, _ptr(k_pic), _ptr(v_pic),
                            k_pic.shape[0], prs, seg_start.numel(), _ptr(seg_start), _ptr(seg_len),
                            _ptr(seg_delta), _ptr(src_start), int(max_seg_len), _ptr(q_new),
                            _ptr(k_new), _ptr(v_new), k_new.shape[0], nq, _ptr(query_row),
                            _ptr(query_pos), _ptr(query_src), _ptr(query_slot), _ptr(q_u),
                            _ptr(probe_k), _ptr(probe_v), npb, qrs, _ptr(probe_src), _ptr(probe_delta),
                            _dtype(k_pic), hq, hkv, d, float(rope_theta))


def qcf_gather_rows(dst, src, idx):
    """dst[i] = src[idx[i]] for every row (rows of equal byte size)."""
    _dev(dst, "dst", src.dtype)
    _dev(src, "src")
    _i32(idx, "idx")
    if dst.shape[0] != idx.numel() or dst.shape[1:] != src.shape[1:]:
        raise QcfError("dst must be [len(idx), *src.shape[1:]]")
    row_bytes = src[0].numel() * src.element_size() if src.shape[0] else dst[0].numel() * dst.element_size()
    _invoke("qcf_gather_rows", _ptr(dst), _ptr(src), _ptr(idx), idx.numel(), src.shape[0], row_bytes,
                               _rows(src, "src") * src.element_size(),
                               _rows(dst, "dst") * dst.element_size())


def qcf_scatter_kv(k_cache, v_cache, k_new, v_new, row_idx, row_pos, rope_theta, q_new=None,
                   q_out=None, src_idx=None):
    """Fused-cache update: rope(k_new[s]) and v_new[s] into cache rows row_idx; rope(q_new[s]) -> q_out."""
    for n, t in (("k_cache", k_cache), ("v_cache", v_cache), ("k_new", k_new), ("v_new", v_new),
                 ("q_new", q_new), ("q_out", q_out)):
        _dev(t, n, k_cache.dtype)
    for n, t in (("row_idx", row_idx), ("row_pos", row_pos), ("src_idx", src_idx)):
        _i32(t, n)
    T, Hkv, d = k_cache.shape
    if v_cache.shape != k_cache.shape or v_cache.stride(0) != k_cache.stride(0):
        raise QcfError("k_cache and v_cache must match")
    if not (k_new.is_contiguous() and v_new.is_contiguous() and k_new.shape[1:] == (Hkv, d)
            and v_new.shape == k_new.shape):
        raise QcfError("k_new/v_new must be dense [rows, H_kv, d]")
    n = row_idx.numel()
    if row_pos.numel() != n or (src_idx is not None and src_idx.numel() != n):
        raise QcfError("row_idx, row_pos and src_idx must have the same length")
    hq = Hkv
    if q_out is not None:
        if q_new is None or not (q_new.is_contiguous() and q_out.is_contiguous()):
            raise QcfError("q_new/q_out must be dense")
        hq = q_new.shape[1]
        if q_out.shape != (n, hq, d) or q_new.shape[1:] != (hq, d) or q_new.shape[0] != k_new.shape[0]:
            raise QcfError("q_out must be [n_rows, H_q, d] and q_new [n_src_rows, H_q, d]")
    _invoke("qcf_scatter_kv", _ptr(k_cache), _ptr(v_cache), T, _rows(k_cache, "k_cache"), _ptr(k_new),
                              _ptr(v_new), _ptr(q_new), _ptr(q_out), k_new.shape[0], _ptr(src_idx),
                              _dtype(k_cache), n, _ptr(row_idx), _ptr(row_pos), hq, Hkv, d,
                              float(rope_theta))


def qcf_probe_scores_workspace_size(batch, max_q_len, max_ctx_len, n_q_heads, n_kv_heads, head_dim):
    return int(lib().qcf_probe_scores_workspace_size(batch, max_q_len, max_ctx_len, n_q_heads,
                                                     n_kv_heads, head_dim))


def qcf_probe_scores(scores, q, k, cu_q, cu_kv, ctx_len, max_q_len, max_ctx_len, softmax_scale,
                     accumulate=False, workspace=None):
    """Critical-layer importance of every context token; q [n_q, H_q, d], k [T, H_kv, d]."""
    _dev(scores, "scores", torch.float32)
    _dev(q, "q")
    _dev(k, "k", q.dtype)
    for n, t in (("cu_q", cu_q), ("cu_kv", cu_kv), ("ctx_len", ctx_len)):
        _i32(t, n)
    if not q.is_contiguous():
        raise QcfError("q must be dense")
    nq, hq, d = q.shape
    T, hkv, d2 = k.shape
    if d2 != d or scores.numel() != T:
        raise QcfError("scores must have one entry per row of k; head_dim must match")
    batch = ctx_len.numel()
    need = qcf_probe_scores_workspace_size(batch, max_q_len, max_ctx_len, hq, hkv, d)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    _invoke("qcf_probe_scores", _ptr(scores), int(bool(accumulate)), _ptr(q), nq, _ptr(k), T,
                                _rows(k, "k"), _dtype(q), batch, _ptr(cu_q), _ptr(cu_kv), _ptr(ctx_len),
                                int(max_q_len), int(max_ctx_len), hq, hkv, d, float(softmax_scale),
                                _ptr(workspace), workspace.numel(), keep=workspace)


def qcf_rope_table(table, pos, rope_theta):
    """table [n, d/2, 2] float32 <- (cos, sin) of the rotations by pos[i] (int32 [n])."""
    _dev(table, "table", torch.float32)
    _i32(pos, "pos")
    if table.dim() != 3 or table.shape[2] != 2 or table.shape[0] != pos.numel() or not table.is_contiguous():
        raise QcfError("table must be a dense [n, head_dim/2, 2] float32 tensor with n = len(pos)")
    _invoke("qcf_rope_table", _ptr(table), _ptr(pos), pos.numel(), 2 * table.shape[1],
                              float(rope_theta))


def qcf_probe_scores_pic(scores, q, k_pic, key_rot, rope_table, cu_q, cu_kv, ctx_len, max_q_len,
                         max_ctx_len, softmax_scale, accumulate=False, workspace=None):
    """qcf_probe_scores over k_pic's keys turned by rope_table[key_rot[t]] on the fly."""
    _dev(scores, "scores", torch.float32)
    _dev(q, "q")
    _dev(k_pic, "k_pic", q.dtype)
    _dev(rope_table, "rope_table", torch.float32)
    for n, t in (("key_rot", key_rot), ("cu_q", cu_q), ("cu_kv", cu_kv), ("ctx_len", ctx_len)):
        _i32(t, n)
    if not q.is_contiguous() or not rope_table.is_contiguous():
        raise QcfError("q and rope_table must be dense")
    nq, hq, d = q.shape
    T, hkv, d2 = k_pic.shape
    if d2 != d or scores.numel() != T or key_rot.numel() != T:
        raise QcfError("scores and key_rot need one entry per row of k_pic; head_dim must match")
    if rope_table.dim() != 3 or tuple(rope_table.shape[1:]) != (d // 2, 2):
        raise QcfError("rope_table must be [n_rot, head_dim/2, 2]")
    batch = ctx_len.numel()
    need = qcf_probe_scores_workspace_size(batch, max_q_len, max_ctx_len, hq, hkv, d)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    _invoke("qcf_probe_scores_pic", _ptr(scores), int(bool(accumulate)), _ptr(q), nq, _ptr(k_pic), T,
                                    _rows(k_pic, "k_pic"), _ptr(key_rot), _ptr(rope_table),
                                    rope_table.shape[0], _dtype(q), batch, _ptr(cu_q), _ptr(cu_kv),
                                    _ptr(ctx_len), int(max_q_len), int(max_ctx_len), hq, hkv, d,
                                    float(softmax_scale), _ptr(workspace), workspace.numel(),
                                    keep=workspace)


def qcf_select_topk(out_idx, scores, seg_start, seg_len, seg_k, out_start, max_seg_len, out_pos=None,
                    pos_base=None):
    """Per-segment top-k rows (ascending, ties to the lower row) into out_idx[out_start[s] ..]."""
    _dev(scores, "scores", torch.float32)
    for n, t in (("out_idx", out_idx), ("seg_start", seg_start), ("seg_len", seg_len),
                 ("seg_k", seg_k), ("out_start", out_start), ("out_pos", out_pos),
                 ("pos_base", pos_base)):
        _i32(t, n)
    if out_pos is not None and out_pos.numel() != out_idx.numel():
        raise QcfError("out_pos must match out_idx")
    _invoke("qcf_select_topk", _ptr(out_idx), _ptr(out_pos), out_idx.numel(), _ptr(scores),
                               scores.numel(), seg_start.numel(), _ptr(seg_start), _ptr(seg_len),
                               _ptr(seg_k), _ptr(out_start), _ptr(pos_base), int(max_seg_len))


def qcf_probe_scores_select(scores, q, k, cu_q, cu_kv, ctx_len, max_q_len, max_ctx_len,
                            softmax_scale, out_idx, seg_start, seg_len, seg_k, out_start, seg_req,
                            max_seg_len, out_pos=None, accumulate=False, workspace=None):
    """qcf_probe_scores then qcf_select_topk on the finished scores, in one call."""
    _dev(scores, "scores", torch.float32)
    _dev(q, "q")
    _dev(k, "k", q.dtype)
    for n, t in (("cu_q", cu_q), ("cu_kv", cu_kv), ("ctx_len", ctx_len), ("out_idx", out_idx),
                 ("seg_start", seg_start), ("seg_len", seg_len), ("seg_k", seg_k),
                 ("out_start", out_start), ("seg_req", seg_req), ("out_pos", out_pos)):
        _i32(t, n)
    if not q.is_contiguous():
        raise QcfError("q must be dense")
    nq, hq, d = q.shape
    T, hkv, d2 = k.shape
    if d2 != d or scores.numel() != T:
        raise QcfError("scores must have one entry per row of k; head_dim must match")
    if out_pos is not None and out_pos.numel() != out_idx.numel():
        raise QcfError("out_pos must match out_idx")
    if seg_req.numel() != seg_start.numel():
        raise QcfError("seg_req needs one request per segment")
    batch = ctx_len.numel()
    need = qcf_probe_scores_workspace_size(batch, max_q_len, max_ctx_len, hq, hkv, d)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    _invoke("qcf_probe_scores_select", _ptr(scores), int(bool(accumulate)), _ptr(q), nq, _ptr(k), T,
            _rows(k, "k"), _dtype(q), batch, _ptr(cu_q), _ptr(cu_kv), _ptr(ctx_len), int(max_q_len),
            int(max_ctx_len), hq, hkv, d, float(softmax_scale), _ptr(out_idx), _ptr(out_pos),
            out_idx.numel(), seg_start.numel(), _ptr(seg_start), _ptr(seg_len), _ptr(seg_k),
            _ptr(out_start), _ptr(seg_req), int(max_seg_len), _ptr(workspace), workspace.numel(),
            keep=workspace)


def qcf_probe_scores_select_noalloc(scores, q, k, cu_q, cu_kv, ctx_len, max_q_len, max_ctx_len,
                                    softmax_scale, out_idx, seg_start, seg_len, seg_k, out_start,
                                    seg_req, max_seg_len, out_pos=None, accumulate=False):
    """qcf_probe_scores_select with the library's fixed device scratch array instead of a
    workspace (nothing is allocated; calls that overlap on one GPU race)."""
    _dev(scores, "scores", torch.float32)
    _dev(q, "q")
    _dev(k, "k", q.dtype)
    for n, t in (("cu_q", cu_q), ("cu_kv", cu_kv), ("ctx_len", ctx_len), ("out_idx", out_idx),
                 ("seg_start", seg_start), ("seg_len", seg_len), ("seg_k", seg_k),
                 ("out_start", out_start), ("seg_req", seg_req), ("out_pos", out_pos)):
        _i32(t, n)
    if not q.is_contiguous():
        raise QcfError("q must be dense")
    nq, hq, d = q.shape
    T, hkv, d2 = k.shape
    if d2 != d or scores.numel() != T:
        raise QcfError("scores must have one entry per row of k; head_dim must match")
    if out_pos is not None and out_pos.numel() != out_idx.numel():
        raise QcfError("out_pos must match out_idx")
    if seg_req.numel() != seg_start.numel():
        raise QcfError("seg_req needs one request per segment")
    _invoke("qcf_probe_scores_select_noalloc", _ptr(scores), int(bool(accumulate)), _ptr(q), nq,
            _ptr(k), T, _rows(k, "k"), _dtype(q), ctx_len.numel(), _ptr(cu_q), _ptr(cu_kv),
            _ptr(ctx_len), int(max_q_len), int(max_ctx_len), hq, hkv, d, float(softmax_scale),
            _ptr(out_idx), _ptr(out_pos), out_idx.numel(), seg_start.numel(), _ptr(seg_start),
            _ptr(seg_len), _ptr(seg_k), _ptr(out_start), _ptr(seg_req), int(max_seg_len))


def qcf_sparse_prefill_attn_workspace_size(batch, max_rows, max_kv, n_q_heads, n_kv_heads, head_dim,
                                           dtype=torch.bfloat16):
    return int(lib().qcf_sparse_prefill_attn_workspace_size(batch, max_rows, max_kv, n_q_heads,
                                                            n_kv_heads, head_dim, _DT[dtype]))


def qcf_sparse_prefill_attn(out, q, row_pos, cu_rows, k_cache, v_cache, cu_kv, max_rows, max_kv,
                            softmax_scale, kv_pos=None, lse=None, workspace=None):
    """Causal GQA attention of rows q over the cache (explicit key positions with kv_pos)."""
    _dev(out, "out", q.dtype)
    _dev(q, "q")
    _dev(k_cache, "k_cache", q.dtype)
    _dev(v_cache, "v_cache", q.dtype)
    _dev(lse, "lse", torch.float32)
    for n, t in (("row_pos", row_pos), ("cu_rows", cu_rows), ("cu_kv", cu_kv), ("kv_pos", kv_pos)):
        _i32(t, n)
    if not (q.is_contiguous() and out.is_contiguous()) or out.shape != q.shape:
        raise QcfError("q and out must be dense and of the same shape")
    n, hq, d = q.shape
    T, hkv, d2 = k_cache.shape
    if v_cache.shape != k_cache.shape or v_cache.stride(0) != k_cache.stride(0) or d2 != d:
        raise QcfError("k_cache/v_cache mismatch")
    if row_pos.numel() != n or (kv_pos is not None and kv_pos.numel() != T):
        raise QcfError("row_pos must have one entry per row, kv_pos one per cache row")
    if lse is not None and lse.shape != (n, hq):
        raise QcfError("lse must be [n_rows, H_q]")
    batch = cu_rows.numel() - 1
    need = qcf_sparse_prefill_attn_workspace_size(batch, max_rows, max_kv, hq, hkv, d, q.dtype)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    _invoke("qcf_sparse_prefill_attn", _ptr(out), _ptr(lse), _ptr(q), _ptr(row_pos), n, _ptr(cu_rows),
                                       _ptr(k_cache), _ptr(v_cache), T, _rows(k_cache, "k_cache"),
                                       _ptr(cu_kv), _ptr(kv_pos), _dtype(q), batch, int(max_rows),
                                       int(max_kv), hq, hkv, d, float(softmax_scale), _ptr(workspace),
                                       0 if workspace is None else workspace.numel(), keep=workspace)


def rope_position_table(n_pos, head_dim, rope_theta, device="cuda"):
    """The (cos, sin) table of positions 0..n_pos-1 that qcf_sparse_prefill_attn_rope reads
    (qcf_rope_table at those positions; a constant of theta and head_dim)."""
    pos = torch.arange(n_pos, dtype=torch.int32, device=device)
    table = torch.empty((n_pos, head_dim // 2, 2), dtype=torch.float32, device=device)
    qcf_rope_table(table, pos, rope_theta)
    return table


def qcf_sparse_prefill_attn_rope(out, q_raw, row_pos, cu_rows, k_cache, v_cache, cu_kv, max_rows,
                                 max_kv, softmax_scale, rope_table, q_src=None, lse=None,
                                 workspace=None):
    """qcf_sparse_prefill_attn on un-rotated query rows (read through q_src when given), turned
    in the kernel by rope_table[row_pos[r]]."""
    _dev(out, "out", torch.bfloat16)
    _dev(q_raw, "q_raw", torch.bfloat16)
    _dev(k_cache, "k_cache", torch.bfloat16)
    _dev(v_cache, "v_cache", torch.bfloat16)
    _dev(rope_table, "rope_table", torch.float32)
    _dev(lse, "lse", torch.float32)
    for n, t in (("row_pos", row_pos), ("cu_rows", cu_rows), ("cu_kv", cu_kv), ("q_src", q_src)):
        _i32(t, n)
    if not (q_raw.is_contiguous() and out.is_contiguous() and rope_table.is_contiguous()):
        raise QcfError("q_raw, out and rope_table must be dense")
    n, hq, d = out.shape
    nq_raw = q_raw.shape[0]
    T, hkv, d2 = k_cache.shape
    if q_raw.shape[1:] != (hq, d) or rope_table.shape[1:] != (d // 2, 2):
        raise QcfError("q_raw must be [rows, H_q, d] and rope_table [positions, d/2, 2]")
    if v_cache.shape != k_cache.shape or v_cache.stride(0) != k_cache.stride(0) or d2 != d:
        raise QcfError("k_cache/v_cache mismatch")
    if row_pos.numel() != n or (q_src is not None and q_src.numel() != n):
        raise QcfError("row_pos (and q_src) must have one entry per recomputed row")
    if q_src is None and nq_raw < n:
        raise QcfError("without q_src, q_raw needs a row per recomputed row")
    if lse is not None and lse.shape != (n, hq):
        raise QcfError("lse must be [n_rows, H_q]")
    batch = cu_rows.numel() - 1
    need = qcf_sparse_prefill_attn_workspace_size(batch, max_rows, max_kv, hq, hkv, d, torch.bfloat16)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=out.device)
    _invoke("qcf_sparse_prefill_attn_rope", _ptr(out), _ptr(lse), _ptr(q_raw), _ptr(q_src), nq_raw,
            _ptr(row_pos), n, _ptr(cu_rows), _ptr(k_cache), _ptr(v_cache), T, _rows(k_cache, "k_cache"),
            _ptr(cu_kv), _ptr(rope_table), rope_table.shape[0], _dtype(out), batch, int(max_rows),
            int(max_kv), hq, hkv, d, float(softmax_scale), _ptr(workspace),
            0 if workspace is None else workspace.numel(), keep=workspace)


def qcf_mfma_loop(operands, sink, clocks, blocks, iters):
    """The attention's product instruction in a plain loop (a yardstick, not a step of the
    method): `blocks` four-wave blocks, iters x 16 products per wave; `clocks` (uint64 [32]
    as int64) gets the start/end counters of blocks 0-7."""
    _dev(operands, "operands", torch.bfloat16)
    _dev(sink, "sink", torch.float32)
    _dev(clocks, "clocks", torch.int64)
    if clocks.numel() < 32 or sink.numel() < blocks * 256 or not operands.is_contiguous():
        raise QcfError("clocks needs 32 entries, sink blocks * 256, operands a dense buffer")
    _invoke("qcf_mfma_loop", _ptr(operands), operands.numel(), _ptr(sink), sink.numel(), _ptr(clocks),
            int(blocks), int(iters))
