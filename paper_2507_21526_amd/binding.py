"""ctypes binding of libtriattn.so (include/triattn.h).

Argument marshalling only: every step of the attention passes runs in the HIP
kernels of the library.  Torch tensors provide device memory and the stream.
The library must have been built (``python -m paper_2507_21526_amd.build``);
loading raises ``RuntimeError`` otherwise -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libtriattn.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "triattn.h")

TA_OK = 0
TA_ERR_INVALID_ARG = 1
TA_ERR_UNSUPPORTED = 2
TA_ERR_BUFFER_TOO_SMALL = 3
TA_ERR_WORKSPACE = 4
TA_ERR_SCHEDULE_MISMATCH = 5
TA_ERR_HIP = 6

TRIANGLE = 0
CAUSAL = 1
BLOCKSPARSE = 2
OUT_BF16 = 0
OUT_F32 = 1

HDR_WORDS, ITEM_WORDS, MERGE_WORDS = 16, 12, 8


class ScheduleInfo(ctypes.Structure):
    _fields_ = [
        ("version", ctypes.c_int32),
        ("kind", ctypes.c_int32),
        ("tile", ctypes.c_int32),
        ("batch", ctypes.c_int32),
        ("sink", ctypes.c_int32),
        ("window", ctypes.c_int32),
        ("last", ctypes.c_int32),
        ("splits_requested", ctypes.c_int32),
        ("total_tokens", ctypes.c_int64),
        ("words", ctypes.c_int64),
        ("n_items", ctypes.c_int32),
        ("n_last_items", ctypes.c_int32),
        ("n_merge_items", ctypes.c_int32),
        ("n_last_rows", ctypes.c_int32),
        ("n_partial_rows", ctypes.c_int32),
        ("max_splits", ctypes.c_int32),
        ("kept_tiles_per_qhead", ctypes.c_int64),
        ("max_item_tiles", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
    ]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class TriAttnError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"status {status}: {message}")
        self.status = status


_lib = None


def lib():
    """Load libtriattn.so; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build it with "
            "`python -m paper_2507_21526_amd.build` (no fallback path exists)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    pinfo = ctypes.POINTER(ScheduleInfo)
    L.ta_abi_version.restype = i32
    L.ta_abi_version.argtypes = []
    L.ta_last_error.restype = ctypes.c_char_p
    L.ta_last_error.argtypes = []
    L.ta_build_schedule.restype = ctypes.c_int
    L.ta_build_schedule.argtypes = [i32, vp, i32, i32, i32, i32, i32, i32, vp,
                                    i64, pinfo]
    L.ta_workspace_bytes.restype = ctypes.c_size_t
    L.ta_workspace_bytes.argtypes = [pinfo, i32, i32]
    L.triangle_attn_fwd.restype = ctypes.c_int
    L.triangle_attn_fwd.argtypes = [vp, vp, vp, vp, i32, vp, vp, pinfo, i64,
                                    i32, i32, i32, ctypes.c_float, vp,
                                    ctypes.c_size_t, vp]
    L.triangle_attn_fwd_noalloc.restype = ctypes.c_int
    L.triangle_attn_fwd_noalloc.argtypes = [vp, vp, vp, vp, i32, vp, vp, pinfo, i64,
                                            i32, i32, i32, ctypes.c_float, vp]
    L.triangle_attn_tiles.restype = ctypes.c_int
    L.triangle_attn_tiles.argtypes = list(L.triangle_attn_fwd.argtypes)
    L.triangle_attn_merge.restype = ctypes.c_int
    L.triangle_attn_merge.argtypes = [vp, i32, vp, vp, pinfo, i64, i32, i32,
                                      vp, ctypes.c_size_t, vp]
    L.causal_attn_fwd.restype = ctypes.c_int
    L.causal_attn_fwd.argtypes = [vp, vp, vp, vp, i32, vp, vp, pinfo, i64,
                                  i32, i32, i32, ctypes.c_float, vp]
    L.ta_build_blocksparse_schedule.restype = ctypes.c_int
    L.ta_build_blocksparse_schedule.argtypes = [vp, i32, i32, vp, vp, i32, vp, i64,
                                                pinfo]
    L.blocksparse_attn_fwd.restype = ctypes.c_int
    L.blocksparse_attn_fwd.argtypes = list(L.triangle_attn_fwd.argtypes)
    L.ta_probe_workspace_bytes.restype = ctypes.c_size_t
    L.ta_probe_workspace_bytes.argtypes = [pinfo, i32]
    L.region_grad_probe.restype = ctypes.c_int
    L.region_grad_probe.argtypes = [vp, vp, vp, vp, vp, vp, pinfo, i64, i32, i32,
                                    i32, ctypes.c_float, i32, i32, i32, vp, vp,
                                    ctypes.c_size_t, vp]
    L.ta_region_counts.restype = ctypes.c_int
    L.ta_region_counts.argtypes = [vp, i32, i32, i32, i32, vp]
    L.ta_region_grad_mean.restype = ctypes.c_int
    L.ta_region_grad_mean.argtypes = [vp, i32, vp, vp]
    L.ta_select_triangle_layers.restype = ctypes.c_int
    L.ta_select_triangle_layers.argtypes = [vp, i32, i32, vp]
    _lib = L
    return L


def ta_last_error() -> str:
    return lib().ta_last_error().decode()


def ta_abi_version() -> int:
    return int(lib().ta_abi_version())


def _check(status):
    if status != TA_OK:
        raise TriAttnError(status, ta_last_error())


def _kind(kind) -> int:
    if kind in (TRIANGLE, "triangle"):
        return TRIANGLE
    if kind in (CAUSAL, "causal"):
        return CAUSAL
    if kind in (BLOCKSPARSE, "blocksparse"):
        return BLOCKSPARSE
    raise ValueError(f"unknown kind {kind!r}")


def ta_build_schedule(kind, cu_seqlens, sink, window, last, tile, splits=0):
    """Build a schedule on the host: returns (int32 words, ScheduleInfo)."""
    L = lib()
    cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
    info = ScheduleInfo()
    _check(L.ta_build_schedule(_kind(kind), cu.ctypes.data, cu.size - 1, sink,
                               window, last, tile, splits, None, 0,
                               ctypes.byref(info)))
    words = np.zeros(info.words, dtype=np.int32)
    _check(L.ta_build_schedule(_kind(kind), cu.ctypes.data, cu.size - 1, sink,
                               window, last, tile, splits, words.ctypes.data,
                               words.size, ctypes.byref(info)))
    return words, info


def ta_build_blocksparse_schedule(cu_seqlens, tile, qtile_ptr, ktile_idx,
                                  max_tiles_per_item=0):
    """Build a block-sparse schedule on the host from per-q-tile k-tile
    lists in CSR form: returns (int32 words, ScheduleInfo)."""
    L = lib()
    cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
    ptr = np.ascontiguousarray(np.asarray(qtile_ptr, dtype=np.int32))
    idx = np.ascontiguousarray(np.asarray(ktile_idx, dtype=np.int32))
    idx_p = idx.ctypes.data if idx.size else None
    info = ScheduleInfo()
    _check(L.ta_build_blocksparse_schedule(cu.ctypes.data, cu.size - 1, tile,
                                           ptr.ctypes.data, idx_p, max_tiles_per_item,
                                           None, 0, ctypes.byref(info)))
    words = np.zeros(info.words, dtype=np.int32)
    _check(L.ta_build_blocksparse_schedule(cu.ctypes.data, cu.size - 1, tile,
                                           ptr.ctypes.data, idx_p, max_tiles_per_item,
                                           words.ctypes.data, words.size,
                                           ctypes.byref(info)))
    return words, info


def ta_workspace_bytes(info: ScheduleInfo, hq: int, head_dim: int) -> int:
    return int(lib().ta_workspace_bytes(ctypes.byref(info), hq, head_dim))


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _out_dtype(o):
    import torch
    if o.dtype == torch.bfloat16:
        return OUT_BF16
    if o.dtype == torch.float32:
        return OUT_F32
    raise ValueError(f"o must be bf16 or fp32, got {o.dtype}")


def _check_tensors(q, k, v, o, lse, sched_dev, info, workspace=None, extra=()):
    """Validate what the C interface cannot see: dtypes, contiguity, shapes
    and devices of the torch tensors whose raw pointers are passed.  Raises
    ValueError before anything is enqueued (a wrong shape or a strided view
    would otherwise be misread, or read out of bounds, by the kernels).
    extra: (name, tensor, dtype, shape) of further operands."""
    import torch
    named = [("q", q), ("k", k), ("v", v), ("o", o)]
    for name, t in named:
        if not isinstance(t, torch.Tensor):
            raise ValueError(f"{name} must be a torch tensor")
    for name, t in (("q", q), ("k", k), ("v", v)):
        if t.dtype != torch.bfloat16:
            raise ValueError(f"{name} must be bfloat16, got {t.dtype}")
        if t.dim() != 3:
            raise ValueError(f"{name} must be [tokens, heads, head_dim], got {tuple(t.shape)}")
    _out_dtype(o)
    total, hq, d = q.shape
    if k.shape[0] != total or v.shape[0] != total:
        raise ValueError(f"k and v must have {total} tokens like q, got "
                         f"{k.shape[0]} and {v.shape[0]}")
    if k.shape != v.shape:
        raise ValueError(f"k {tuple(k.shape)} and v {tuple(v.shape)} differ")
    if k.shape[2] != d:
        raise ValueError(f"k/v head_dim {k.shape[2]} != q head_dim {d}")
    if tuple(o.shape) != tuple(q.shape):
        raise ValueError(f"o must have q's shape {tuple(q.shape)}, got {tuple(o.shape)}")
    if lse is not None:
        named.append(("lse", lse))
        if lse.dtype != torch.float32 or tuple(lse.shape) != (hq, total):
            raise ValueError(f"lse must be float32 [{hq}, {total}], got "
                             f"{lse.dtype} {tuple(lse.shape)}")
    named.append(("sched_dev", sched_dev))
    if not isinstance(sched_dev, torch.Tensor) or sched_dev.dtype != torch.int32:
        raise ValueError("sched_dev must be an int32 tensor of schedule words")
    if sched_dev.numel() != info.words:
        raise ValueError(f"sched_dev holds {sched_dev.numel()} words, the schedule "
                         f"info says {info.words}")
    if workspace is not None:
        named.append(("workspace", workspace))
    for name, t, dtype, shape in extra:
        named.append((name, t))
        if t.dtype != dtype or tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} must be {dtype} {tuple(shape)}, got "
                             f"{t.dtype} {tuple(t.shape)}")
    for name, t in named:
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    dev = q.device
    for name, t in named:
        if t.device != dev:
            raise ValueError(f"{name} is on {t.device}, q on {dev}: all operands "
                             "must be on one device")
    if dev.type != "cuda":
        raise ValueError(f"operands must be on a GPU, got {dev}")


def triangle_attn_fwd(q, k, v, o, lse, sched_dev, info, softmax_scale,
                      workspace, stream=None):
    """Enqueue Triangle attention on ``stream`` (torch current stream if None).

    q [T, Hq, d], k/v [T, Hkv, d] bf16 cuda tensors; o [T, Hq, d] bf16/fp32;
    lse [Hq, T] fp32 or None; sched_dev int32 cuda tensor of the schedule
    words; workspace uint8 cuda tensor of >= ta_workspace_bytes bytes or None.
    """
    _check_tensors(q, k, v, o, lse, sched_dev, info, workspace)
    total, hq, d = q.shape
    hkv = k.shape[1]
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().triangle_attn_fwd(
        _ptr(q), _ptr(k), _ptr(v), _ptr(o), _out_dtype(o), _ptr(lse),
        _ptr(sched_dev), ctypes.byref(info), total, hq, hkv, d,
        float(softmax_scale), _ptr(workspace), ws_bytes, _stream(stream)))


def triangle_attn_fwd_noalloc(q, k, v, o, lse, sched_dev, info, softmax_scale,
                              stream=None):
    """Triangle attention without a workspace argument: the split partials
    go to the library's own per-GPU scratch array (no allocation in the
    call; at most TA_NOALLOC_SCRATCH_BYTES of partials).  Calls that overlap
    on one GPU race on that array."""
    _check_tensors(q, k, v, o, lse, sched_dev, info)
    total, hq, d = q.shape
    hkv = k.shape[1]
    _check(lib().triangle_attn_fwd_noalloc(
        _ptr(q), _ptr(k), _ptr(v), _ptr(o), _out_dtype(o), _ptr(lse),
        _ptr(sched_dev), ctypes.byref(info), total, hq, hkv, d,
        float(softmax_scale), _stream(stream)))


def triangle_attn_tiles(q, k, v, o, lse, sched_dev, info, softmax_scale,
                        workspace, stream=None):
    """Enqueue the attention pass of Triangle attention (no merge)."""
    _check_tensors(q, k, v, o, lse, sched_dev, info, workspace)
    total, hq, d = q.shape
    hkv = k.shape[1]
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().triangle_attn_tiles(
        _ptr(q), _ptr(k), _ptr(v), _ptr(o), _out_dtype(o), _ptr(lse),
        _ptr(sched_dev), ctypes.byref(info), total, hq, hkv, d,
        float(softmax_scale), _ptr(workspace), ws_bytes, _stream(stream)))


def triangle_attn_merge(o, lse, sched_dev, info, workspace, stream=None):
    """Enqueue the merge of the Last-row split partials into o / lse."""
    import torch
    _out_dtype(o)
    total, hq, d = o.shape
    named = [("o", o), ("sched_dev", sched_dev)]
    if lse is not None:
        named.append(("lse", lse))
        if lse.dtype != torch.float32 or tuple(lse.shape) != (hq, total):
            raise ValueError(f"lse must be float32 [{hq}, {total}]")
    if workspace is not None:
        named.append(("workspace", workspace))
    if sched_dev.dtype != torch.int32 or sched_dev.numel() != info.words:
        raise ValueError("sched_dev must hold the schedule's int32 words")
    for name, t in named:
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        if t.device != o.device:
            raise ValueError(f"{name} is on {t.device}, o on {o.device}")
    if o.device.type != "cuda":
        raise ValueError(f"operands must be on a GPU, got {o.device}")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().triangle_attn_merge(
        _ptr(o), _out_dtype(o), _ptr(lse), _ptr(sched_dev), ctypes.byref(info),
        total, hq, d, _ptr(workspace), ws_bytes, _stream(stream)))


def blocksparse_attn_fwd(q, k, v, o, lse, sched_dev, info, softmax_scale,
                         workspace, stream=None):
    """Enqueue block-sparse causal attention (tiles + merge)."""
    _check_tensors(q, k, v, o, lse, sched_dev, info, workspace)
    total, hq, d = q.shape
    hkv = k.shape[1]
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().blocksparse_attn_fwd(
        _ptr(q), _ptr(k), _ptr(v), _ptr(o), _out_dtype(o), _ptr(lse),
        _ptr(sched_dev), ctypes.byref(info), total, hq, hkv, d,
        float(softmax_scale), _ptr(workspace), ws_bytes, _stream(stream)))


def causal_attn_fwd(q, k, v, o, lse, sched_dev, info, softmax_scale,
                    stream=None):
    """Enqueue dense causal attention on ``stream``; arguments as above."""
    _check_tensors(q, k, v, o, lse, sched_dev, info)
    total, hq, d = q.shape
    hkv = k.shape[1]
    _check(lib().causal_attn_fwd(
        _ptr(q), _ptr(k), _ptr(v), _ptr(o), _out_dtype(o), _ptr(lse),
        _ptr(sched_dev), ctypes.byref(info), total, hq, hkv, d,
        float(softmax_scale), _stream(stream)))


def ta_probe_workspace_bytes(info: ScheduleInfo, hq: int) -> int:
    return int(lib().ta_probe_workspace_bytes(ctypes.byref(info), hq))


def region_grad_probe(q, k, v, dout, lse, sched_dev, info, softmax_scale, sink,
                      window, last, region_sums, workspace, stream=None):
    """Enqueue the region-contribution probe on ``stream``.

    q, dout [T, Hq, d], k/v [T, Hkv, d] bf16 cuda tensors; lse [Hq, T] fp32
    (the causal normaliser); sched_dev/info a causal schedule; region_sums
    float64 cuda tensor [Hq, 3] (streaming, middle, last) that receives the
    per-head sums of A_ij <dO_i, V_j>; workspace uint8 cuda tensor of >=
    ta_probe_workspace_bytes bytes or None.
    """
    import torch
    if lse is None:
        raise ValueError("the probe needs the causal LSE [Hq, T]")
    if not isinstance(dout, torch.Tensor) or dout.dtype != torch.bfloat16:
        raise ValueError(f"dout must be a bfloat16 tensor, got {getattr(dout, 'dtype', dout)}")
    _check_tensors(q, k, v, dout, lse, sched_dev, info, workspace,
                   extra=(("region_sums", region_sums, torch.float64, (q.shape[1], 3)),))
    total, hq, d = q.shape
    hkv = k.shape[1]
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().region_grad_probe(
        _ptr(q), _ptr(k), _ptr(v), _ptr(dout), _ptr(lse), _ptr(sched_dev),
        ctypes.byref(info), total, hq, hkv, d, float(softmax_scale), sink, window,
        last, _ptr(region_sums), _ptr(workspace), ws_bytes, _stream(stream)))


def ta_region_counts(cu_seqlens, sink, window, last) -> np.ndarray:
    """Pairs per head in the (streaming, middle, last) sections."""
    cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
    out = np.zeros(3, dtype=np.int64)
    _check(lib().ta_region_counts(cu.ctypes.data, cu.size - 1, sink, window, last,
                                  out.ctypes.data))
    return out


def ta_region_grad_mean(region_sums, counts) -> np.ndarray:
    """Grad per section from host per-head sums [Hq, 3] and the counts."""
    sums = np.ascontiguousarray(np.asarray(region_sums, dtype=np.float64))
    cnt = np.ascontiguousarray(np.asarray(counts, dtype=np.int64))
    assert sums.ndim == 2 and sums.shape[1] == 3 and cnt.shape == (3,)
    out = np.zeros(3, dtype=np.float64)
    _check(lib().ta_region_grad_mean(sums.ctypes.data, sums.shape[0], cnt.ctypes.data,
                                     out.ctypes.data))
    return out


def region_grad(q, k, v, dout, cu_seqlens, sink, window, last, tile=128,
                softmax_scale=None, stream=None):
    """Grad(M-hat, l) of one layer for the (streaming, middle, last)
    sections, and the per-head sums behind it: the causal pass writes each
    row's LSE, the probe sums A_ij <dO_i, V_j> per head and section, and the
    library divides by Hq times the section's pair count.  Returns (grad [3],
    sums [Hq, 3]) as numpy float64; synchronises the stream to read them."""
    import torch
    total, hq, d = q.shape
    if softmax_scale is None:
        softmax_scale = 1.0 / float(d) ** 0.5
    plan = Plan("causal", cu_seqlens, 0, 1, 0, tile, hq, d, device=q.device)
    o = torch.empty(q.shape, dtype=torch.bfloat16, device=q.device)
    lse = torch.empty((hq, total), dtype=torch.float32, device=q.device)
    plan.run(q, k, v, o, lse, softmax_scale, stream)
    nbytes = ta_probe_workspace_bytes(plan.info, hq)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=q.device) if nbytes else None
    sums = torch.empty((hq, 3), dtype=torch.float64, device=q.device)
    region_grad_probe(q, k, v, dout, lse, plan.sched, plan.info, softmax_scale, sink,
                      window, last, sums, ws, stream)
    (stream or torch.cuda.current_stream()).synchronize()
    sums_host = sums.cpu().numpy()
    return ta_region_grad_mean(sums_host, ta_region_counts(cu_seqlens, sink, window, last)), \
        sums_host


def ta_select_triangle_layers(grad_middle, n_triangle) -> list:
    """The n_triangle layers with the smallest |Grad(middle)|, ascending."""
    g = np.ascontiguousarray(np.asarray(grad_middle, dtype=np.float64))
    out = np.zeros(max(int(n_triangle), 1), dtype=np.int32)
    _check(lib().ta_select_triangle_layers(g.ctypes.data if g.size else None, g.size,
                                           int(n_triangle), out.ctypes.data))
    return [int(x) for x in out[:int(n_triangle)]]


class Plan:
    """A schedule built once and uploaded to the device, plus its workspace.

    Buffers come from torch; the plan can be reused for every call with the
    same (cu_seqlens, sink, window, last, tile, splits, hq, head_dim).
    """

    def __init__(self, kind, cu_seqlens, sink, window, last, tile, hq,
                 head_dim, splits=0, device="cuda", blocks=None):
        """blocks: (qtile_ptr, ktile_idx) for kind "blocksparse" (splits is
        then the work bound per item)."""
        import torch
        self.kind = _kind(kind)
        if self.kind == BLOCKSPARSE:
            if blocks is None:
                raise ValueError("a block-sparse plan needs blocks=(qtile_ptr, ktile_idx)")
            self.words, self.info = ta_build_blocksparse_schedule(
                cu_seqlens, tile, blocks[0], blocks[1], splits)
        else:
            self.words, self.info = ta_build_schedule(self.kind, cu_seqlens, sink,
                                                      window, last, tile, splits)
        self.sched = torch.from_numpy(self.words).to(device)
        nbytes = ta_workspace_bytes(self.info, hq, head_dim)
        self.workspace = (torch.empty(nbytes, dtype=torch.uint8, device=device)
                          if nbytes > 0 else None)

    def run(self, q, k, v, o, lse=None, softmax_scale=None, stream=None):
        if softmax_scale is None:
            softmax_scale = 1.0 / float(q.shape[-1]) ** 0.5
        if self.kind == TRIANGLE:
            triangle_attn_fwd(q, k, v, o, lse, self.sched, self.info,
                              softmax_scale, self.workspace, stream)
        elif self.kind == BLOCKSPARSE:
            blocksparse_attn_fwd(q, k, v, o, lse, self.sched, self.info,
                                 softmax_scale, self.workspace, stream)
        else:
            causal_attn_fwd(q, k, v, o, lse, self.sched, self.info,
                            softmax_scale, stream)
        return o


def attention(kind, q, k, v, cu_seqlens, sink=0, window=1, last=0, tile=128,
              splits=0, softmax_scale=None, out_dtype=None, return_lse=False):
    """Allocate outputs with torch and run one pass (convenience wrapper)."""
    import torch
    out_dtype = out_dtype or torch.bfloat16
    plan = Plan(kind, cu_seqlens, sink, window, last, tile, q.shape[1],
                q.shape[2], splits, device=q.device)
    o = torch.empty(q.shape, dtype=out_dtype, device=q.device)
    lse = (torch.empty((q.shape[1], q.shape[0]), dtype=torch.float32,
                       device=q.device) if return_lse else None)
    plan.run(q, k, v, o, lse, softmax_scale)
    return (o, lse) if return_lse else o
