"""The C interface: symbols, versions and argument checking.

Runs without a GPU: every call here is rejected by the host-side checks,
before any HIP call, so nothing is launched.
"""
import ctypes
import re

import numpy as np
import pytest

from paper_2507_21526_amd import binding as B


def _declared_functions():
    text = open(B.HEADER_PATH).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, re.M)
    return sorted(set(n for n in names if n not in ("defined",)))


def test_library_exports_every_declared_function():
    names = _declared_functions()
    assert {"ta_build_schedule", "ta_workspace_bytes", "triangle_attn_fwd",
            "causal_attn_fwd", "ta_last_error", "ta_abi_version"} <= set(names)
    lib = B.lib()
    for n in names:
        assert hasattr(lib, n), n


def test_versions_match_header():
    text = open(B.HEADER_PATH).read()
    abi = int(re.search(r"#define TA_ABI_VERSION (\d+)", text).group(1))
    ver = int(re.search(r"#define TA_SCHEDULE_VERSION (\d+)", text).group(1))
    assert B.ta_abi_version() == abi
    _, info = B.ta_build_schedule("triangle", [0, 100], 4, 8, 2, 64)
    assert info.version == ver


def _status_build(**kw):
    args = dict(kind=0, cu=[0, 100], sink=4, window=8, last=2, tile=64,
                splits=0, out=None, out_words=0)
    args.update(kw)
    cu = np.asarray(args["cu"], dtype=np.int32)
    info = B.ScheduleInfo()
    st = B.lib().ta_build_schedule(args["kind"], cu.ctypes.data, cu.size - 1,
                                   args["sink"], args["window"], args["last"],
                                   args["tile"], args["splits"], args["out"],
                                   args["out_words"], ctypes.byref(info))
    return st, info


def test_build_schedule_rejects_bad_arguments():
    assert _status_build()[0] == B.TA_OK
    assert _status_build(kind=7)[0] == B.TA_ERR_INVALID_ARG
    assert _status_build(window=0)[0] == B.TA_ERR_INVALID_ARG
    assert _status_build(sink=-1)[0] == B.TA_ERR_INVALID_ARG
    assert _status_build(last=-1)[0] == B.TA_ERR_INVALID_ARG
    assert _status_build(splits=-2)[0] == B.TA_ERR_INVALID_ARG
    assert _status_build(tile=32)[0] == B.TA_ERR_UNSUPPORTED
    assert _status_build(cu=[0, 50, 40])[0] == B.TA_ERR_INVALID_ARG
    assert _status_build(cu=[5, 50])[0] == B.TA_ERR_INVALID_ARG
    st = B.lib().ta_build_schedule(0, None, 1, 0, 1, 0, 64, 0, None, 0, None)
    assert st == B.TA_ERR_INVALID_ARG
    assert "info" in B.ta_last_error()


def test_build_schedule_size_query_and_small_buffer():
    st, info = _status_build()
    assert st == B.TA_OK and info.words > 16
    buf = np.full(info.words - 1, -7, dtype=np.int32)
    st, info2 = _status_build(out=buf.ctypes.data, out_words=buf.size)
    assert st == B.TA_ERR_BUFFER_TOO_SMALL
    assert np.all(buf == -7)            # nothing written
    assert info2.words == info.words
    assert "needs" in B.ta_last_error()


def test_empty_and_zero_length_sequences():
    words, info = B.ta_build_schedule("triangle", [0], 4, 8, 2, 64)
    assert info.n_items == 0 and info.total_tokens == 0 and words.size == 16
    words, info = B.ta_build_schedule("triangle", [0, 0, 0], 4, 8, 2, 64)
    assert info.n_items == 0 and info.n_merge_items == 0
    assert B.ta_workspace_bytes(info, 8, 128) == 0


def test_workspace_bytes():
    _, info = B.ta_build_schedule("triangle", [0, 131072], 128, 2048, 128, 128)
    rows = 57 * 128 * 32
    want = ((rows * 128 * 4 + 255) // 256) * 256 + ((rows * 4 + 255) // 256) * 256
    assert B.ta_workspace_bytes(info, 32, 128) == want
    _, cinfo = B.ta_build_schedule("causal", [0, 131072], 128, 2048, 128, 128)
    assert B.ta_workspace_bytes(cinfo, 32, 128) == 0


FAKE = 0x10000  # never dereferenced: every call below fails its checks first


def _fwd(fn="triangle", info=None, total=100, hq=8, hkv=2, d=128, scale=0.1,
         o_dtype=0, ptr=FAKE, ws=FAKE, ws_bytes=1 << 30, sched=FAKE):
    L = B.lib()
    pinfo = ctypes.byref(info) if info is not None else None
    p = ctypes.c_void_p(ptr)
    if fn in ("triangle", "blocksparse"):
        f = L.triangle_attn_fwd if fn == "triangle" else L.blocksparse_attn_fwd
        return f(p, p, p, p, o_dtype, None,
                                   ctypes.c_void_p(sched), pinfo, total, hq,
                                   hkv, d, scale, ctypes.c_void_p(ws),
                                   ws_bytes, None)
    return L.causal_attn_fwd(p, p, p, p, o_dtype, None, ctypes.c_void_p(sched),
                             pinfo, total, hq, hkv, d, scale, None)


def test_fwd_rejects_bad_arguments_without_launching():
    _, tri = B.ta_build_schedule("triangle", [0, 100], 4, 8, 2, 64)
    _, cau = B.ta_build_schedule("causal", [0, 100], 4, 8, 2, 64)
    assert _fwd(info=None) == B.TA_ERR_INVALID_ARG
    assert _fwd(info=cau) == B.TA_ERR_SCHEDULE_MISMATCH
    assert _fwd("causal", info=tri) == B.TA_ERR_SCHEDULE_MISMATCH
    assert _fwd(info=tri, total=99) == B.TA_ERR_SCHEDULE_MISMATCH
    assert _fwd(info=tri, hq=7, hkv=2) == B.TA_ERR_INVALID_ARG
    assert _fwd(info=tri, hq=0) == B.TA_ERR_INVALID_ARG
    assert _fwd(info=tri, hq=18, hkv=2) == B.TA_ERR_UNSUPPORTED
    assert _fwd(info=tri, d=96) == B.TA_ERR_UNSUPPORTED
    assert _fwd(info=tri, o_dtype=5) == B.TA_ERR_INVALID_ARG
    assert _fwd(info=tri, scale=0.0) == B.TA_ERR_INVALID_ARG
    assert _fwd(info=tri, scale=float("nan")) == B.TA_ERR_INVALID_ARG
    assert _fwd(info=tri, ptr=0) == B.TA_ERR_INVALID_ARG
    assert _fwd(info=tri, ptr=FAKE + 2) == B.TA_ERR_INVALID_ARG
    assert _fwd(info=tri, sched=0) == B.TA_ERR_INVALID_ARG
    assert _fwd(info=tri, ws=0) == B.TA_ERR_WORKSPACE
    assert _fwd(info=tri, ws_bytes=16) == B.TA_ERR_WORKSPACE
    assert "workspace" in B.ta_last_error()
    bad = B.ScheduleInfo.from_buffer_copy(tri)
    bad.version = 99
    assert _fwd(info=bad) == B.TA_ERR_SCHEDULE_MISMATCH
    bad = B.ScheduleInfo.from_buffer_copy(tri)
    bad.tile = 32
    assert _fwd(info=bad) == B.TA_ERR_UNSUPPORTED
    assert _fwd("causal", info=cau, d=80) == B.TA_ERR_UNSUPPORTED
    # row pitches of Q (2 hq d bytes) and K/V must stay below 2^24 bytes:
    # hq 65536 with d 128 is rejected even though hkv alone would pass
    assert _fwd(info=tri, hq=65536, hkv=8192) == B.TA_ERR_UNSUPPORTED
    assert "hq * head_dim" in B.ta_last_error()
    assert _fwd("causal", info=cau, hq=65536, hkv=8192) == B.TA_ERR_UNSUPPORTED
    # the word count must match the items (and a block-sparse list section)
    bad = B.ScheduleInfo.from_buffer_copy(tri)
    bad.words += 1
    assert _fwd(info=bad) == B.TA_ERR_SCHEDULE_MISMATCH
    _, bs = B.ta_build_blocksparse_schedule([0, 100], 64, [0, 1, 3], [0, 0, 1], 1)
    assert bs.window == 3
    assert _fwd("blocksparse", info=bs, ws=0) == B.TA_ERR_WORKSPACE  # checks passed
    assert _fwd("blocksparse", info=tri) == B.TA_ERR_SCHEDULE_MISMATCH
    for field, delta in (("words", -1), ("window", 1), ("window", -4)):
        bad = B.ScheduleInfo.from_buffer_copy(bs)
        setattr(bad, field, getattr(bad, field) + delta)
        assert _fwd("blocksparse", info=bad) == B.TA_ERR_SCHEDULE_MISMATCH, field


def test_noalloc_rejects_partials_beyond_the_scratch_size():
    """triangle_attn_fwd_noalloc refuses, before any HIP call, a schedule
    whose split partials exceed the library's scratch array."""
    text = open(B.HEADER_PATH).read()
    limit = re.search(r"#define TA_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", text)
    limit = int(limit.group(1)) << int(limit.group(2))
    assert limit == 128 << 20
    cu = [0, 8192, 32768, 81920, 147456]   # four packed sequences, automatic splits
    _, info = B.ta_build_schedule("triangle", cu, 128, 2048, 128, 128)
    need = B.ta_workspace_bytes(info, 32, 128)
    assert need > limit
    L = B.lib()
    p = ctypes.c_void_p(FAKE)
    st = L.triangle_attn_fwd_noalloc(p, p, p, p, 0, None, p, ctypes.byref(info),
                                     cu[-1], 32, 8, 128, 0.1, None)
    assert st == B.TA_ERR_WORKSPACE
    assert "scratch holds" in B.ta_last_error()
    # the ordinary checks come first
    st = L.triangle_attn_fwd_noalloc(p, p, p, p, 0, None, p, ctypes.byref(info),
                                     cu[-1] - 1, 32, 8, 128, 0.1, None)
    assert st == B.TA_ERR_SCHEDULE_MISMATCH
    _, cau = B.ta_build_schedule("causal", [0, 100], 4, 8, 2, 64)
    st = L.triangle_attn_fwd_noalloc(p, p, p, p, 0, None, p, ctypes.byref(cau),
                                     100, 8, 2, 128, 0.1, None)
    assert st == B.TA_ERR_SCHEDULE_MISMATCH


def _host_tensors(total=100, hq=8, hkv=2, d=128):
    import torch
    q = torch.zeros((total, hq, d), dtype=torch.bfloat16)
    k = torch.zeros((total, hkv, d), dtype=torch.bfloat16)
    v = torch.zeros((total, hkv, d), dtype=torch.bfloat16)
    o = torch.zeros((total, hq, d), dtype=torch.float32)
    lse = torch.zeros((hq, total), dtype=torch.float32)
    return q, k, v, o, lse


def test_binding_rejects_bad_tensors_before_any_gpu_call():
    """The binding checks dtypes, contiguity, shapes and devices of the
    tensors whose raw pointers it passes; every case here is CPU tensors
    and fails in Python before anything is enqueued."""
    import torch
    words, info = B.ta_build_schedule("triangle", [0, 100], 4, 8, 2, 64)
    sched = torch.from_numpy(words)
    ws = torch.zeros(B.ta_workspace_bytes(info, 8, 128), dtype=torch.uint8)

    def call(q, k, v, o, lse, s=sched, fn=B.triangle_attn_fwd):
        fn(q, k, v, o, lse, s, info, 0.1, ws)

    q, k, v, o, lse = _host_tensors()
    cases = {
        "q must be bfloat16": (q.half(), k, v, o, lse),
        "k must be bfloat16": (q, k.float(), v, o, lse),
        "v must be [tokens": (q, k, v[0], o, lse),
        "k and v must have 100 tokens": (q, k[:99], v[:99], o, lse),
        "differ": (q, k, v[:, :1], o, lse),
        "head_dim 64": (q, k[..., :64], v[..., :64], o, lse),
        "o must have q's shape": (q, k, v, o[:50], lse),
        "o must be bf16 or fp32": (q, k, v, o.half(), lse),
        "lse must be float32": (q, k, v, o, lse.T.contiguous()),
        "q must be contiguous": (q.transpose(0, 1).contiguous().transpose(0, 1), k, v, o, lse),
        "k must be contiguous": (q, torch.zeros((100, 4, 128), dtype=torch.bfloat16)[:, ::2],
                                 v, o, lse),
        "operands must be on a GPU": (q, k, v, o, lse),
    }
    for msg, args in cases.items():
        with pytest.raises(ValueError, match=re.escape(msg)):
            call(*args)
    with pytest.raises(ValueError, match="sched_dev holds"):
        call(q, k, v, o, lse, s=sched[:-1])
    with pytest.raises(ValueError, match="int32"):
        call(q, k, v, o, lse, s=sched.long())
    for fn in (B.triangle_attn_tiles, B.blocksparse_attn_fwd):
        with pytest.raises(ValueError, match="k and v must have"):
            call(q, k[:99], v[:99], o, lse, fn=fn)
    _, cinfo = B.ta_build_schedule("causal", [0, 100], 4, 8, 2, 64)
    with pytest.raises(ValueError, match="o must have"):
        B.causal_attn_fwd(q, k, v, o[:, :4], lse, sched, cinfo, 0.1)
    with pytest.raises(ValueError, match="lse must be"):
        B.triangle_attn_merge(o, lse[:4], sched, info, ws)
    with pytest.raises(ValueError, match="must be on a GPU"):
        B.triangle_attn_merge(o, lse, sched, info, ws)
    sums = torch.zeros((8, 3), dtype=torch.float64)
    with pytest.raises(ValueError, match="region_sums"):
        B.region_grad_probe(q, k, v, q, lse, sched, info, 0.1, 4, 8, 2, sums[:4], ws)
    with pytest.raises(ValueError, match="dout must be"):
        B.region_grad_probe(q, k, v, q.float(), lse, sched, info, 0.1, 4, 8, 2, sums, ws)


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="missing"):
        B.lib()
