"""C ABI checks that need no GPU: exports, config validation, argument errors.

create / workspace_size / destroy / strerror make no HIP call, and run() rejects
bad arguments before touching the device, so all of this runs on the CPU.
"""
import ctypes
import os
import re

import pytest

from paper_2607_09207_amd import _abi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_abi.LIB_PATH):
        from paper_2607_09207_amd import build
        build.build()
    return _abi.load()


def declared_functions():
    txt = open(os.path.join(ROOT, "include", "rl_decode_attn.h")).read()
    return sorted(set(re.findall(r"^(?:rlda_status|const char\*)\s+(rl_decode_attn_\w+)\s*\(", txt, re.M)))


def test_every_declared_function_is_exported(lib):
    names = declared_functions()
    assert set(names) == set(_abi.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def test_probe_library_exports_its_declared_functions():
    """The read-bandwidth reference kernels (include/hbm_probe.h) load and export
    every declared function; argument errors return -1 before any HIP call."""
    from paper_2607_09207_amd import build, probe
    if not os.path.exists(probe.LIB_PATH):
        build.build(out=build.PROBE_LIB, sources=build.PROBE_SOURCES)
    plib = probe.load()
    txt = open(os.path.join(ROOT, "include", "hbm_probe.h")).read()
    names = sorted(set(re.findall(r"^int\s+(hbm_probe_\w+)\s*\(", txt, re.M)))
    assert names == ["hbm_probe_stream_read", "hbm_probe_tile_gather", "hbm_probe_tile_gather_balanced"]
    for n in names:
        assert hasattr(plib, n), n
    sink = ctypes.c_void_p(256)
    assert plib.hbm_probe_stream_read(None, 1024, sink, 1, 256, 8, None) == -1          # null buffer
    assert plib.hbm_probe_stream_read(ctypes.c_void_p(256), 1000, sink, 1, 256, 8, None) == -1   # not a multiple of 16
    assert plib.hbm_probe_stream_read(ctypes.c_void_p(256), 1024, sink, 1, 100, 8, None) == -1   # threads % 64
    assert plib.hbm_probe_stream_read(ctypes.c_void_p(256), 1024, sink, 1, 1024, 8, None) == -1  # more than 512 threads
    assert plib.hbm_probe_stream_read(ctypes.c_void_p(256), 1024, sink, 1, 256, 3, None) == -1   # unroll
    assert plib.hbm_probe_tile_gather(ctypes.c_void_p(256), ctypes.c_void_p(256), None, 4, 4096, sink, 1, 256, 2,
                                      None) == -1                                              # no offsets
    assert plib.hbm_probe_tile_gather(ctypes.c_void_p(256), ctypes.c_void_p(256), ctypes.c_void_p(256), 4, 1000,
                                      sink, 1, 256, 2, None) == -1                             # tile size
    assert plib.hbm_probe_tile_gather(ctypes.c_void_p(256), ctypes.c_void_p(256), ctypes.c_void_p(256), 4, 4096,
                                      sink, 1, 256, 5, None) == -1                             # depth
    pv = ctypes.c_void_p(256)
    bal = plib.hbm_probe_tile_gather_balanced
    assert bal(pv, pv, pv, 64, 0, 16, None, 4096, sink, 1, 256, 3, None) == -1    # no counter
    assert bal(pv, pv, pv, 64, 0, 2, pv, 4096, sink, 1, 256, 3, None) == -1       # chunk below the depth
    assert bal(pv, pv, pv, 64, 0, 65, pv, 4096, sink, 1, 256, 3, None) == -1      # chunk above 64
    assert bal(pv, pv, pv, 64, 10, 16, pv, 4096, sink, 1, 256, 3, None) == -1     # pool not whole chunks
    assert bal(pv, pv, pv, 64, 8, 8, pv, 4096, sink, 1, 256, 3, None) == -1       # shares of 2 entries < depth
    assert bal(pv, pv, pv, 64, 80, 16, pv, 4096, sink, 1, 256, 3, None) == -1     # more static entries than tiles
    assert bal(pv, pv, pv, 64, 0, 16, pv, 4096, sink, 1, 256, 1, None) == -1      # depth


def test_tile_offsets_follow_the_stream_order():
    import numpy as np
    from paper_2607_09207_amd import inputs as I, probe
    w = I.make_custom([17, 0, 40], 8, 2, 128, seed=3)
    off = probe.tile_offsets(w)
    sp, sh = w.strides()[0] * 2, w.strides()[1] * 2
    want = []
    for b, L in enumerate(w.seq_lens):
        n = (int(L) + 15) // 16
        for g in range(2):
            want += [int(w.block_table[b, j]) * sp + g * sh for j in range(n)]
    assert off.tolist() == want and off.dtype == np.int64


def cfg(**kw):
    c = _abi.Config()
    base = dict(num_q_heads=28, num_kv_heads=4, head_dim=128, page_size=16, max_batch=64, max_pages_per_seq=1024,
                q_dtype=_abi.RLDA_BF16, kv_dtype=_abi.RLDA_BF16, out_dtype=_abi.RLDA_F32, softmax_scale=0.0,
                kv_stride_page=0, kv_stride_head=0, kv_stride_slot=0, num_work_ranges=0)
    base.update(kw)
    for k, v in base.items():
        setattr(c, k, v)
    return c


def create(lib, c):
    h = ctypes.c_void_p()
    st = lib.rl_decode_attn_create(ctypes.byref(c), ctypes.byref(h))
    return st, h


def test_create_accepts_the_workload_configurations(lib):
    for kw in [dict(num_q_heads=4, num_kv_heads=4, head_dim=64, q_dtype=0, kv_dtype=0, out_dtype=0, max_pages_per_seq=16),
               dict(),
               dict(num_q_heads=12, num_kv_heads=2, max_batch=256, max_pages_per_seq=1568),
               dict(num_q_heads=40, num_kv_heads=8, kv_dtype=_abi.RLDA_FP8_E4M3FN, max_batch=128, max_pages_per_seq=2048),
               dict(num_q_heads=64, num_kv_heads=8, max_batch=512, max_pages_per_seq=2048, out_dtype=_abi.RLDA_BF16)]:
        st, h = create(lib, cfg(**kw))
        assert st == 0, kw
        n = ctypes.c_size_t()
        assert lib.rl_decode_attn_workspace_size(h, ctypes.byref(n)) == 0 and n.value > 0 and n.value % 256 == 0
        assert lib.rl_decode_attn_destroy(h) == 0


@pytest.mark.parametrize("kw,want", [
    (dict(num_q_heads=30), -1),                     # Hq not a multiple of Hkv
    (dict(num_kv_heads=0), -1),
    (dict(max_batch=0), -1),
    (dict(max_batch=9000), -1),
    (dict(head_dim=96), -2),
    (dict(page_size=32), -2),
    (dict(num_q_heads=68, num_kv_heads=4), -2),     # G = 17 > 16
    (dict(q_dtype=_abi.RLDA_F32), -2),              # f32 q with bf16 KV
    (dict(q_dtype=0, kv_dtype=0, out_dtype=0, num_q_heads=8, num_kv_heads=2), -2),   # f32 G*d > 128
    (dict(kv_stride_page=1000, kv_stride_head=128, kv_stride_slot=100), -1),          # slot stride < d
    (dict(kv_stride_page=1001 * 8, kv_stride_head=2048, kv_stride_slot=132), -1),      # row not 16-B aligned
    (dict(softmax_scale=-1.0), -1),
    (dict(num_work_ranges=5000), -1),
    (dict(max_batch=8192, max_pages_per_seq=65536, num_kv_heads=4, num_q_heads=28), -2),   # > 2^31 units
    # 8192 * 65535 * 4 units fit, but not with the start costs of the (sequence, KV head) segments
    (dict(max_batch=8192, max_pages_per_seq=65535, num_kv_heads=4, num_q_heads=28), -2),
])
def test_create_rejects_bad_configurations(lib, kw, want):
    st, h = create(lib, cfg(**kw))
    assert st == want and not h.value


def test_head_map_must_give_each_kv_head_g_query_heads(lib):
    c = cfg(num_q_heads=4, num_kv_heads=2)
    bad = (ctypes.c_int32 * 4)(0, 0, 0, 1)
    c.kv_head_of_q = bad
    assert create(lib, c)[0] == -1
    good = (ctypes.c_int32 * 4)(1, 0, 0, 1)
    c.kv_head_of_q = good
    st, h = create(lib, c)
    assert st == 0
    lib.rl_decode_attn_destroy(h)


def test_run_rejects_bad_arguments_before_launch(lib):
    st, h = create(lib, cfg())
    assert st == 0
    n = ctypes.c_size_t()
    lib.rl_decode_attn_workspace_size(h, ctypes.byref(n))
    fake = 0x10000   # never dereferenced: every case fails validation first
    args = dict(batch=2, num_pages=10, q=fake, k=fake, v=fake, ks=None, vs=None, bt=fake, sl=fake, out=fake,
                ws=fake * 16, wsb=n.value, stream=None)

    def run(**kw):
        a = dict(args, **kw)
        return lib.rl_decode_attn_run(h, a["batch"], a["num_pages"], a["q"], a["k"], a["v"], a["ks"], a["vs"],
                                      a["bt"], a["sl"], a["out"], a["ws"], a["wsb"], a["stream"])

    assert run(batch=65) == -1            # beyond max_batch
    assert run(batch=-1) == -1
    assert run(q=None) == -1
    assert run(k=fake + 8) == -1          # misaligned cache
    assert run(out=fake + 4) == -1
    assert run(bt=fake + 2) == -1
    assert run(ws=None) == -4
    assert run(ws=fake * 16 + 64) == -4   # workspace not 256-byte aligned
    assert run(wsb=n.value - 1) == -4
    assert run(batch=0) == 0              # nothing to do, nothing launched
    assert lib.rl_decode_attn_run(None, 1, 1, *([fake] * 8), fake, 1, None) == -1
    lib.rl_decode_attn_destroy(h)


def test_fp8_run_requires_scales(lib):
    st, h = create(lib, cfg(kv_dtype=_abi.RLDA_FP8_E4M3FN))
    n = ctypes.c_size_t()
    lib.rl_decode_attn_workspace_size(h, ctypes.byref(n))
    f = 0x10000
    assert lib.rl_decode_attn_run(h, 1, 1, f, f, f, None, None, f, f, f, f * 16, n.value, None) == -1
    assert lib.rl_decode_attn_run(h, 1, 0, f, None, None, None, None, f, f, f, None, n.value, None) == -4
    lib.rl_decode_attn_destroy(h)


def test_destroy_null_and_strerror(lib):
    assert lib.rl_decode_attn_destroy(None) == 0
    for s in (0, -1, -2, -3, -4, -5):
        assert lib.rl_decode_attn_strerror(s)
    assert lib.rl_decode_attn_strerror(7) == b"unknown status"


def test_workspace_grows_with_forced_ranges_and_kv_heads(lib):
    # partial slots per work range (16 rows each), counters per (sequence, KV head)
    sizes = []
    for kw in [dict(num_work_ranges=16), dict(num_work_ranges=512), dict(num_work_ranges=512, num_q_heads=64, num_kv_heads=8)]:
        st, h = create(lib, cfg(**kw))
        n = ctypes.c_size_t()
        lib.rl_decode_attn_workspace_size(h, ctypes.byref(n))
        sizes.append(n.value)
        lib.rl_decode_attn_destroy(h)
    assert sizes[0] < sizes[1] < sizes[2]


def test_grouped_run_rejects_bad_arguments_before_launch(lib):
    st, h = create(lib, cfg(num_q_heads=12, num_kv_heads=2, max_batch=256, max_pages_per_seq=1568))
    assert st == 0
    n, ng = ctypes.c_size_t(), ctypes.c_size_t()
    lib.rl_decode_attn_workspace_size(h, ctypes.byref(n))
    assert lib.rl_decode_attn_grouped_workspace_size(h, ctypes.byref(ng)) == 0
    # the prompt pass adds per-row (m, l, O) and one clamped length per group
    assert ng.value >= n.value + 256 * (12 * (128 + 2) + 1) * 4 and ng.value % 256 == 0
    f = 0x10000

    def run(batch=8, gs=4, pp=f, wsb=None, e0=None, e1=None, handle=h):
        return lib.rl_decode_attn_run_grouped(handle, batch, 10, gs, pp, -1, f, f, f, None, None, f, f, f, f * 16,
                                              ng.value if wsb is None else wsb, None, e0, e1)

    assert run(gs=0) == -1                # group size must be >= 1
    assert run(gs=-3) == -1
    assert run(pp=None) == -1             # prefix_pages required
    assert run(pp=f + 2) == -1            # misaligned
    assert run(e0=f) == -1                # events: both or neither
    assert run(wsb=n.value) == -4         # the plain workspace is too small for the prompt pass
    assert run(batch=300) == -1           # beyond max_batch
    assert run(batch=0) == 0
    assert lib.rl_decode_attn_grouped_workspace_size(None, ctypes.byref(ng)) == -1
    lib.rl_decode_attn_destroy(h)
    st, h32 = create(lib, cfg(num_q_heads=4, num_kv_heads=4, head_dim=64, q_dtype=0, kv_dtype=0, out_dtype=0,
                              max_pages_per_seq=16))
    assert st == 0
    lib.rl_decode_attn_grouped_workspace_size(h32, ctypes.byref(ng))
    assert run(handle=h32) == -2          # fp32 caches: no grouped path
    lib.rl_decode_attn_destroy(h32)


def test_append_rejects_bad_arguments_before_launch(lib):
    st, h = create(lib, cfg(kv_dtype=_abi.RLDA_FP8_E4M3FN))
    assert st == 0
    n = ctypes.c_size_t()
    lib.rl_decode_attn_workspace_size(h, ctypes.byref(n))
    f = 0x10000

    def app(batch=4, kn=f, vn=f, kc=f, vc=f, ks=f, vs=f, bt=f, sl=f, ws=f * 16, wsb=None):
        return lib.rl_decode_attn_append(h, batch, 10, kn, vn, kc, vc, ks, vs, bt, sl, ws,
                                         n.value if wsb is None else wsb, None)

    assert app(kn=None) == -1
    assert app(vn=f + 2) == -1            # misaligned rows
    assert app(kc=None) == -1
    assert app(ks=None) == -1             # fp8 needs scales
    assert app(sl=f + 1) == -1
    assert app(batch=65) == -1
    assert app(ws=None) == -4
    assert app(wsb=n.value - 1) == -4
    assert app(batch=0) == 0
    assert lib.rl_decode_attn_append(None, 1, 1, *([f] * 8), f, 1, None) == -1
    lib.rl_decode_attn_destroy(h)


def test_multi_rejects_bad_arguments_before_launch(lib):
    st, h = create(lib, cfg(kv_dtype=_abi.RLDA_FP8_E4M3FN, max_batch=8192, max_pages_per_seq=64))
    assert st == 0
    n = ctypes.c_size_t()
    lib.rl_decode_attn_workspace_size(h, ctypes.byref(n))
    f = 0x10000

    def multi(batch=4, total=100, q=f, ks=f, qs=f, out=f, ws=f * 16, wsb=None, e0=None, e1=None, handle=h, mq=0):
        return lib.rl_decode_attn_run_multi(handle, batch, 10, total, mq, q, f, f, ks, f, f, f, qs, out, ws,
                                            n.value if wsb is None else wsb, None, e0, e1)

    assert multi(q=None) == -1
    assert multi(q=f + 8) == -1           # misaligned
    assert multi(qs=None) == -1           # q_start required
    assert multi(qs=f + 2) == -1
    assert multi(out=None) == -1
    assert multi(ks=None) == -1           # fp8 needs scales
    assert multi(total=-1) == -1
    assert multi(e0=f) == -1              # events: both or neither
    assert multi(ws=None) == -4
    assert multi(wsb=n.value - 1) == -4
    assert multi(batch=4097) == -2        # beyond the multi-token kernel's batch limit
    assert multi(mq=-1) == -1
    # max_q_len beyond what the decode kernel's rows path takes (17 rows; 10 * G = 70
    # rows > 64): the multi-token kernel, with its batch limit
    assert multi(batch=4097, mq=17) == -2 and multi(batch=4097, mq=10) == -2
    assert multi(total=(1 << 31) // (28 * 128 * 2) + 1) == -2   # q beyond 2^31 bytes
    assert multi(batch=0) == 0 and multi(total=0) == 0
    lib.rl_decode_attn_destroy(h)
    st, h32 = create(lib, cfg(num_q_heads=4, num_kv_heads=4, head_dim=64, q_dtype=0, kv_dtype=0, out_dtype=0,
                              max_pages_per_seq=16))
    assert st == 0
    assert multi(handle=h32) == -2        # fp32 caches: no multi-token path
    lib.rl_decode_attn_destroy(h32)


def test_noalloc_rejects_requests_beyond_its_static_scratch_before_any_hip_call(lib):
    """rl_decode_attn_run_noalloc keeps counters for batch * Hkv <= 65536 segments in
    its static scratch; larger batches get RLDA_ERR_SCRATCH (-6) with nothing
    launched, and a misaligned flag word RLDA_ERR_INVALID_ARG."""
    st, h = create(lib, cfg(num_q_heads=16, num_kv_heads=16, max_batch=8192, max_pages_per_seq=4))
    assert st == 0
    p = ctypes.c_void_p(4096)
    try:
        args = lambda B, flags: (h, B, 10, p, p, p, None, None, p, p, p, flags, None)
        assert lib.rl_decode_attn_run_noalloc(*args(4097, None)) == -6     # 4097 * 16 > 65536
        assert lib.rl_decode_attn_run_noalloc(*args(8192, None)) == -6
        assert lib.rl_decode_attn_run_noalloc(*args(100, ctypes.c_void_p(4098))) == -1   # flags not 4-byte aligned
        assert lib.rl_decode_attn_run_noalloc(*args(9000, None)) == -1     # beyond max_batch
        assert lib.rl_decode_attn_run_noalloc(*args(0, None)) == 0         # empty batch: nothing to do
        assert lib.rl_decode_attn_strerror(-6).startswith(b"request exceeds the static scratch")
    finally:
        lib.rl_decode_attn_destroy(h)


def test_binding_rejects_host_tensors_before_any_launch(lib):
    import torch
    from paper_2607_09207_amd import DecodeAttention, RldaError
    h = DecodeAttention(8, 2, 128, 4, 8)
    q = torch.zeros((3, 8, 128), dtype=torch.bfloat16)
    kv = torch.zeros((5, 2, 16, 128), dtype=torch.bfloat16)
    bt, sl = torch.zeros((3, 8), dtype=torch.int32), torch.zeros(3, dtype=torch.int32)
    for fn in (h, h.run_noalloc):
        with pytest.raises(RldaError) as e:
            fn(q, kv, kv, bt, sl)
        assert e.value.status == -1 and "GPU" in str(e.value)
    with pytest.raises(RldaError):
        h.multi(q, kv, kv, bt, sl, torch.zeros(4, dtype=torch.int32))
    with pytest.raises(RldaError):
        h.append(torch.zeros((3, 2, 128), dtype=torch.bfloat16), None, kv, kv, bt, sl)
