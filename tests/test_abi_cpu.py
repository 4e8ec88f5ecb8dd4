"""The C ABI without a GPU: the library loads, exports every function that
include/conduit.h declares, and rejects bad arguments on the host before any
HIP call (nothing is launched, so no device is needed)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2609_05821_amd import api

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "conduit.h")

pytestmark = pytest.mark.skipif(not os.path.exists(api.LIB_PATH),
                                 reason="libconduit.so not built (run __graft_entry__.build())")

FAKE = 0x100000  # a 256-byte aligned non-NULL address; never dereferenced here


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(conduit_[a-z_]+)\s*\(", text)))


def test_every_declared_function_is_exported():
    L = api.lib()
    declared = header_functions()
    assert len(declared) >= 11
    for name in declared:
        assert hasattr(L, name), name
    assert sorted(declared) == sorted(api.EXPORTS)


def test_budget_closed_form():
    assert api.conduit_budget(576, 1, 10) == 57
    assert api.conduit_budget(65536, 1, 10) == 6553
    assert api.conduit_budget(100, 29, 100) == 29
    assert api.conduit_budget(16384, 1, 10) == 1638
    assert api.conduit_budget(7, 0, 1) == 0
    assert api.conduit_budget(7, 1, 1) == 7
    assert api.conduit_budget(2 ** 40, 3, 7) == (3 * 2 ** 40) // 7
    for bad in ((-1, 1, 2), (5, 1, 0), (5, -1, 2), (5, 3, 2)):
        assert api.conduit_budget(*bad) == -1


def test_status_strings_and_version():
    L = api.lib()
    names = [L.conduit_status_str(s).decode() for s in range(5)]
    assert names == ["CONDUIT_OK", "CONDUIT_ERR_INVALID_ARG", "CONDUIT_ERR_UNSUPPORTED",
                     "CONDUIT_ERR_WORKSPACE", "CONDUIT_ERR_HIP"]
    assert b"gfx950" in L.conduit_version()


def kv(**over):
    d = dict(k=FAKE, v=FAKE, k_stride=512, v_stride=512, n_ctx=1344, n_q_heads=28, n_kv_heads=4,
             head_dim=128, dtype=api.BF16)
    d.update(over)
    return api.KV(**d)


IMG = api.ImageTable([256], [0, 1024])


def score(kvd=None, q=FAKE, n_q=64, q_pos0=1280, img=IMG, norm=0, agg=0, scale=0.088, s=FAKE, a=FAKE,
          acc=0, ws=FAKE, ws_bytes=1 << 30):
    kvd = kvd or kv()
    return api.lib().conduit_score(ctypes.byref(kvd), q, n_q, q_pos0, ctypes.byref(img.desc), norm,
                                   agg, scale, None, None, None, s, a, acc, None, None, ws, ws_bytes,
                                   None)


@pytest.mark.parametrize("case,status", [
    (dict(kvd=kv(k=0)), api.ERR_INVALID_ARG),
    (dict(kvd=kv(v=FAKE + 8)), api.ERR_INVALID_ARG),
    (dict(kvd=kv(n_q_heads=30)), api.ERR_INVALID_ARG),
    (dict(kvd=kv(head_dim=96, k_stride=384, v_stride=384)), api.ERR_UNSUPPORTED),
    (dict(kvd=kv(dtype=7)), api.ERR_INVALID_ARG),
    (dict(kvd=kv(k_stride=100)), api.ERR_INVALID_ARG),
    (dict(kvd=kv(k_stride=516)), api.ERR_INVALID_ARG),
    (dict(kvd=kv(k_stride=1 << 24)), api.ERR_UNSUPPORTED),                  # a 32 MiB row
    (dict(kvd=kv(v_stride=(1 << 24) + 8)), api.ERR_UNSUPPORTED),
    (dict(q=0), api.ERR_INVALID_ARG),
    (dict(q=FAKE + 2), api.ERR_INVALID_ARG),
    (dict(n_q=0), api.ERR_INVALID_ARG),
    (dict(q_pos0=1300), api.ERR_INVALID_ARG),
    (dict(norm=5), api.ERR_INVALID_ARG),
    (dict(agg=2), api.ERR_INVALID_ARG),
    (dict(kvd=kv(n_kv_heads=512, n_q_heads=512, k_stride=65536, v_stride=65536)), api.ERR_UNSUPPORTED),
    (dict(scale=0.0), api.ERR_INVALID_ARG),
    (dict(scale=float("nan")), api.ERR_INVALID_ARG),
    (dict(s=0), api.ERR_INVALID_ARG),
    (dict(acc=2), api.ERR_INVALID_ARG),
    (dict(img=api.ImageTable([1200], [0, 1024])), api.ERR_INVALID_ARG),   # runs into the span
    (dict(img=api.ImageTable([256, 300], [0, 100, 200])), api.ERR_INVALID_ARG),  # overlap
    (dict(img=api.ImageTable([400, 256], [0, 10, 20])), api.ERR_INVALID_ARG),    # out of order
    (dict(img=api.ImageTable([256, 400], [0, 10, 10])), api.ERR_INVALID_ARG),    # empty image
    (dict(img=api.ImageTable([256], [1, 1024])), api.ERR_INVALID_ARG),
    (dict(img=api.ImageTable(list(range(0, 1028, 4)), list(range(0, 1032, 4)))), api.ERR_UNSUPPORTED),
    (dict(kvd=kv(page_size=64)), api.ERR_INVALID_ARG),                         # no table
    (dict(kvd=kv(n_pages=4)), api.ERR_INVALID_ARG),
    (dict(kvd=kv(block_table=FAKE, page_size=32, n_pages=64)), api.ERR_UNSUPPORTED),
    (dict(kvd=kv(block_table=FAKE, page_size=96, n_pages=64)), api.ERR_INVALID_ARG),
    (dict(kvd=kv(block_table=FAKE, page_size=1 << 21, n_pages=1)), api.ERR_UNSUPPORTED),
    (dict(kvd=kv(block_table=FAKE, page_size=64, n_pages=0)), api.ERR_INVALID_ARG),
    (dict(kvd=kv(block_table=FAKE + 2, page_size=64, n_pages=64)), api.ERR_INVALID_ARG),
    (dict(ws_bytes=16), api.ERR_WORKSPACE),
    (dict(ws=FAKE + 64), api.ERR_INVALID_ARG),
])
def test_score_rejects(case, status):
    assert score(**case) == status
    assert api.lib().conduit_last_error().decode() != ""


def test_image_table_n_vis_mismatch():
    img = api.ImageTable([256], [0, 1024])
    img.desc.n_vis = 1000
    assert score(img=img) == api.ERR_INVALID_ARG


def select(s=FAKE, a=FAKE, n_layers=1, img=IMG, lam=1.0, rule=0, k=102, idx=FAKE, pos=FAKE, ws=FAKE,
           ws_bytes=1 << 20):
    return api.lib().conduit_select_topk(s, a, n_layers, ctypes.byref(img.desc), lam, rule, k, idx,
                                         pos, None, None, None, None, ws, ws_bytes, None)


@pytest.mark.parametrize("case", [dict(s=0), dict(n_layers=0), dict(lam=-0.1), dict(lam=1.5),
                                  dict(lam=float("nan")), dict(k=-1), dict(k=1025), dict(idx=0),
                                  dict(pos=0), dict(rule=3), dict(rule=-1)])
def test_select_rejects(case):
    assert select(**case) == api.ERR_INVALID_ARG


def test_select_workspace_too_small():
    assert select(ws_bytes=100) == api.ERR_WORKSPACE


def test_scatter_rejects():
    L = api.lib()
    kvd = kv()
    assert L.conduit_scatter_kv(ctypes.byref(kvd), FAKE, -1, FAKE, FAKE, None, None, None) == api.ERR_INVALID_ARG
    assert L.conduit_scatter_kv(ctypes.byref(kvd), None, 3, FAKE, FAKE, None, None, None) == api.ERR_INVALID_ARG
    assert L.conduit_scatter_kv(ctypes.byref(kvd), FAKE, 3, FAKE + 4, FAKE, None, None, None) == api.ERR_INVALID_ARG
    assert L.conduit_scatter_kv(ctypes.byref(kvd), FAKE, 3, FAKE, FAKE, FAKE + 4, None, None) == api.ERR_INVALID_ARG
    assert L.conduit_scatter_kv(ctypes.byref(kvd), FAKE, 2000, FAKE, FAKE, None, None, None) == api.ERR_INVALID_ARG
    # k = 0 enqueues nothing and succeeds even without a device
    assert L.conduit_scatter_kv(ctypes.byref(kvd), None, 0, None, None, None, None, None) == api.OK


def test_refresh_rejects_and_sizes():
    L = api.lib()
    kvd = kv()
    need = L.conduit_refresh_workspace_bytes(ctypes.byref(kvd), 102)
    assert need > 0
    # fp32 needs a workspace only when the rows' keys are split over several
    # workgroups (few rows): then it holds every split's (m, l) and output
    assert L.conduit_refresh_workspace_bytes(ctypes.byref(kv(dtype=api.F32)), 102) == 0
    small = kv(dtype=api.F32, n_ctx=672, n_q_heads=8, n_kv_heads=8, head_dim=64, k_stride=512, v_stride=512)
    f32_need = L.conduit_refresh_workspace_bytes(ctypes.byref(small), 57)
    assert f32_need >= 2 * 57 * 8 * (64 * 4 + 8) and f32_need % 256 == 0
    assert L.conduit_refresh_attn(ctypes.byref(small), FAKE, FAKE, 57, 0.125, FAKE, None, FAKE, f32_need - 256,
                                  None) == api.ERR_WORKSPACE
    args = lambda **o: dict(dict(q=FAKE, pos=FAKE, k=102, scale=0.088, o=FAKE, ws=FAKE, wsb=need), **o)
    def call(a):
        return L.conduit_refresh_attn(ctypes.byref(kvd), a["q"], a["pos"], a["k"], a["scale"], a["o"],
                                      None, a["ws"], a["wsb"], None)
    assert call(args(pos=None)) == api.ERR_INVALID_ARG
    assert call(args(q=FAKE + 2)) == api.ERR_INVALID_ARG
    assert call(args(o=None)) == api.ERR_INVALID_ARG
    assert call(args(scale=-1.0)) == api.ERR_INVALID_ARG
    assert call(args(k=-1)) == api.ERR_INVALID_ARG
    assert call(args(wsb=need - 1)) == api.ERR_WORKSPACE
    assert call(args(k=0, q=None, pos=None, o=None)) == api.OK


def test_workspace_queries_are_consistent():
    L = api.lib()
    kvd = kv()
    a = L.conduit_score_workspace_bytes(ctypes.byref(kvd), 64, ctypes.byref(IMG.desc))
    assert a > 1024 * 4 * 4 * 2   # at least the two per-head partial arrays
    assert L.conduit_select_workspace_bytes(1024, 1) >= 4096
    assert L.conduit_score_workspace_bytes(ctypes.byref(kvd), 0, ctypes.byref(IMG.desc)) == 0


@pytest.mark.skipif(__import__("torch").cuda.device_count() > 0,
                    reason="needs a host without a GPU (the call would launch on fake pointers)")
def test_valid_call_without_device_reports_hip_error():
    assert score() == api.ERR_HIP
    assert "row statistics" in api.lib().conduit_last_error().decode()


def test_kernel_timing_without_records():
    """conduit_profile_*: nothing recorded before any launch; reading an
    unrecorded launch or passing NULL outputs is rejected."""
    L = api.lib()
    assert L.conduit_profile_enable(1) == api.OK
    assert L.conduit_profile_count() == 0
    name, ms = ctypes.c_char_p(), ctypes.c_float()
    assert L.conduit_profile_read(0, ctypes.byref(name), ctypes.byref(ms)) == api.ERR_INVALID_ARG
    assert L.conduit_profile_read(-1, ctypes.byref(name), ctypes.byref(ms)) == api.ERR_INVALID_ARG
    assert L.conduit_profile_read(0, None, None) == api.ERR_INVALID_ARG
    assert L.conduit_profile_enable(0) == api.OK


def test_paged_descriptor_is_accepted_on_the_host():
    """A valid paged descriptor passes every host check (the call then fails
    only at the first HIP call, or succeeds where a GPU is present)."""
    kvd = kv(block_table=FAKE, page_size=256, n_pages=8)
    L = api.lib()
    assert L.conduit_scatter_kv(ctypes.byref(kvd), None, 0, None, None, None, None, None) == api.OK
    need = L.conduit_refresh_workspace_bytes(ctypes.byref(kvd), 102)
    assert need == L.conduit_refresh_workspace_bytes(ctypes.byref(kv()), 102)


def test_value_norms_rejects():
    L = api.lib()
    out = ctypes.c_void_p(FAKE)
    assert L.conduit_value_norms(ctypes.byref(kv()), ctypes.byref(IMG.desc), None, None) == api.ERR_INVALID_ARG
    assert L.conduit_value_norms(ctypes.byref(kv(v=0)), ctypes.byref(IMG.desc), out, None) == api.ERR_INVALID_ARG
    bad = api.ImageTable([1500], [0, 1024])  # runs past the cache
    assert L.conduit_value_norms(ctypes.byref(kv()), ctypes.byref(bad.desc), out, None) == api.ERR_INVALID_ARG


def residual(kvd=None, q=FAKE, n_q=64, q_pos0=1280, img=IMG, scale=0.088, lse=FAKE, refreshed=FAKE,
             z=FAKE, n_samples=5, kappa=0.5, err=FAKE, ws=FAKE, ws_bytes=1 << 30):
    kvd = kvd or kv()
    return api.lib().conduit_residual_error(ctypes.byref(kvd), q, n_q, q_pos0, ctypes.byref(img.desc), scale,
                                            lse, refreshed, z, n_samples, kappa, err, ws, ws_bytes, None)


@pytest.mark.parametrize("case,status", [
    (dict(lse=None), api.ERR_INVALID_ARG),
    (dict(refreshed=None), api.ERR_INVALID_ARG),
    (dict(err=None), api.ERR_INVALID_ARG),
    (dict(z=FAKE + 4), api.ERR_INVALID_ARG),
    (dict(kappa=0.0), api.ERR_INVALID_ARG),
    (dict(kappa=float("inf")), api.ERR_INVALID_ARG),
    (dict(n_samples=0), api.ERR_INVALID_ARG),
    (dict(z=None, n_samples=2), api.ERR_INVALID_ARG),
    (dict(n_samples=20000), api.ERR_UNSUPPORTED),
    (dict(q_pos0=1300), api.ERR_INVALID_ARG),
    (dict(scale=-1.0), api.ERR_INVALID_ARG),
    (dict(img=api.ImageTable([1200], [0, 1024])), api.ERR_INVALID_ARG),
    (dict(ws_bytes=64), api.ERR_WORKSPACE),
    (dict(kvd=kv(head_dim=96, k_stride=384, v_stride=384)), api.ERR_UNSUPPORTED),
])
def test_residual_rejects(case, status):
    assert residual(**case) == status


def test_residual_workspace_sizes():
    L = api.lib()
    kvd = kv()
    iso = L.conduit_residual_workspace_bytes(ctypes.byref(kvd), 64, ctypes.byref(IMG.desc), 5, 1)
    proj = L.conduit_residual_workspace_bytes(ctypes.byref(kvd), 64, ctypes.byref(IMG.desc), 1, 0)
    assert iso > proj > 64 * 28 * 4
    assert L.conduit_residual_workspace_bytes(ctypes.byref(kvd), 0, ctypes.byref(IMG.desc), 5, 1) == 0


def test_ceiling_reference_library():
    """The benchmark's matrix-core reference (a separate library, not part of
    the C ABI): it loads, sizes its operands and counts its FLOP without a
    GPU, and rejects bad arguments before launching."""
    path = os.path.join(ROOT, "paper_2609_05821_amd", "libconduit_ceiling.so")
    if not os.path.exists(path):
        pytest.skip("libconduit_ceiling.so not built")
    L = ctypes.CDLL(path)
    L.conduit_ceiling_ops_bytes.restype = ctypes.c_int64
    L.conduit_ceiling_ops_bytes.argtypes = [ctypes.c_int32]
    L.conduit_ceiling_flop.restype = ctypes.c_double
    L.conduit_ceiling_flop.argtypes = [ctypes.c_int32, ctypes.c_int32]
    L.conduit_ceiling_mfma_bf16.restype = ctypes.c_int
    L.conduit_ceiling_mfma_bf16.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                            ctypes.c_void_p]
    assert L.conduit_ceiling_ops_bytes(2) == 2 * 256 * 16 * 16
    # 4 waves x 16 products of 2*32*32*16 FLOP per iteration and workgroup
    assert L.conduit_ceiling_flop(3, 5) == 3 * 4 * 5 * 16 * 32768.0
    assert L.conduit_ceiling_mfma_bf16(None, FAKE, 1, 1, None) != 0
    assert L.conduit_ceiling_mfma_bf16(FAKE + 8, FAKE, 1, 1, None) != 0
    assert L.conduit_ceiling_mfma_bf16(FAKE, FAKE, 0, 1, None) != 0


def test_noalloc_rejects_calls_beyond_its_scratch():
    """conduit_score_noalloc refuses, before any HIP call, a call whose
    workspace exceeds its fixed scratch (256 KV heads: the per-head column sums
    alone need 2 * 256 * 4 bytes per visual token)."""
    import ctypes
    L = api.lib()
    fake = 1 << 20  # aligned, never dereferenced: the call is refused first
    n_vis = 9000
    kv = api.KV(fake, fake, 256 * 64, 256 * 64, n_vis + 64, 256, 256, 64, api.BF16, 0, None, 0)
    img = api.ImageTable([16], [0, n_vis])
    need = api.score_workspace_bytes(kv, 8, img)
    assert need > api.SCORE_NOALLOC_MAX_BYTES
    st = L.conduit_score_noalloc(ctypes.byref(kv), fake, 8, n_vis + 16, ctypes.byref(img.desc), 0, 0, 0.125,
                                 None, None, None, fake, fake, 0, None, None, None)
    assert st == api.ERR_UNSUPPORTED
    assert b"conduit_score_noalloc holds at most" in L.conduit_last_error()
    # an invalid argument is still reported as such
    st = L.conduit_score_noalloc(None, fake, 8, 0, ctypes.byref(img.desc), 0, 0, 0.125,
                                 None, None, None, fake, fake, 0, None, None, None)
    assert st == api.ERR_INVALID_ARG


def test_layer_calls_reject_and_size():
    """The multi-layer merge and refresh validate every layer before anything
    is enqueued; the refresh workspace covers the split partials of 16 layers."""
    L = api.lib()
    good = (api.KV * 3)(kv(), kv(k=FAKE + 4096, v=FAKE + 8192), kv())
    ptrs = (ctypes.c_void_p * 3)(FAKE, FAKE, FAKE)
    bad_shape = (api.KV * 2)(kv(), kv(n_ctx=1000))
    bad_align = (ctypes.c_void_p * 3)(FAKE, FAKE + 4, FAKE)
    null_entry = (ctypes.c_void_p * 3)(FAKE, None, FAKE)
    sc = L.conduit_scatter_kv_layers
    assert sc(good, 0, FAKE, 3, ptrs, ptrs, None) == api.ERR_INVALID_ARG
    assert sc(None, 1, FAKE, 3, ptrs, ptrs, None) == api.ERR_INVALID_ARG
    assert sc(bad_shape, 2, FAKE, 3, ptrs, ptrs, None) == api.ERR_INVALID_ARG
    assert sc(good, 3, FAKE, 3, bad_align, ptrs, None) == api.ERR_INVALID_ARG
    assert sc(good, 3, FAKE, 3, ptrs, null_entry, None) == api.ERR_INVALID_ARG
    assert sc(good, 3, None, 3, ptrs, ptrs, None) == api.ERR_INVALID_ARG
    assert sc(good, 3, None, 0, None, None, None) == api.OK  # k = 0: nothing to do
    rf = L.conduit_refresh_attn_layers
    one = L.conduit_refresh_workspace_bytes(ctypes.byref(good[0]), 300)
    many = L.conduit_refresh_layers_workspace_bytes(ctypes.byref(good[0]), 300, 20)
    assert L.conduit_refresh_layers_workspace_bytes(ctypes.byref(good[0]), 300, 1) == one
    assert many > one
    assert L.conduit_refresh_layers_workspace_bytes(ctypes.byref(good[0]), 300, 16) == many
    assert L.conduit_refresh_layers_workspace_bytes(ctypes.byref(good[0]), 300, 0) == 0
    assert rf(bad_shape, 2, ptrs, FAKE, 300, 0.1, ptrs, None, FAKE, many, None) == api.ERR_INVALID_ARG
    assert rf(good, 3, ptrs, FAKE, 300, 0.1, bad_align, None, FAKE, many, None) == api.ERR_INVALID_ARG
    assert rf(good, 3, ptrs, FAKE, 300, -1.0, ptrs, None, FAKE, many, None) == api.ERR_INVALID_ARG
    need3 = L.conduit_refresh_layers_workspace_bytes(ctypes.byref(good[0]), 300, 3)
    assert one < need3 < many
    assert rf(good, 3, ptrs, FAKE, 300, 0.1, ptrs, None, FAKE, need3 - 256, None) == api.ERR_WORKSPACE
    assert rf(good, 3, ptrs, None, 0, 0.1, ptrs, None, None, 0, None) == api.OK


def test_score_layers_reject_and_size():
    """The multi-layer scoring validates every layer and argument before
    anything is enqueued; its workspace covers 16 layers' partials (bf16) or
    one layer's (fp32, which runs the per-layer calls)."""
    L = api.lib()
    good = (api.KV * 3)(kv(), kv(k=FAKE + 4096, v=FAKE + 8192), kv())
    qs = (ctypes.c_void_p * 3)(FAKE, FAKE, FAKE)
    img = ctypes.byref(IMG.desc)
    one = L.conduit_score_workspace_bytes(ctypes.byref(good[0]), 64, img)
    sz = lambda n, k=good[0]: L.conduit_score_layers_workspace_bytes(ctypes.byref(k), 64, img, n)
    assert sz(1) == one
    assert sz(0) == 0
    assert one < sz(3) < sz(16)
    assert sz(16) == sz(20)
    f32 = kv(dtype=api.F32, n_q_heads=8, n_kv_heads=8, head_dim=64, k_stride=512, v_stride=512)
    assert sz(5, f32) == L.conduit_score_workspace_bytes(ctypes.byref(f32), 64, img)
    need = sz(3)
    sc = L.conduit_score_layers

    def call(kvs=good, n=3, q=qs, n_q=64, q_pos0=1280, norm=api.NORM_CAUSAL_ROW, agg=api.AGG_MEAN, scale=0.1,
             s_acc=FAKE, acc=0, nbytes=need):
        return sc(kvs, n, q, n_q, q_pos0, img, norm, agg, scale, None, s_acc, FAKE, acc, FAKE, nbytes, None)

    assert call(n=0) == api.ERR_INVALID_ARG
    assert call(kvs=None) == api.ERR_INVALID_ARG
    assert call(kvs=(api.KV * 2)(kv(), kv(n_ctx=1000)), n=2) == api.ERR_INVALID_ARG
    assert call(q=None) == api.ERR_INVALID_ARG
    assert call(q=(ctypes.c_void_p * 3)(FAKE, FAKE + 4, FAKE)) == api.ERR_INVALID_ARG
    assert call(q=(ctypes.c_void_p * 3)(FAKE, None, FAKE)) == api.ERR_INVALID_ARG
    assert call(n_q=0) == api.ERR_INVALID_ARG
    assert call(q_pos0=1300) == api.ERR_INVALID_ARG
    assert call(norm=7) == api.ERR_INVALID_ARG
    assert call(agg=9) == api.ERR_INVALID_ARG
    assert call(scale=0.0) == api.ERR_INVALID_ARG
    assert call(s_acc=None) == api.ERR_INVALID_ARG
    assert call(acc=2) == api.ERR_INVALID_ARG
    assert call(nbytes=need - 256) == api.ERR_WORKSPACE


def test_score_rejects_span_queries_past_2_gib():
    """bf16 scoring reads the span's queries with 32-bit byte offsets: a span
    of 2^31 bytes or more is refused before anything is enqueued."""
    L = api.lib()
    big = kv(n_ctx=1 << 20, n_q_heads=256, n_kv_heads=256, k_stride=256 * 128, v_stride=256 * 128)
    img = api.ImageTable([256], [0, 1024])
    n_q = 32768  # 32768 * 256 heads * 128 dims * 2 bytes = 2^31
    assert L.conduit_score(ctypes.byref(big), FAKE, n_q, 1280, ctypes.byref(img.desc), api.NORM_CAUSAL_ROW,
                           api.AGG_MEAN, 0.1, None, None, None, FAKE, FAKE, 0, None, None, FAKE, 1 << 40,
                           None) == api.ERR_UNSUPPORTED
    assert b"2^31" in L.conduit_last_error()


def test_merge_refresh_rejects_before_enqueueing():
    """conduit_merge_refresh_attn checks the merge's and the refresh's
    arguments and the workspace before anything is enqueued."""
    L = api.lib()
    d = kv()
    need = L.conduit_refresh_workspace_bytes(ctypes.byref(d), 300)
    mr = L.conduit_merge_refresh_attn

    def call(kvd=d, pos=FAKE, k=300, kn=FAKE, vn=FAKE, q=FAKE, scale=0.1, o=FAKE, nbytes=need):
        return mr(ctypes.byref(kvd) if kvd is not None else None, pos, k, kn, vn, q, scale, o, None, FAKE, nbytes,
                  None)

    assert call(kvd=None) == api.ERR_INVALID_ARG
    assert call(k=-1) == api.ERR_INVALID_ARG
    assert call(k=2000) == api.ERR_INVALID_ARG
    assert call(scale=0.0) == api.ERR_INVALID_ARG
    assert call(pos=None) == api.ERR_INVALID_ARG
    assert call(kn=None) == api.ERR_INVALID_ARG
    assert call(vn=FAKE + 4) == api.ERR_INVALID_ARG
    assert call(q=None) == api.ERR_INVALID_ARG
    assert call(o=FAKE + 8) == api.ERR_INVALID_ARG
    assert call(nbytes=need - 256) == api.ERR_WORKSPACE
    assert call(k=0, pos=None, kn=None, vn=None, q=None, o=None, nbytes=0) == api.OK
