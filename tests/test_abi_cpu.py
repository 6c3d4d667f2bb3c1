"""CPU tests of the C ABI library: it loads, exports every function include/delta_attn.h
declares, and rejects bad arguments on the host before touching the GPU."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "delta_attn.h")
PROBE_HEADER = os.path.join(ROOT, "include", "delta_probe.h")


@pytest.fixture(scope="module")
def D():
    from paper_2510_09883_amd import delta
    return delta


def declared_functions(path=HEADER):
    text = open(path).read()
    return sorted(set(re.findall(r"^\s*(?:int|const char\*)\s+(delta_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_symbol(D):
    names = declared_functions()
    assert len(names) == 12
    lib = ctypes.CDLL(D.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(D.EXPORTED) == names
    probe = declared_functions(PROBE_HEADER)
    assert probe == ["delta_hbm_gather_probe", "delta_hbm_read_probe"]
    assert all(hasattr(lib, n) for n in probe)


def test_probe_rejects_bad_arguments(D):
    lib = D._lib
    fake = ctypes.c_void_p(0x1000)
    assert lib.delta_hbm_read_probe(None, 1 << 20, fake, 64, 4, None) == -1
    assert lib.delta_hbm_read_probe(fake, 1 << 20, fake, 64, 3, None) == -1
    assert lib.delta_hbm_read_probe(ctypes.c_void_p(0x1001), 1 << 20, fake, 64, 4, None) == -1
    g = lib.delta_hbm_gather_probe
    assert g(None, 1 << 20, fake, 16, fake, 4, None) == -1           # no buffer
    assert g(fake, 1 << 20, None, 16, fake, 4, None) == -1           # no chunk list
    assert g(fake, 1 << 20, fake, 0, fake, 4, None) == -1            # nothing to read
    assert g(fake, 1 << 20, fake, 4096 * 4 + 1, fake, 4, None) == -1  # > 4096 chunks per workgroup
    assert g(ctypes.c_void_p(0x1001), 1 << 20, fake, 16, fake, 4, None) == -1


def test_build_flags(D):
    """The library the binding loads is the release build; the debug build, where it has been
    built (python -m paper_2510_09883_amd.build --debug), says so."""
    if not os.environ.get("DELTA_ATTN_LIB"):
        assert D.delta_build_flags() == 0
    dbg = os.path.join(ROOT, "paper_2510_09883_amd", "libdelta_attn_debug.so")
    if os.path.exists(dbg):
        lib = ctypes.CDLL(dbg)
        assert lib.delta_build_flags() == D.DELTA_BUILD_DEBUG


def test_negative_page_count_is_refused(D):
    s = shape(D)
    kv = D.delta_kv_t(1, 2, 3, 4, -1)
    fake = ctypes.c_void_p(0x1000)
    need = D.delta_workspace_bytes(s)
    assert D._lib.delta_full_attn(ctypes.byref(s), ctypes.byref(kv), fake, fake, fake, need, None) == -1


def test_status_strings(D):
    assert D.delta_status_string(0) == "ok"
    assert D.delta_status_string(-3) == "workspace too small"


def shape(D, **kw):
    s = dict(batch=2, n_q_heads=32, n_kv_heads=8, head_dim=128, max_pages_per_seq=512,
             max_seq_len=8192)
    s.update(kw)
    return D.make_shape(**s)


def test_workspace_sizes(D):
    s = shape(D)
    a = D.delta_workspace_bytes(s)
    b = D.delta_workspace_bytes(s, D.make_select(2048, 128))
    c = D.delta_workspace_bytes(s, D.make_select(2048, 128, unit_tokens=1))
    # the Delta path adds fp32 logits [B, Hq, s] + log-sum-exp + unit scores
    assert b >= a + 4 * 2 * 32 * 8192
    assert c > b
    assert a % 256 == 0 and b % 256 == 0


@pytest.mark.parametrize("kw,status", [
    (dict(n_kv_heads=5), -1),          # Hq % Hkv != 0
    (dict(head_dim=96), -2),           # unsupported head dim
    (dict(page_size=32), -2),          # page size must be 16
    (dict(n_kv_heads=2), -2),          # group 16 > 8 not built
    (dict(max_seq_len=8193), -1),      # more tokens than the page table holds
    (dict(batch=0), -1),
    (dict(sm_scale=-1.0), -1),
])
def test_shape_validation(D, kw, status):
    with pytest.raises(D.DeltaError) as e:
        D.delta_workspace_bytes(shape(D, **kw))
    assert e.value.status == status


@pytest.mark.parametrize("sel,status", [
    ((2048, 2048), -1),                # L >= K (only L < K is valid, App. C)
    ((2048, 4096), -1),
    ((2040, 128), -1),                 # budget not a whole number of pages
    ((2048, 2033), -1),                # a window of 2033 tokens rounds up to 128 pages = K
    ((0, 0), -1),
])
def test_select_validation(D, sel, status):
    with pytest.raises(D.DeltaError) as e:
        D.delta_workspace_bytes(shape(D), D.make_select(*sel))
    assert e.value.status == status
    with pytest.raises(D.DeltaError):
        D.delta_workspace_bytes(shape(D), D.make_select(2048, 128, unit_tokens=8))
    with pytest.raises(D.DeltaError):
        D.delta_workspace_bytes(shape(D), D.make_select(2048, 128, agg=2))


@pytest.mark.parametrize("budget,recent", [(2048, 120), (2048, 8), (2048, 2032), (128, 1), (32, 15)])
def test_recency_window_of_any_token_count(D, budget, recent):
    """App. A, Alg. 1 keeps ceil(L / P) pages for a window of L tokens: a window that is not a
    whole number of pages is valid as long as its rounded-up page count stays below K."""
    assert D.delta_workspace_bytes(shape(D), D.make_select(budget, recent)) > 0
    # token-level units take every window as is
    assert D.delta_workspace_bytes(shape(D), D.make_select(budget, recent, unit_tokens=1)) > 0


def test_selection_key_limit(D):
    # token-level units: at most 8192 candidate units per sequence
    ok = shape(D, max_pages_per_seq=1024, max_seq_len=8192 + 128)
    assert D.delta_workspace_bytes(ok, D.make_select(2048, 128, unit_tokens=1)) > 0
    big = shape(D, max_pages_per_seq=1024, max_seq_len=8192 + 129)
    with pytest.raises(D.DeltaError) as e:
        D.delta_workspace_bytes(big, D.make_select(2048, 128, unit_tokens=1))
    assert e.value.status == -2
    pages = shape(D, max_pages_per_seq=8192, max_seq_len=131072)
    assert D.delta_workspace_bytes(pages, D.make_select(2048, 128)) > 0


def test_calls_reject_before_launch(D):
    """Every error path returns before anything reaches the (absent) GPU."""
    s = shape(D)
    sel = D.make_select(2048, 128)
    kv = D.delta_kv_t(1, 2, 3, 4)          # fake device pointers: never dereferenced
    lib = D._lib
    P = ctypes.byref
    need = D.delta_workspace_bytes(s, sel)
    fake = ctypes.c_void_p(0x1000)
    assert lib.delta_full_attn(P(s), P(kv), fake, fake, fake, 16, None) == -3
    assert lib.delta_full_attn(P(s), None, fake, fake, fake, need, None) == -1
    assert lib.delta_full_attn(P(s), P(kv), None, fake, fake, need, None) == -1
    assert lib.delta_delta_attn_select(P(s), P(kv), fake, fake, P(sel), None, fake, None, None, fake, need, None) == -1
    assert lib.delta_delta_attn_select(P(s), P(kv), fake, fake, None, fake, fake, None, None, fake, need, None) == -1
    assert lib.delta_sparse_attn(P(s), P(kv), fake, fake, P(sel), fake, fake, None, fake, need - 1, None) == -3
    bad = D.make_shape(2, 32, 8, 80, 512, 8192)
    assert lib.delta_full_attn(P(bad), P(kv), fake, fake, fake, need, None) == -2
    roles = (ctypes.c_int32 * 3)(0, 1, 2)
    kvs = (D.delta_kv_t * 3)(kv, kv, kv)
    ptrs = (ctypes.c_void_p * 3)(0x1000, 0x1000, 0x1000)
    # a Delta/sparse role needs selection parameters and selection buffers
    assert lib.delta_decode_step(P(s), 3, roles, kvs, ptrs, ptrs, None, fake, fake, fake, need, None) == -1
    assert lib.delta_decode_step(P(s), 3, roles, kvs, ptrs, ptrs, P(sel), None, fake, fake, need, None) == -1
    roles_bad = (ctypes.c_int32 * 3)(0, 3, 2)
    assert lib.delta_decode_step(P(s), 3, roles_bad, kvs, ptrs, ptrs, P(sel), fake, fake, fake, need, None) == -1
    nullq = (ctypes.c_void_p * 3)(0x1000, None, 0x1000)
    assert lib.delta_decode_step(P(s), 3, roles, kvs, nullq, ptrs, P(sel), fake, fake, fake, need, None) == -1


def test_noalloc_step_rejects_before_any_device_call(D):
    """The allocation-free step checks its arguments and its scratch size on the host: a shape
    whose workspace exceeds the library's scratch returns DELTA_ERR_WORKSPACE (not a HIP error:
    there is no GPU here), and bad arguments DELTA_ERR_INVALID_ARG."""
    lib = D._lib
    P = ctypes.byref
    fake = ctypes.c_void_p(0x1000)
    kv = D.delta_kv_t(1, 2, 3, 4)
    kvs = (D.delta_kv_t * 3)(kv, kv, kv)
    ptrs = (ctypes.c_void_p * 3)(0x1000, 0x1000, 0x1000)
    roles = (ctypes.c_int32 * 3)(0, 1, 2)
    sel = D.make_select(2048, 128)
    big = D.make_shape(64, 32, 8, 128, 2048, 32768)
    assert D.delta_workspace_bytes(big, sel) > D.DELTA_NOALLOC_SCRATCH_BYTES
    assert lib.delta_decode_step_noalloc(P(big), 3, roles, kvs, ptrs, ptrs, P(sel), fake, fake, None) == -3
    s = shape(D)
    assert D.delta_workspace_bytes(s, sel) <= D.DELTA_NOALLOC_SCRATCH_BYTES
    assert lib.delta_decode_step_noalloc(P(s), 3, roles, kvs, ptrs, ptrs, None, fake, fake, None) == -1
    assert lib.delta_decode_step_noalloc(P(s), 3, roles, kvs, ptrs, ptrs, P(sel), None, fake, None) == -1
    bad_roles = (ctypes.c_int32 * 3)(0, 5, 2)
    assert lib.delta_decode_step_noalloc(P(s), 3, bad_roles, kvs, ptrs, ptrs, P(sel), fake, fake, None) == -1
    assert lib.delta_decode_step_noalloc(P(s), -1, roles, kvs, ptrs, ptrs, P(sel), fake, fake, None) == -1


def test_append_and_hooked_step_reject_before_launch(D):
    """delta_kv_append and delta_decode_step_hooked check every argument on the host; a
    rejected hooked step has run no hook."""
    s = shape(D)
    sel = D.make_select(2048, 128)
    lib = D._lib
    P = ctypes.byref
    fake = ctypes.c_void_p(0x1000)
    assert lib.delta_kv_append(P(s), fake, fake, fake, fake, None, fake, None) == -1
    assert lib.delta_kv_append(P(s), None, fake, fake, fake, fake, fake, None) == -1
    assert lib.delta_kv_append(P(D.make_shape(2, 32, 8, 80, 512, 8192)), fake, fake, fake, fake,
                               fake, fake, None) == -2
    assert lib.delta_kv_append(None, fake, fake, fake, fake, fake, fake, None) == -1
    calls = []
    hooks = D.LayerHooks(before=lambda i: calls.append(("before", i)),
                         after=lambda i: calls.append(("after", i)))
    kv = D.delta_kv_t(1, 2, 3, 4)
    roles = (ctypes.c_int32 * 3)(0, 3, 2)          # invalid role
    kvs = (D.delta_kv_t * 3)(kv, kv, kv)
    ptrs = (ctypes.c_void_p * 3)(0x1000, 0x1000, 0x1000)
    need = D.delta_workspace_bytes(s, sel)
    assert lib.delta_decode_step_hooked(P(s), 3, roles, kvs, ptrs, ptrs, P(sel), fake, fake, fake,
                                        need, None, P(hooks.c)) == -1
    roles_ok = (ctypes.c_int32 * 3)(0, 1, 2)
    assert lib.delta_decode_step_hooked(P(s), 3, roles_ok, kvs, ptrs, ptrs, P(sel), fake, fake, fake,
                                        16, None, P(hooks.c)) == -3
    assert calls == []
    assert D.delta_status_string(-5) == "a layer hook stopped the step"


def test_binding_refuses_host_and_mistyped_buffers(D):
    """The binding checks every tensor it hands to the library before any launch: host
    memory, a wrong element type, a non-contiguous view or a wrong shape never reaches it."""
    import torch
    k = torch.zeros((4, 2, 16, 64), dtype=torch.bfloat16)
    pt = torch.zeros((1, 4), dtype=torch.int32)
    sl = torch.ones((1,), dtype=torch.int32)
    with pytest.raises(ValueError, match="GPU tensor"):
        D.make_kv(k, k, pt, sl)
    with pytest.raises(TypeError):
        D.make_kv(np.zeros((4, 2, 16, 64)), k, pt, sl)
    # the per-call checks, on a descriptor built by hand (no tensors attached: skipped) and on
    # the q / out / selection buffers, which are always checked
    s = D.make_shape(1, 8, 2, 64, 4, 64)
    sel = D.make_select(32, 16)
    kv = D.delta_kv_t(1, 2, 3, 4)
    q = torch.zeros((1, 8, 64), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="GPU tensor"):
        D.delta_full_attn(s, kv, q, q, torch.zeros(16, dtype=torch.uint8))
    with pytest.raises(ValueError):
        D._dev("q", q, torch.float32)
    with pytest.raises(ValueError):
        D._check_sel(s, sel, torch.zeros((1, 3), dtype=torch.int32), torch.zeros((1,), dtype=torch.int32))


def test_delta_path_query(D):
    """The Delta-layer path is a field of the selection parameters: SPLIT is always the split
    path, AUTO and FUSED need a device to measure (none here: split); a bad value and bad
    arguments are refused."""
    shape = D.make_shape(8, 28, 4, 128, 2048, 32768)
    for path in (D.DELTA_PATH_AUTO, D.DELTA_PATH_SPLIT, D.DELTA_PATH_FUSED):
        assert D.delta_delta_path(shape, D.make_select(2048, 128, 16, 0, path)) is False
    sel = D.make_select(2048, 128, 16, 0)
    f = ctypes.c_int(7)
    assert D._lib.delta_delta_path(ctypes.byref(shape), None, ctypes.byref(f)) == D.DELTA_ERR_INVALID_ARG
    assert D._lib.delta_delta_path(ctypes.byref(shape), ctypes.byref(sel), None) == D.DELTA_ERR_INVALID_ARG
    bad = D.make_select(2048, 4096, 16, 0)   # recency window not below the budget
    assert D._lib.delta_delta_path(ctypes.byref(shape), ctypes.byref(bad), ctypes.byref(f)) == D.DELTA_ERR_INVALID_ARG
    bad_path = D.make_select(2048, 128, 16, 0, 3)
    assert D._lib.delta_delta_path(ctypes.byref(shape), ctypes.byref(bad_path), ctypes.byref(f)) == D.DELTA_ERR_INVALID_ARG
    with pytest.raises(D.DeltaError):
        D.delta_workspace_bytes(shape, bad_path)
    assert f.value == 7
