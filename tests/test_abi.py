"""The C ABI without a GPU: libams.so loads, exports every function that
include/ams.h declares, sizes workspaces, and reports host-detectable errors
before touching the device (these calls return before any HIP call)."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_1711_06505_amd import ams

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ams.h")

OK, NULL, SIZE, DTYPE, DIMS, WS, HIP, IDR, MODE, CAPACITY = range(10)
FAKE = ctypes.c_void_p(0x1000)      # never dereferenced: validation fails first


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ams_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ams.LIB_PATH):
        pytest.skip("libams.so not built")
    return ams.load()


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(ams.EXPORTS)


def test_every_declared_symbol_is_exported(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", ams.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT (ams_\w+)", out))
    for name in declared_functions():
        assert name in exported, name
        assert getattr(lib, name) is not None


def test_status_strings(lib):
    for s in range(10):
        assert lib.ams_status_str(s).decode() != "unknown status"
    assert lib.ams_status_str(10).decode() == "unknown status"
    assert b"gfx950" in lib.ams_build_info()


def test_workspace_sizes(lib):
    assert lib.ams_dedup_workspace(-1, 10) == 0
    assert lib.ams_dedup_workspace(57_000, 200_000) >= 4 * 57_000 * 4


def test_dedup_workspace_serves_smaller_calls(lib):
    # one workspace sized for the largest ID table serves the smaller ones
    # (the look-back words grow with the digit width, which is not monotonic
    # in the ID range: 100 IDs sort in one 7-bit pass, 1000 in two of 5)
    ks = list(range(1, 300)) + [2 ** b + o for b in range(9, 31) for o in (-1, 0, 1)] + [2 ** 31 - 1]
    for n in (1, 100, 2047, 2048, 2049, 57_000, 750_000):
        ws = [lib.ams_dedup_workspace(n, k) for k in ks]
        assert all(b >= a for a, b in zip(ws, ws[1:])), n
    for k in (7, 100, 1000, 200_000, 2 ** 31 - 1):
        ws = [lib.ams_dedup_workspace(n, k) for n in range(0, 20_000, 97)]
        assert all(b >= a for a, b in zip(ws, ws[1:])), k
    m = ams.make_mlp((4096, 256, 64, 12), "f32")
    assert lib.ams_embed_workspace(ctypes.byref(m), 57_000) >= 57_000 * 256 * 4
    bad = ams.make_mlp((4000, 256, 64, 12), "f32")
    assert lib.ams_embed_workspace(ctypes.byref(bad), 100) == 0
    # the split float32 forward also holds W1's three bf16 parts
    x3 = ams.make_mlp((4096, 256, 64, 12), "f32x3")
    assert (lib.ams_embed_workspace(ctypes.byref(x3), 57_000)
            >= lib.ams_embed_workspace(ctypes.byref(m), 57_000) + 3 * 4096 * 256 * 2 - 256)
    assert lib.ams_pool_workspace(2, 1024, 56_000, 12, 57_000) > 0
    assert lib.ams_pool_workspace(9, 1024, 56_000, 12, 57_000) == 0


def test_dedup_host_errors(lib):
    args = [FAKE, 100, 10, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30, None]
    a = list(args); a[1] = -1
    assert lib.ams_dedup(*a) == SIZE
    a = list(args); a[2] = 0
    assert lib.ams_dedup(*a) == SIZE
    a = list(args); a[1] = 2 ** 31
    assert lib.ams_dedup(*a) == SIZE
    a = list(args); a[0] = None
    assert lib.ams_dedup(*a) == NULL
    a = list(args); a[7] = None               # n_uniq
    assert lib.ams_dedup(*a) == NULL
    a = list(args); a[10] = 16
    assert lib.ams_dedup(*a) == WS


def test_dedup_noalloc_host_errors(lib):
    # every check here returns before the scratch is looked up or anything enqueued
    args = [FAKE, 100, 10, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None]
    a = list(args); a[1] = -1
    assert lib.ams_dedup_noalloc(*a) == SIZE
    a = list(args); a[2] = 0
    assert lib.ams_dedup_noalloc(*a) == SIZE
    a = list(args); a[1] = ams.DEDUP_NOALLOC_MAX_OCC + 1
    assert lib.ams_dedup_noalloc(*a) == CAPACITY
    a = list(args); a[0] = None
    assert lib.ams_dedup_noalloc(*a) == NULL
    a = list(args); a[8] = None               # dev_status
    assert lib.ams_dedup_noalloc(*a) == NULL
    hdr = open(HEADER).read()
    assert f"#define AMS_DEDUP_NOALLOC_MAX_OCC (1 << {ams.DEDUP_NOALLOC_MAX_OCC.bit_length() - 1})" in hdr


def _embed_args(m, slope=None):
    return [ctypes.byref(m), FAKE, 1000, FAKE, FAKE, 100, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, slope,
            FAKE, FAKE, FAKE, FAKE, 1 << 30, None]


def test_embed_host_errors(lib):
    m = ams.make_mlp((4096, 256, 64, 12), "f32")
    assert lib.ams_embed_fwd(None, *_embed_args(m)[1:]) == NULL
    for dims, code in [((4000, 256, 64, 12), DIMS), ((4096, 300, 64, 12), DIMS),
                       ((4096, 256, 65, 12), DIMS), ((4096, 256, 64, 33), DIMS),
                       ((4096, 512, 64, 12), DIMS)]:
        bad = ams.make_mlp(dims, "f32")
        assert lib.ams_embed_fwd(*_embed_args(bad)) == code, dims
    bad = ams.make_mlp((4096, 256, 64, 12), "f32")
    bad.dtype = 5
    assert lib.ams_embed_fwd(*_embed_args(bad)) == DTYPE
    a = _embed_args(m); a[5] = -1
    assert lib.ams_embed_fwd(*a) == SIZE
    a = _embed_args(m); a[1] = None
    assert lib.ams_embed_fwd(*a) == NULL
    a = _embed_args(m); a[5] = 0              # nothing to do: returns before any launch
    assert lib.ams_embed_fwd(*a) == OK
    # fp32 without H1_save keeps H1 in the workspace, which is then required
    a = _embed_args(m); a[13] = None; a[16] = None; a[17] = 0
    assert lib.ams_embed_fwd(*a) == WS
    # PReLU: float32, or bf16 with the 256-wide first layer of the bf16 tails;
    # every hidden layer needs its slopes
    P = ctypes.c_void_p
    two = (P * 2)(0x1000, 0x1000)
    half = (P * 2)(0x1000, None)
    mb = ams.make_mlp((4096, 128, 64, 12), "bf16")
    assert lib.ams_embed_fwd(*_embed_args(mb, two)) == DTYPE
    mb256 = ams.make_mlp((4096, 256, 64, 12), "bf16")
    a = _embed_args(mb256, two); a[5] = 0
    assert lib.ams_embed_fwd(*a) == OK
    assert lib.ams_embed_fwd(*_embed_args(m, half)) == NULL
    a = _embed_args(m, two); a[5] = 0
    assert lib.ams_embed_fwd(*a) == OK
    bw = [ctypes.byref(m), FAKE, 1000, FAKE, FAKE, 100, FAKE, FAKE, FAKE, None, FAKE, FAKE, None,
          FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, 16, None]
    assert lib.ams_embed_bwd(*bw) == WS
    b2 = list(bw); b2[10] = None              # H1_save
    assert lib.ams_embed_bwd(*b2) == NULL
    fr = ams.make_mlp((4096, 256, 64, 12), "f32", final_relu=True)
    b3 = list(bw); b3[0] = ctypes.byref(fr)   # final_relu needs the forward's E
    assert lib.ams_embed_bwd(*b3) == NULL
    b4 = list(bw); b4[0] = ctypes.byref(mb); b4[9] = two
    assert lib.ams_embed_bwd(*b4) == DTYPE
    b5 = list(bw); b5[9] = half
    assert lib.ams_embed_bwd(*b5) == NULL


def test_pool_host_errors(lib):
    f = [2, 4, 12, FAKE, 40, FAKE, 44, FAKE, FAKE, FAKE, FAKE, None]
    a = list(f); a[0] = 3
    assert lib.ams_pool_fwd(*a) == MODE
    a = list(f); a[2] = 0
    assert lib.ams_pool_fwd(*a) == SIZE
    a = list(f); a[2] = 33
    assert lib.ams_pool_fwd(*a) == SIZE
    a = list(f); a[1] = -1
    assert lib.ams_pool_fwd(*a) == SIZE
    a = list(f); a[6] = -1                    # capacity (rows of E)
    assert lib.ams_pool_fwd(*a) == SIZE
    a = list(f); a[10] = None                 # attention needs its weights buffer
    assert lib.ams_pool_fwd(*a) == NULL
    a = list(f); a[1] = 0                     # empty batch: nothing to do
    assert lib.ams_pool_fwd(*a) == OK
    b = [2, 4, 12, FAKE, 40, FAKE, FAKE, FAKE, FAKE, 44, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE,
         FAKE, 16, None]
    assert lib.ams_pool_bwd(*b) == WS
    a = list(b); a[6] = None                  # occ_perm
    assert lib.ams_pool_bwd(*a) == NULL
    a = list(b); a[9] = -3
    assert lib.ams_pool_bwd(*a) == SIZE


def test_timing_switch_and_empty_read(lib):
    # no launch is recorded without a GPU: the read returns an empty record
    assert lib.ams_timing_enable(1) == OK
    assert ams.ams_timing_read() == {}
    assert lib.ams_timing_enable(0) == OK
    n = ctypes.c_int(-1)
    assert lib.ams_timing_read(None, 0, ctypes.byref(n)) == OK and n.value == 0
    assert lib.ams_timing_read(None, 0, None) == NULL
    assert lib.ams_timing_read(None, 4, ctypes.byref(n)) == NULL


def test_joint_host_errors(lib):
    # bag forward
    assert lib.ams_bag_fwd(-1, 12, FAKE, 40, FAKE, FAKE, 100, FAKE, None) == SIZE
    assert lib.ams_bag_fwd(4, 0, FAKE, 40, FAKE, FAKE, 100, FAKE, None) == DIMS
    assert lib.ams_bag_fwd(4, 33, FAKE, 40, FAKE, FAKE, 100, FAKE, None) == DIMS
    assert lib.ams_bag_fwd(4, 12, FAKE, 40, None, FAKE, 100, FAKE, None) == NULL
    assert lib.ams_bag_fwd(0, 12, None, 0, None, None, 100, None, None) == OK
    # bag backward = the SUM aggregator's backward: its checks apply
    assert lib.ams_bag_workspace(4, 40, 12, 44) == lib.ams_pool_workspace(0, 4, 40, 12, 44) > 0
    bb = [4, 12, FAKE, 40, FAKE, FAKE, FAKE, FAKE, 44, FAKE, None, FAKE, FAKE, 16, None]
    assert lib.ams_bag_bwd(*bb) == WS
    a = list(bb); a[10] = FAKE                # with the ads' second gradient
    assert lib.ams_bag_bwd(*a) == WS
    a = list(bb); a[9] = None                 # dbag
    assert lib.ams_bag_bwd(*a) == NULL
    a = list(bb); a[5] = None                 # occ_perm
    assert lib.ams_bag_bwd(*a) == NULL
    a = list(bb); a[11] = None                # grad
    assert lib.ams_bag_bwd(*a) == NULL
    # CTR
    net = ams.make_ctr((60, 200, 80, 2))
    assert lib.ams_ctr_workspace(ctypes.byref(net), 4096) >= 256 * (60 * 200 + 200 * 80 + 80 * 2) * 4
    for dims in [(129, 200, 80, 2), (60, 257, 80, 2), (60, 200, 80, 1), (60, 200, 80, 9)]:
        assert lib.ams_ctr_workspace(ctypes.byref(ams.make_ctr(dims)), 10) == 0, dims
    P = ctypes.c_void_p
    fields = (P * 5)(*[0x1000] * 5)
    widths = (ctypes.c_int32 * 5)(12, 12, 12, 12, 12)
    ptr3 = (P * 3)(*[0x1000] * 3)
    args = [ctypes.byref(net), 4096, 5, fields, widths, FAKE, ptr3, ptr3, None, FAKE, None, ptr3, ptr3, None, None,
            FAKE, 1 << 30, None]
    a = list(args); a[16] = 16
    assert lib.ams_ctr_fwd_bwd(*a) == WS
    a = list(args); a[1] = 0
    assert lib.ams_ctr_fwd_bwd(*a) == SIZE
    bad_w = (ctypes.c_int32 * 5)(12, 12, 12, 12, 11)      # widths must sum to dims[0]
    a = list(args); a[4] = bad_w
    assert lib.ams_ctr_fwd_bwd(*a) == DIMS
    a = list(args); a[2] = 9
    assert lib.ams_ctr_fwd_bwd(*a) == DIMS
    a = list(args); a[5] = None               # labels
    assert lib.ams_ctr_fwd_bwd(*a) == NULL
    a = list(args); a[9] = None               # loss
    assert lib.ams_ctr_fwd_bwd(*a) == NULL
    a = list(args); a[12] = None              # db
    assert lib.ams_ctr_fwd_bwd(*a) == NULL
    # Adagrad
    assert lib.ams_adagrad_rows(12, FAKE, FAKE, -1, FAKE, FAKE, 100, FAKE, 0.01, 1e-8, None) == SIZE
    assert lib.ams_adagrad_rows(12, FAKE, FAKE, 0, None, None, 100, None, 0.01, 1e-8, None) == OK
    assert lib.ams_adagrad_rows(12, FAKE, FAKE, 10, FAKE, None, 100, FAKE, 0.01, 1e-8, None) == NULL


def test_query_pool_host_errors(lib):
    f = [4, 12, FAKE, 40, FAKE, 44, FAKE, None, FAKE, FAKE, None]
    assert lib.ams_pool_query_fwd(*f) == NULL                # Q
    a = list(f); a[1] = 33
    assert lib.ams_pool_query_fwd(*a) == SIZE
    a = list(f); a[5] = -1
    assert lib.ams_pool_query_fwd(*a) == SIZE
    a = list(f); a[0] = 0
    assert lib.ams_pool_query_fwd(*a) == OK
    b = [4, 12, FAKE, 40, FAKE, FAKE, FAKE, FAKE, 44, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0, FAKE, 16, None]
    assert lib.ams_pool_query_bwd(*b) == WS
    a = list(b); a[14] = None                                 # dQ
    assert lib.ams_pool_query_bwd(*a) == NULL
    a = list(b); a[8] = -1
    assert lib.ams_pool_query_bwd(*a) == SIZE


def test_adam_host_errors(lib):
    assert lib.ams_adam_update(-1, FAKE, FAKE, FAKE, FAKE, 1e-3, 0.9, 0.999, 1e-8, 1, None, None) == SIZE
    assert lib.ams_adam_update(10, FAKE, FAKE, FAKE, FAKE, 1e-3, 0.9, 0.999, 1e-8, 0, None, None) == SIZE
    assert lib.ams_adam_update(10, FAKE, None, FAKE, FAKE, 1e-3, 0.9, 0.999, 1e-8, 1, None, None) == NULL
    assert lib.ams_adam_update(0, None, None, None, None, 1e-3, 0.9, 0.999, 1e-8, 1, None, None) == OK


def test_concat_pool_host_errors(lib):
    f = [4, 12, 5, FAKE, 40, FAKE, 44, FAKE, FAKE, None, None]
    assert lib.ams_pool_concat_fwd(*f) == NULL                # A
    a = list(f); a[6] = -1
    assert lib.ams_pool_concat_fwd(*a) == SIZE
    a = list(f); a[2] = 0
    assert lib.ams_pool_concat_fwd(*a) == SIZE                # Lc
    a = list(f); a[1] = 33
    assert lib.ams_pool_concat_fwd(*a) == SIZE
    a = list(f); a[0] = 0
    assert lib.ams_pool_concat_fwd(*a) == OK
    b = [4, 12, 5, FAKE, 40, FAKE, FAKE, FAKE, FAKE, 44, FAKE, None, FAKE, FAKE, 16, None]
    assert lib.ams_pool_concat_bwd(*b) == WS
    a = list(b); a[10] = None                                 # dU
    assert lib.ams_pool_concat_bwd(*a) == NULL
    a = list(b); a[2] = -3
    assert lib.ams_pool_concat_bwd(*a) == SIZE


def test_dssm_host_errors(lib):
    P = ctypes.c_void_p
    user, ad = ams.make_ctr((36, 64, 32)), ams.make_ctr((24, 32))
    assert lib.ams_dssm_workspace(ctypes.byref(user), ctypes.byref(ad), 4096) >= 256 * (36 * 64 + 64 * 32) * 4
    assert lib.ams_dssm_workspace(ctypes.byref(user), ctypes.byref(ams.make_ctr((24, 65))), 10) == 0
    uf, uw = (P * 3)(*[0x1000] * 3), (ctypes.c_int32 * 3)(12, 12, 12)
    af, aw = (P * 2)(*[0x1000] * 2), (ctypes.c_int32 * 2)(12, 12)
    p2 = (P * 2)(*[0x1000] * 2)
    p1 = (P * 1)(0x1000)
    args = [ctypes.byref(user), ctypes.byref(ad), 4096, 3, uf, uw, 2, af, aw, FAKE, p2, p2, None, p1, p1, None,
            FAKE, None, p2, p2, None, p1, p1, None, None, None, FAKE, 1 << 30, None]
    a = list(args); a[27] = 16
    assert lib.ams_dssm_fwd_bwd(*a) == WS
    a = list(args); a[1] = ctypes.byref(ams.make_ctr((24, 31)))   # towers of unequal width
    assert lib.ams_dssm_fwd_bwd(*a) == DIMS
    a = list(args); a[2] = 0
    assert lib.ams_dssm_fwd_bwd(*a) == SIZE
    a = list(args); a[8] = (ctypes.c_int32 * 2)(12, 11)
    assert lib.ams_dssm_fwd_bwd(*a) == DIMS
    a = list(args); a[9] = None                                     # labels
    assert lib.ams_dssm_fwd_bwd(*a) == NULL
    a = list(args); a[21] = None                                    # dWa
    assert lib.ams_dssm_fwd_bwd(*a) == NULL


def test_step_rejects_an_unchecked_capacity_below_the_occurrences():
    # the check runs before any buffer is allocated
    with pytest.raises(ValueError, match="cap_checked"):
        ams.Step((256, 64, 16), "f32", "sum", 4, 10, device="cpu", cap=13)
