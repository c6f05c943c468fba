"""The C ABI library loads, exports every symbol include/hardkv.h declares, and rejects
invalid arguments on the host (no GPU needed: validation happens before any launch)."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hardkv.h")


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:hk_status|size_t|const char\*)\s+(hk_\w+)\s*\(", text,
                                 flags=re.M)))


@pytest.fixture(scope="module")
def hk():
    import paper_2606_28831_amd as hk
    if not os.path.exists(hk.LIB_PATH):
        from paper_2606_28831_amd.build import build
        build()
    return hk


def test_header_declares_the_boundary():
    names = _declared()
    for n in ["hk_score", "hk_calibrate", "hk_calibrate_solve_T", "hk_topp_select", "hk_compact",
              "hk_decode_attn", "hk_append_kv", "hk_workspace_size", "hk_status_string"]:
        assert n in names


def test_library_exports_every_declared_symbol(hk):
    L = C.CDLL(hk.LIB_PATH)
    for n in _declared():
        assert hasattr(L, n), n
    assert sorted(_declared()) == sorted(hk.EXPORTED)


def test_status_strings(hk):
    for code in range(8):
        assert hk.hk_status_string(code).startswith("HK_")
    for f in (1, 2, 4):
        assert hk.hk_status_string(f, True).startswith("HK_FLAG")


def test_workspace_sizes(hk):
    d = hk.dims(32, 28, 4, 128, 32)
    # row-LSE partials: at least one (max, sum) pair per window row and head, plus the LSEs
    assert hk.hk_workspace_size(hk.OP_SCORE, d, 2048) >= 128 * 224 * 8 + 32 * 32 * 28 * 4
    assert hk.hk_workspace_size(hk.OP_SCORE, d, 4096) > hk.hk_workspace_size(hk.OP_SCORE, d, 2048)
    assert hk.hk_workspace_size(hk.OP_COMPACT, d, 2048) >= 2 * 128 * 2048 * 4
    assert hk.hk_workspace_size(hk.OP_DECODE, d, 2048) > 0
    # the whole step: the scores (4 bytes per slot) and the larger stage scratch at least
    cw = hk.hk_workspace_size(hk.OP_COMPRESS, d, 2048)
    assert cw >= 128 * 2048 * 16 * 4 + max(hk.hk_workspace_size(hk.OP_SCORE, d, 2048),
                                           hk.hk_workspace_size(hk.OP_COMPACT, d, 2048))
    # the wide selector: a key per slot, and the same figure through the dims form
    sw = hk.hk_select_workspace_size(128, 32768)
    assert sw >= 128 * 32768 * 4 and hk.hk_workspace_size(hk.OP_SELECT, d, 2048) == sw
    assert cw >= 128 * 2048 * 16 * 4 + sw
    assert hk.hk_workspace_size(99, d, 2048) == 0


def _kv(hk, dtype=1, max_pages=4, D=128, addr=1 << 20):
    return hk.hk_paged_kv(addr, addr, addr, addr, addr, 64, max_pages, dtype)


def test_validation_errors_without_gpu(hk):
    L = hk.lib()
    d = hk.dims(1, 8, 2, 128, 16)
    kv = _kv(hk)
    P = 1 << 20
    ws = 1 << 24
    score = lambda d_, kv_, **kw: L.hk_score(C.byref(d_), kw.get("q", P), C.byref(kv_), 0,
                                             kw.get("scale", 0.125), None, None, P, P, None, 0,
                                             None, kw.get("ws", ws), 1 << 30, None)
    assert score(hk.dims(1, 8, 2, 96, 16), kv) == 3          # D not 64/128 -> SHAPE
    assert score(hk.dims(1, 9, 2, 128, 16), kv) == 3         # Hq % Hkv -> SHAPE
    assert score(hk.dims(1, 8, 2, 128, 128), kv) == 3        # G*W > 256 -> SHAPE
    assert score(d, _kv(hk, dtype=7)) == 2                   # dtype
    assert score(d, _kv(hk, max_pages=3)) == 3               # odd table width
    assert score(d, kv, scale=-1.0) == 1                     # scale
    assert score(d, kv, q=P + 4) == 4                        # alignment
    assert score(d, kv, ws=P + 16) == 4                      # workspace alignment
    assert L.hk_topp_select(4, 100, P, None, P, 0.9, 1, 0, P, P, None, None, None) == 3
    assert L.hk_topp_select(4, 65536, P, None, P, 0.9, 1, 0, P, P, None, None, None) == 3
    assert L.hk_topp_select(4, 128, P, None, P, 1.5, 1, 0, P, P, None, None, None) == 1
    assert L.hk_topp_select(4, 128, None, None, P, 0.9, 1, 0, P, P, None, None, None) == 1
    assert L.hk_calibrate_solve_T(4, 128, P, None, P, P, P, 1.0, 0.5, 40, P, None) == 1
    assert L.hk_calibrate_solve_T(4, 128, P, None, P, P, P, 1e-4, 1e4, 0, P, None) == 1
    assert L.hk_calibrate_solve_T(4, 262144 + 32, P, None, P, P, P, 1e-4, 1e4, 40, P, None) == 3
    alloc = hk.hk_allocator(P, P, 64)
    assert L.hk_compact(C.byref(d), C.byref(kv), P, -1, 0, C.byref(alloc), P, P, 1 << 30, None) == 1
    # a free stack shorter than the pool (64 pages) could overflow when the rewrite pushes
    short = hk.hk_allocator(P, P, 63)
    assert L.hk_compact(C.byref(d), C.byref(kv), P, 0, 0, C.byref(short), P, P, 1 << 30, None) == 1
    assert L.hk_compact_modes(C.byref(d), C.byref(kv), P, 0, P, C.byref(short), P, P, 1 << 30,
                              None) == 1
    assert L.hk_compress(C.byref(d), P, C.byref(kv), 0, 0, 0.125, None, 0.9, 1, 0, C.byref(short),
                         None, P, None, P, 1 << 30, None) == 1
    assert L.hk_compact(C.byref(d), C.byref(kv), P, 0, 0, C.byref(alloc), P, P, 16, None) == 5
    assert L.hk_decode_attn(C.byref(hk.dims(1, 12, 2, 128)), P, C.byref(kv), 0.1, P, P, P,
                            1 << 30, None) == 3              # group of 6 unsupported
    assert L.hk_decode_attn(C.byref(d), P, C.byref(kv), 0.1, P, P, P, 16, None) == 5
    # the allocation-free decode: a call whose split states exceed the 16 MiB static scratch
    # (all 32 layers of config 5 at once) is refused before anything is launched
    d5 = hk.dims(2048, 32, 8, 128)
    assert L.hk_decode_noalloc_scratch_bytes(C.byref(d5), 768) > 16 << 20
    assert L.hk_decode_attn_noalloc(C.byref(d5), P, C.byref(_kv(hk, max_pages=768)), 0.1, P, P,
                                    None) == 7
    assert L.hk_decode_noalloc_scratch_bytes(C.byref(hk.dims(64, 32, 8, 128)), 768) == 64 * 8 * 6 * 4 * 130 * 4
    assert L.hk_decode_attn_noalloc(C.byref(d), None, C.byref(kv), 0.1, P, P, None) == 1
    assert L.hk_append_kv(C.byref(d), C.byref(kv), None, P, C.byref(alloc), P, None, 0, None) == 1
    kvnull = hk.hk_paged_kv(None, P, P, P, P, 64, 4, 1)
    assert L.hk_decode_attn(C.byref(d), P, C.byref(kvnull), 0.1, P, P, P, 1 << 30, None) == 1
    assert L.hk_pool_max(4, 128, P, None, P, 65, P + 64, None) == 3     # radius > 64
    assert L.hk_pool_max(4, 128, P, None, P, -1, P + 64, None) == 3     # negative radius
    assert L.hk_pool_max(4, 128, P, None, P, 3, P, None) == 1           # in place
    assert L.hk_pool_max(4, 100, P, None, P, 3, P + 64, None) == 3      # S_max % 32
    assert L.hk_pool_max(4, 262144 + 32, P, None, P, 3, P + 64, None) == 3  # longer than 262144
    xs = (C.c_void_p * 1)(P)
    wts = (C.c_float * 1)(1.0)
    assert L.hk_calibrate_topp(4, 128, P, None, 3, xs, None, wts, 0.9, 1, 0, None, None, P, P,
                               None, None, None) == 1                   # three metrics
    assert L.hk_calibrate_topp(4, 128, P, None, 1, xs, None, wts, 1.5, 1, 0, None, None, P, P,
                               None, None, None) == 1                   # p outside [0, 1]
    assert L.hk_calibrate_topp(4, 128, P, None, 1, xs, None, wts, 0.9, 1, 0, None, None, P + 4, P,
                               None, None, None) == 4                   # bitmap alignment
    # the multi-workgroup selector: up to 262144 slots, and a workspace of the stated size
    need = L.hk_select_workspace_size(4, 131072)
    assert need >= 4 * 131072 * 4
    assert L.hk_select_workspace_size(4, 262144) > need
    assert L.hk_topp_select_ws(4, 262144 + 32, P, None, P, 0.9, 1, 0, P, P, None, None, P,
                               1 << 40, None) == 3              # beyond 262144 slots
    assert L.hk_topp_select_ws(4, 131072, P, None, P, 0.9, 1, 0, P, P, None, None, P, need - 1,
                               None) == 5                       # workspace too small
    assert L.hk_topp_select_ws(4, 131072, P, None, P, 0.9, 1, 0, P, P, None, None, P + 16, need,
                               None) == 4                       # workspace alignment
    assert L.hk_topp_select_ws(4, 131072, P, None, None, 0.9, 1, 0, P, P, None, None, P, need,
                               None) == 1                       # no c
    assert L.hk_calibrate_topp_ws(4, 131072, P, None, 3, xs, None, wts, 0.9, 1, 0, None, None, P,
                                  P, None, None, P, need, None) == 1   # three metrics
    assert L.hk_calibrate_topp_ws(4, 131072, P, None, 1, xs, None, wts, 0.9, 1, 0, None, None,
                                  P + 4, P, None, None, P, need, None) == 4   # bitmap alignment
    assert L.hk_calibrate_topp_ws(4, 100, P, None, 1, xs, None, wts, 0.9, 1, 0, None, None, P, P,
                                  None, None, P, need, None) == 3      # S_max % 32
    assert L.hk_calibrate_solve_T_gd(4, 128, P, None, P, P, P, 0.0, 0.05, 10, 0.0, P, None,
                                     None) == 1                 # T_init
    assert L.hk_calibrate_solve_T_gd(4, 128, P, None, P, P, P, 1.0, -0.1, 10, 0.0, P, None,
                                     None) == 1                 # lr
    assert L.hk_calibrate_solve_T_gd(4, 128, P, None, P, P, P, 1.0, 0.05, -1, 0.0, P, None,
                                     None) == 1                 # iters
    assert L.hk_calibrate_solve_T_gd(4, 262144 + 32, P, None, P, P, P, 1.0, 0.05, 10, 0.0, P, None,
                                     None) == 3                 # rows too long
    assert L.hk_compress(C.byref(d), P, C.byref(kv), 0, 0, 0.125, None, 0.9, 1, 0, C.byref(alloc),
                         None, P, None, P, 16, None) == 5       # workspace too small
    assert L.hk_compress(C.byref(d), P, C.byref(kv), 0, 0, 0.125, None, 1.5, 1, 0, C.byref(alloc),
                         None, P, None, P, 1 << 30, None) == 1  # p outside [0, 1]
    kv_long = _kv(hk, max_pages=262144 // 16 + 2)
    assert L.hk_compress(C.byref(d), P, C.byref(kv_long), 0, 0, 0.125, None, 0.9, 1, 0,
                         C.byref(alloc), None, P, None, P, 1 << 40, None) == 3   # rows too long
    a64 = hk.hk_allocator(P, P, 64)
    assert L.hk_alloc_init(C.byref(a64), -1, 10, None) == 1
    assert L.hk_alloc_init(C.byref(a64), 10, 5, None) == 1           # num_pages < first_free
    assert L.hk_alloc_init(C.byref(a64), 0, 65, None) == 1           # beyond the capacity
    assert L.hk_alloc_init(C.byref(hk.hk_allocator(P + 4, P, 64)), 0, 8, None) == 4
    # Step 4: hard budget
    assert L.hk_score_rows(C.byref(d), P, C.byref(kv), 0, 0.125, None, P, None) == 1   # no LSE
    assert L.hk_score_rows(C.byref(hk.dims(1, 8, 2, 128, 128)), P, C.byref(kv), 0, 0.125, P, P,
                           None) == 3                                   # G*W > 256
    assert L.hk_score_rows(C.byref(d), P + 4, C.byref(kv), 0, 0.125, P, P, None) == 4
    assert L.hk_vote_topp(4, 0, 128, P, None, P, 0.9, P, P, None, None, None) == 3    # R = 0
    assert L.hk_vote_topp(4, 257, 128, P, None, P, 0.9, P, P, None, None, None) == 3  # R > 256
    assert L.hk_vote_topp(4, 8, 100, P, None, P, 0.9, P, P, None, None, None) == 3    # S_max % 32
    assert L.hk_vote_topp(4, 8, 128, P, None, P, -0.1, P, P, None, None, None) == 1   # p
    assert L.hk_vote_topp(4, 8, 128, P, None, P, 0.9, P + 2, P, None, None, None) == 4
    assert L.hk_vote_topp(4, 8, 128, P, None, P, 0.9, P, None, None, None, None) == 1  # row_sel
    assert L.hk_budget_plan(C.byref(d), C.byref(kv), 0, 10, 5, P, P, None) == 1   # L_upper < L_lower
    assert L.hk_budget_plan(C.byref(d), C.byref(kv), 0, 5, 10, None, P, None) == 1
    assert L.hk_budget_select(4, 128, P, None, None, None, None, None, None, -1, P, P, None) == 1
    assert L.hk_budget_select(4, 128, P, None, None, None, None, None, None, 0, P + 4, P, None) == 4
    assert L.hk_budget_select(4, 65536 + 32, P, None, None, None, None, None, None, 0, P, P,
                              None) == 3                                # past 65536 slots
    assert L.hk_vote_topp(4, 8, 65536 + 32, P, None, P, 0.9, P, P, None, None, None) == 3
    assert L.hk_compact_modes(C.byref(d), C.byref(kv), P, 0, None, C.byref(alloc), P, P, 1 << 30,
                              None) == 1                                # no head modes
    assert L.hk_compact_modes(C.byref(d), C.byref(kv), P, 0, P, C.byref(alloc), P, P, 16,
                              None) == 5                                # workspace too small
    # rate probes
    assert L.hk_probe(hk.PROBE_EXP, 0, 8, P, None) == 1                 # no workgroups
    assert L.hk_probe(hk.PROBE_MFMA, 4, 0, P, None) == 1                # no iterations
    assert L.hk_probe(hk.PROBE_EXP, 4, 8, None, None) == 1              # no output
    assert L.hk_probe(6, 4, 8, P, None) == 1                            # unknown kind
    assert L.hk_probe(-1, 4, 8, P, None) == 1


def test_kernel_timing_host_side(hk):
    """Timing off by default: nothing recorded, reads are empty; bad ids are rejected."""
    L = C.CDLL(hk.LIB_PATH)
    ms, n = C.c_double(1.0), C.c_int64(7)
    for k in range(len(hk.TIMED_KERNELS)):
        assert L.hk_timing_read(k, C.byref(ms), C.byref(n)) == 0
        assert ms.value == 0.0 and n.value == 0
    assert L.hk_timing_read(len(hk.TIMED_KERNELS), C.byref(ms), C.byref(n)) == 1
    assert L.hk_timing_read(-1, C.byref(ms), C.byref(n)) == 1
    assert L.hk_timing_read(0, None, C.byref(n)) == 1
    assert L.hk_timing_enable(C.c_uint32(0xFFFFFFFF)) == 0 and L.hk_timing_enable(C.c_uint32(0)) == 0
    text = open(HEADER).read()
    assert int(re.search(r"HK_TK_COUNT = (\d+)", text).group(1)) == len(hk.TIMED_KERNELS)


def test_decode_split_plan_invariants():
    """The decode split plan (host logic): pages per split a power of two in [16, 128], the
    splits cover the table width, a launch offers at least 2048 workgroups unless its
    splits are already the shortest, and the split states fit the workspace the library
    asks for (sized for 16-page splits)."""
    import paper_2606_28831_amd as hk
    for NS, Hkv in ((1, 1), (1, 2), (2, 4), (64, 8), (2048, 8)):
        for max_pages in (1, 15, 16, 17, 768, 8192, 16384):
            d = hk.dims(NS, 4 * Hkv, Hkv, 128)
            n_split, pps = hk.hk_decode_plan(d, max_pages)
            heads = NS * Hkv
            assert pps in (16, 32, 64, 128), (NS, Hkv, max_pages, pps)
            assert n_split == -(-max_pages // pps)
            assert heads * n_split >= 2048 or pps == 16
            # the most pages one split can be given never exceeds pps (the kernel stages a
            # split's page ids in an LDS array of 128)
            share = min(pps, max(-(-max_pages // n_split), 16))
            assert share <= pps and share * n_split >= max_pages
            ws = hk.hk_workspace_size(hk.OP_DECODE, d, max_pages)
            assert ws >= heads * n_split * 4 * 130 * 4
