"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every entry point the header declares, and rejects bad arguments before
launching anything."""
import ctypes
import os
import re

import pytest

from paper_2609_37842_amd import eogp as E

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    hdr = open(os.path.join(ROOT, "include", "eogp.h")).read()
    hdr = re.sub(r"/\*.*?\*/", "", hdr, flags=re.S)
    return sorted(set(re.findall(r"\b(eogp_[a-z_]+)\s*\(", hdr)))


def test_library_exports_every_declared_symbol():
    L = E.load()
    names = header_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(E.EXPORTED)


def test_status_strings_and_version():
    L = E.load()
    assert L.eogp_status_string(0) == b"ok"
    assert L.eogp_status_string(-1) == b"invalid argument"
    assert L.eogp_status_string(-4) == b"workspace too small"
    assert E.eogp_version() >= 100


def test_plan_argument_validation_without_device():
    L = E.load()
    h = ctypes.c_void_p()
    fake = ctypes.c_void_p(0x1000)
    # NULL eigvals
    assert L.eogp_plan_create(None, 4, 4, 0.1, 3, fake, fake, None, ctypes.byref(h)) == -1
    assert b"NULL" in L.eogp_last_error()
    # m out of range, damping <= 0, bad sizes
    assert L.eogp_plan_create(fake, 4, 4, 0.1, 17, fake, fake, None, ctypes.byref(h)) == -1
    assert L.eogp_plan_create(fake, 4, 4, 0.1, 0, fake, fake, None, ctypes.byref(h)) == -1
    assert L.eogp_plan_create(fake, 4, 4, 0.0, 3, fake, fake, None, ctypes.byref(h)) == -1
    assert L.eogp_plan_create(fake, 4, 4, float("nan"), 3, fake, fake, None, ctypes.byref(h)) == -1
    assert L.eogp_plan_create(fake, 0, 4, 0.1, 3, fake, fake, None, ctypes.byref(h)) == -1
    assert L.eogp_plan_create(fake, 1 << 16, 1 << 16, 0.1, 3, fake, fake, None, ctypes.byref(h)) == -1
    assert L.eogp_plan_set_input_exponents(None, 0, 0) == -1


def test_token_compaction_argument_validation_without_device():
    """eogp_compact_tokens / eogp_rotate_retain_compacted reject bad arguments
    before touching the device; the list's size query matches the head of
    every first-stage workspace."""
    L = E.load()
    fake = ctypes.c_void_p(0x1000)
    align = lambda b: -(-b // 256) * 256
    N, T = 5, 7
    assert L.eogp_compact_tokens_workspace_size(N, T) == align(4 * (N + 1)) + align(4 * N) + align(4 * (N * T + 8 * N))
    assert L.eogp_compact_tokens_workspace_size(-1, T) == 0
    assert L.eogp_compact_tokens_workspace_size(1 << 20, 1 << 12) == 0     # N*T + 8N + 256 >= 2^31
    assert L.eogp_compact_tokens(fake, -1, T, E.PREC_F16, fake, 1 << 20, None) == -1
    assert L.eogp_compact_tokens(fake, 1 << 20, 1 << 12, E.PREC_F16, fake, 1 << 40, None) == -1
    assert L.eogp_compact_tokens(fake, N, T, 9, fake, 1 << 20, None) == -1            # precision
    assert L.eogp_compact_tokens(fake, N, T, E.PREC_F16, fake, 16, None) == -4        # workspace
    assert L.eogp_compact_tokens(fake, N, T, E.PREC_F16, None, 1 << 20, None) == -4
    assert L.eogp_compact_tokens(fake, 0, T, E.PREC_F16, None, 0, None) == 0          # nothing to do
    # the compacted first stage: NULL plan, Z dtype
    assert L.eogp_rotate_retain_compacted(None, fake, 0, fake, 0, 0, N, T, fake, 0, 8, 1, fake,
                                          1 << 20, None) == -1
    with pytest.raises(ValueError):
        E.eogp_rotate_retain_compacted(None, None, None, None)


def test_encode_and_score_argument_validation_without_device():
    L = E.load()
    fake = ctypes.c_void_p(0x1000)
    # sign_pack: k < 1, ldx < k, stride too small
    assert L.eogp_sign_pack(fake, 8, 2, 0, fake, 1, fake, 1, None) == -1
    assert L.eogp_sign_pack(fake, 8, 2, 16, fake, 2, fake, 1, None) == -1
    assert L.eogp_sign_pack(fake, 16, 2, 16, fake, 1, fake, 1, None) == -1
    # pca: k > m, ld too small
    assert L.eogp_pca_project(fake, 0, 8, 2, 8, fake, 2, 8, 9, fake, 9, 0, None, 0, None) == -1
    assert L.eogp_pca_project(fake, 0, 4, 2, 8, fake, 2, 8, 4, fake, 4, 0, None, 0, None) == -1
    # 16-bit Z must have P's type and 16-byte rows; unknown Z dtype
    assert L.eogp_pca_project(fake, 1, 8, 2, 8, fake, 2, 8, 4, fake, 4, 0, None, 0, None) == -2
    assert L.eogp_pca_project(fake, 2, 12, 2, 8, fake, 2, 8, 4, fake, 4, 0, None, 0, None) == -2
    assert L.eogp_pca_project(fake, 7, 8, 2, 8, fake, 2, 8, 4, fake, 4, 0, None, 0, None) == -1
    # ekfac: bad sizes, NULL bases, bad precision, exponent out of range, small workspace
    assert L.eogp_ekfac_eigenvalues(fake, 0, fake, 0, 0, None, 2, 3, 0, 4, fake, fake, 1, 0, 0,
                                    fake, 0, fake, 1 << 30, None) == -1
    assert L.eogp_ekfac_eigenvalues(fake, 0, fake, 0, 0, None, 2, 3, 4, 4, None, fake, 1, 0, 0,
                                    fake, 0, fake, 1 << 30, None) == -1
    assert L.eogp_ekfac_eigenvalues(fake, 0, fake, 0, 0, None, 2, 3, 4, 4, fake, fake, 7, 0, 0,
                                    fake, 0, fake, 1 << 30, None) == -1
    assert L.eogp_ekfac_eigenvalues(fake, 0, fake, 0, 0, None, 2, 3, 4, 4, fake, fake, 2, 61, 0,
                                    fake, 0, fake, 1 << 30, None) == -1
    assert L.eogp_ekfac_eigenvalues(fake, 0, fake, 0, 0, None, 2, 3, 4, 4, fake, fake, 1, 0, 0,
                                    fake, 0, fake, 16, None) == -4
    # the compacted token list is indexed in 32 bits
    assert L.eogp_ekfac_eigenvalues(fake, 0, fake, 0, 0, None, 1 << 20, (1 << 11) - 8, 4, 4, fake,
                                    fake, 1, 0, 0, fake, 0, fake, 1 << 30, None) == -1
    # srht: k > p, m too large, ld too small, two-stage form without workspace
    assert L.eogp_srht_project(fake, 100, 2, 100, fake, fake, 129, fake, 129, None, 0, None) == -1
    assert L.eogp_srht_project(fake, (1 << 20) + 1, 2, (1 << 20) + 1, fake, fake, 8, fake, 8,
                               None, 0, None) == -2
    assert L.eogp_srht_project(fake, 50, 2, 100, fake, fake, 8, fake, 8, None, 0, None) == -1
    assert L.eogp_srht_project(fake, 40000, 2, 40000, fake, fake, 8, fake, 8, None, 0, None) == -4
    assert L.eogp_srht_project_workspace_size(2, 32768) == 0
    assert L.eogp_srht_project_workspace_size(2, 40000) == 2 * 65536 * 4
    # pca fit: k > min(n, m), ld too small, NULL workspace; the size query
    # rejects bad sizes
    assert L.eogp_pca_fit(fake, 8, 4, 8, 5, fake, 8, fake, fake, 1 << 20, None) == -1
    assert L.eogp_pca_fit(fake, 8, 10, 8, 9, fake, 8, fake, fake, 1 << 20, None) == -1
    assert L.eogp_pca_fit(fake, 6, 10, 8, 4, fake, 8, fake, fake, 1 << 20, None) == -1
    assert L.eogp_pca_fit(fake, 8, 10, 8, 4, fake, 7, fake, fake, 1 << 20, None) == -1
    assert L.eogp_pca_fit(fake, 8, 10, 8, 4, fake, 8, fake, None, 1 << 20, None) == -1
    assert L.eogp_pca_fit_workspace_size(10, 8, 9) == 0
    assert L.eogp_pca_fit_workspace_size(10, 8, 0) == 0
    # score: k_u not a multiple of 64, topk out of range, misaligned stride
    ks = (ctypes.c_int64 * 2)(64, 100)
    assert L.eogp_score_topk(fake, 32, fake, 4, 2, ks, fake, 164, 1, 3, fake, fake, None,
                             fake, 1 << 20, None) == -1
    ks = (ctypes.c_int64 * 1)(64)
    assert L.eogp_score_topk(fake, 8, fake, 4, 1, ks, fake, 64, 1, 0, fake, fake, None,
                             fake, 1 << 20, None) == -1
    assert L.eogp_score_topk(fake, 8, fake, 4, 1, ks, fake, 64, 1, 257, fake, fake, None,
                             fake, 1 << 20, None) == -1
    assert L.eogp_score_topk(fake, 12, fake, 4, 1, ks, fake, 64, 1, 5, fake, fake, None,
                             fake, 1 << 20, None) == -1
    # a module longer than 2^22 bits (its integer sums could overflow)
    big = (ctypes.c_int64 * 1)((1 << 22) + 64)
    assert L.eogp_score_topk(fake, (1 << 19) + 8, fake, 4, 1, big, fake, (1 << 22) + 64, 1, 5,
                             fake, fake, None, fake, 1 << 20, None) == -1
    # workspace too small
    assert L.eogp_score_topk(fake, 8, fake, 4, 1, ks, fake, 64, 1, 5, fake, fake, None,
                             fake, 16, None) == -4


def test_workspace_size_queries_are_consistent():
    ks = [128, 256]
    small = E.eogp_score_topk_workspace_size(100, 3, ks, 10)
    big = E.eogp_score_topk_workspace_size(100000, 40, ks, 10)
    assert 0 < small < big
    L = E.load()
    a = L.eogp_rotate_retain_oneshot_workspace_size(4, 16, 64, 64, 500)
    b = L.eogp_rotate_retain_oneshot_workspace_size(8, 16, 64, 64, 500)
    c = L.eogp_rotate_retain_oneshot_workspace_size(8, 16, 64, 64, 4000)
    assert 0 < a < b < c
    assert L.eogp_rotate_retain_oneshot_workspace_size(8, 16, 64, 64, 0) == 0
    f16 = L.eogp_pca_project_workspace_size(100, 512, 128, 2, 0)     # fp16 P: split-K scratch
    f32 = L.eogp_pca_project_workspace_size(100, 512, 128, 0, 1)     # fp32 P: + split copy
    assert 0 < f16 < f32
    assert L.eogp_pca_project_workspace_size(1000, 512, 128, 2, 0) > f16


def test_score_binding_rejects_bad_layouts():
    """The Python binding checks dtypes and strides before anything reaches
    the library: codes must be uint8 with unit column stride, scales
    contiguous fp16 bit patterns [N, U], Y float32 with unit column stride."""
    import pytest
    import torch
    codes = torch.zeros((4, 16), dtype=torch.uint8)
    scales = torch.zeros((4, 2), dtype=torch.int16)
    Y = torch.zeros((3, 128), dtype=torch.float32)
    ks = [64, 64]
    with pytest.raises(ValueError, match="codes"):
        E.eogp_score_topk(codes.to(torch.int16), scales, ks, Y, 5)
    with pytest.raises(ValueError, match="codes"):
        E.eogp_score_topk(torch.zeros((16, 4), dtype=torch.uint8).t(), scales, ks, Y, 5)
    with pytest.raises(ValueError, match="scales"):
        E.eogp_score_topk(codes, scales.float(), ks, Y, 5)
    with pytest.raises(ValueError, match="scales"):
        E.eogp_score_topk(codes, torch.zeros((2, 4), dtype=torch.int16).t(), ks, Y, 5)
    with pytest.raises(ValueError, match="scales"):
        E.eogp_score_topk(codes, torch.zeros((4, 3), dtype=torch.int16), ks, Y, 5)
    with pytest.raises(ValueError, match="Y"):
        E.eogp_score_topk(codes, scales, ks, Y.half(), 5)
    with pytest.raises(ValueError, match="Y"):
        E.eogp_score_topk(codes, scales, ks, torch.zeros((128, 3)).t(), 5)
    # well-formed host tensors reach the device check
    with pytest.raises(ValueError, match="device"):
        E.eogp_score_topk(codes, scales, ks, Y, 5)


def test_multi_module_score_workspace_holds_the_exact_dots():
    """With several modules the workspace carries one 16-query pass of
    per-(module, query, row) integer dots: 4 bytes each while every k_u is at
    most 2^16, 8 bytes beyond."""
    N = 10000
    one = E.eogp_score_topk_workspace_size(N, 16, [4096], 10)
    two = E.eogp_score_topk_workspace_size(N, 16, [2048, 2048], 10)
    assert two - one >= 2 * 16 * N * 4
    wide = E.eogp_score_topk_workspace_size(N, 16, [1 << 17, 64], 10)
    assert wide - E.eogp_score_topk_workspace_size(N, 16, [1 << 17], 10) >= 2 * 16 * N * 8


def test_tiled_layout_argument_validation_without_device():
    """The tiled layout needs k (and every k_u) a multiple of 512, the
    module's steps inside the row, and 16-byte aligned codes."""
    L = E.load()
    fake = ctypes.c_void_p(0x1000)
    assert L.eogp_sign_pack_tiled(fake, 768, 4, 768, 0, fake, 4, 0, fake, 1, None) == -1
    assert L.eogp_sign_pack_tiled(fake, 1024, 4, 1024, 0, fake, 4, 3, fake, 1, None) == -1
    assert L.eogp_sign_pack_tiled(fake, 1024, 4, 1024, 0, ctypes.c_void_p(0x1008), 4, 0, fake, 1,
                                  None) == -1
    assert L.eogp_sign_pack_tiled(fake, 512, 4, 1024, 0, fake, 4, 0, fake, 1, None) == -1
    ks = (ctypes.c_int64 * 2)(512, 64)
    assert L.eogp_score_topk_tiled(fake, fake, 4, 2, ks, fake, 576, 1, 3, fake, fake, None, fake,
                                   1 << 20, None) == -1
    ks = (ctypes.c_int64 * 1)(512)
    assert L.eogp_score_topk_tiled(ctypes.c_void_p(0x1008), fake, 4, 1, ks, fake, 512, 1, 3, fake,
                                   fake, None, fake, 1 << 20, None) == -1
    assert L.eogp_score_topk_tiled(fake, fake, 4, 1, ks, fake, 512, 1, 3, fake, fake, None, fake,
                                   16, None) == -4
    assert E.tiled_store_bytes(33, [512, 1024]) == 2 * 3 * 2048
