"""The C-ABI library on the CPU: it loads, exports every symbol the header
declares, and rejects bad arguments on the host before any HIP call."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dit_block.h")

B = pytest.importorskip("paper_2606_13501_amd.binding")


def _lib():
    if not os.path.exists(B.LIB_PATH):
        pytest.skip("libditblock.so not built")
    return B.lib()


def header_functions():
    txt = "".join(open(os.path.join(ROOT, "include", h)).read() for h in ("dit_block.h", "dit_sim.h", "dit_migrate.h"))
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(dit_[a-z_0-9]+)\s*\(", txt)))


def test_header_declares_expected_entry_points():
    fns = header_functions()
    for need in ("dit_block_forward", "dit_attention_varlen", "dit_adaln_modulate"):
        assert need in fns


def test_library_exports_every_header_function():
    _lib()
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (dit_[a-z_0-9]+)", out))
    missing = [f for f in header_functions() if f not in exported]
    assert not missing, f"declared but not exported: {missing}"
    assert sorted(header_functions()) == sorted(B.exported_symbols())


def test_abi_version_and_strings():
    L = _lib()
    assert L.dit_abi_version() == 4
    assert L.dit_status_string(B.DIT_ERR_WORKSPACE) == b"workspace too small"
    assert L.dit_status_string(B.DIT_OK) == b"ok"


# Fake, aligned, never-dereferenced device addresses: every call below must
# fail validation on the host before it could reach a kernel.
P = ctypes.c_void_p(0x10000)
P_MIS = ctypes.c_void_p(0x10008)


def _cu(a):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def test_attention_rejects_bad_arguments():
    L = _lib()
    cu, pcu = _cu([0, 10])
    bad, pbad = _cu([0, 10, 5])
    nz, pnz = _cu([1, 10])
    S = ctypes.c_void_p(0)
    # q, k, v, o in distinct (fake) ranges, so overlap is not what fails
    PK, PV, PO = ctypes.c_void_p(0x1000000), ctypes.c_void_p(0x2000000), ctypes.c_void_p(0x3000000)
    call = lambda q, pq, pk, n_req, H, d, scale, dt, qs=128: L.dit_attention_varlen(
        q, PK, PV, PO, qs, 128, 128, 128, pq, pk, n_req, H, d, scale, dt, S)
    assert call(None, pcu, pcu, 1, 1, 128, 0.1, B.DIT_BF16) == B.DIT_ERR_INVALID_ARG
    assert b"q is NULL" in L.dit_last_error()
    assert call(P_MIS, pcu, pcu, 1, 1, 128, 0.1, B.DIT_BF16) == B.DIT_ERR_INVALID_ARG
    assert b"aligned" in L.dit_last_error()
    assert call(P, pbad, pbad, 2, 1, 128, 0.1, B.DIT_BF16) == B.DIT_ERR_INVALID_ARG
    assert b"decreases" in L.dit_last_error()
    assert call(P, pnz, pnz, 1, 1, 128, 0.1, B.DIT_BF16) == B.DIT_ERR_INVALID_ARG
    assert call(P, pcu, pcu, 0, 1, 128, 0.1, B.DIT_BF16) == B.DIT_ERR_INVALID_ARG
    assert call(P, pcu, pcu, 65, 1, 128, 0.1, B.DIT_BF16) == B.DIT_ERR_INVALID_ARG
    assert call(P, pcu, pcu, 1, 1, 64, 0.1, B.DIT_BF16) == B.DIT_ERR_UNSUPPORTED
    assert call(P, pcu, pcu, 1, 1, 96, 0.1, B.DIT_F32) == B.DIT_ERR_UNSUPPORTED
    assert call(P, pcu, pcu, 1, 2, 128, 0.1, B.DIT_BF16) == B.DIT_ERR_INVALID_ARG   # stride < H*d
    # k / v row strides past 2^24 elements (the bf16 kernel's 32-bit tile offsets)
    big = lambda ks, vs: L.dit_attention_varlen(P, PK, PV, PO, 128, ks, vs, 128, pcu, pcu, 1, 1, 128, 0.1,
                                                B.DIT_BF16, S)
    assert big((1 << 24) + 8, 128) == B.DIT_ERR_INVALID_ARG and b"at most" in L.dit_last_error()
    assert big(128, (1 << 24) + 8) == B.DIT_ERR_INVALID_ARG and b"at most" in L.dit_last_error()
    assert call(P, pcu, pcu, 1, 1, 128, float("inf"), B.DIT_BF16) == B.DIT_ERR_INVALID_ARG
    assert call(P, pcu, pcu, 1, 1, 128, float("nan"), B.DIT_BF16) == B.DIT_ERR_INVALID_ARG
    assert b"softmax_scale" in L.dit_last_error()
    assert call(P, pcu, pcu, 1, 1, 128, 0.1, 7) == B.DIT_ERR_INVALID_ARG


def test_attention_rejects_output_overlapping_inputs():
    """o is written while q, k, v are read: any shared byte is rejected on the
    host (10 rows of stride 128 bf16 span 2,560 bytes)."""
    L = _lib()
    S = ctypes.c_void_p(0)
    cu, pcu = _cu([0, 10])
    q, k, v = 0x1000000, 0x2000000, 0x3000000
    f = lambda o, qs=128: L.dit_attention_varlen(ctypes.c_void_p(q), ctypes.c_void_p(k), ctypes.c_void_p(v),
                                                 ctypes.c_void_p(o), qs, 128, 128, 128, pcu, pcu, 1, 1, 128, 0.0,
                                                 B.DIT_BF16, S)
    assert f(q) == B.DIT_ERR_INVALID_ARG and b"o overlaps q" in L.dit_last_error()
    assert f(k + 2560 - 16) == B.DIT_ERR_INVALID_ARG and b"o overlaps k" in L.dit_last_error()
    assert f(v - 2560 + 16) == B.DIT_ERR_INVALID_ARG and b"o overlaps v" in L.dit_last_error()
    # o inside q's rows (interleaved columns of one buffer) counts as overlap
    assert f(q + 256, qs=256) == B.DIT_ERR_INVALID_ARG and b"o overlaps q" in L.dit_last_error()
    # q, k and v may share one buffer: only o's range matters (fails later, on the work-item count)
    cu2, pcu2 = _cu([0, 1 << 30])
    st = L.dit_attention_varlen(ctypes.c_void_p(q), ctypes.c_void_p(q + 256), ctypes.c_void_p(q + 512),
                                ctypes.c_void_p(1 << 46), 64 * 128 * 3, 64 * 128 * 3, 64 * 128 * 3, 64 * 128, pcu2,
                                pcu2, 1, 64, 128, 0.0, B.DIT_BF16, S)
    assert st == B.DIT_ERR_UNSUPPORTED and b"work items" in L.dit_last_error(), L.dit_last_error()


def test_linear_rejects_bad_arguments():
    L = _lib()
    S = ctypes.c_void_p(0)
    cu, pcu = _cu([0, 5, 12])
    f = lambda a, lda, M, N, K, epi, res, gate, pc, nreq, dt: L.dit_linear(
        a, lda, P, K, None, P, N, M, N, K, epi, res, N, gate, 0, pc, nreq, dt, S)
    assert f(P, 100, 12, 64, 100, B.EPI_NONE, None, None, None, 0, B.DIT_BF16) == B.DIT_ERR_INVALID_ARG  # lda % 8
    assert f(P, 96, 12, 64, 96, B.EPI_NONE, None, None, None, 0, B.DIT_BF16) == B.DIT_ERR_UNSUPPORTED   # K % 64
    assert f(P, 128, 12, 64, 128, B.EPI_RESIDUAL, None, None, None, 0, B.DIT_BF16) == B.DIT_ERR_INVALID_ARG
    assert f(P, 128, 12, 64, 128, B.EPI_GATED_RESIDUAL, P, None, pcu, 2, B.DIT_BF16) == B.DIT_ERR_INVALID_ARG
    assert f(P, 128, 13, 64, 128, B.EPI_GATED_RESIDUAL, P, P, pcu, 2, B.DIT_BF16) == B.DIT_ERR_INVALID_ARG
    assert b"cu_seqlens ends" in L.dit_last_error()
    assert f(P, 128, 12, 64, 128, 9, None, None, None, 0, B.DIT_BF16) == B.DIT_ERR_INVALID_ARG


def test_gemm_tile_width_hook():
    L = _lib()
    for bad in (1, 128, 200, -1, 512):
        assert L.dit_debug_gemm_tile_n(bad) == B.DIT_ERR_INVALID_ARG
        assert b"tile width" in L.dit_last_error()
    for good in (192, 256, 0):   # ends on 0: the per-shape choice
        assert L.dit_debug_gemm_tile_n(good) == B.DIT_OK


def test_attention_split_hook():
    L = _lib()
    for bad in (3, 8, -1, 5):
        assert L.dit_debug_attention_split(bad) == B.DIT_ERR_INVALID_ARG
        assert b"split mode" in L.dit_last_error()
    for good in (1, 2, 4, 0):   # ends on 0: the per-shape choice
        assert L.dit_debug_attention_split(good) == B.DIT_OK


def test_attention_shape_hook():
    L = _lib()
    for bad in (1, 2, 16, -4):
        assert L.dit_debug_attention_shape(bad) == B.DIT_ERR_INVALID_ARG
        assert b"waves" in L.dit_last_error()
    for good in (4, 8, 0):   # ends on 0: the choice per call
        assert L.dit_debug_attention_shape(good) == B.DIT_OK


def _cum(lens):
    out = [0]
    for n in lens:
        out.append(out[-1] + n)
    return out


def test_attention_plan_per_launch():
    """The bf16 attention's shape and split per launch on 256 compute units
    (host arithmetic).  Self-attention of one request: the 4-wave shape where
    the 8-wave items would end in a split last round and the launch is short
    (each such choice measured faster), else the 8-wave shape, split when
    its last round is at most half full."""
    plan = B.debug_attention_plan
    cases = {   # (tokens, heads): (waves, pieces, split items)
        (1024, 24): (4, 0, 0),       # at most 1024 keys
        (2048, 24): (8, 0, 0),       # 192 items: one round
        (3072, 24): (4, 0, 0),       # 288 items, 48-tile items
        (4096, 24): (4, 0, 0),       # 384 items: a half round left (the image block)
        (5120, 24): (8, 0, 0),       # 480 items: the last round 7/8 full
        (6144, 24): (8, 4, 64),      # 576 items of 96 tiles: too long for 4 waves
        (2048, 40): (4, 0, 0),
        (4096, 40): (4, 0, 0),       # 640 items of 64 tiles: 160 tiles per CU
        (8192, 40): (8, 0, 0),       # 5 full rounds
        (75600, 40): (8, 4, 64),     # 720p: 11,840 items, 64 left for a 47th round
    }
    for (T, H), want in cases.items():
        assert plan(_cum([T]), _cum([T]), H, 256) == want, (T, H)
    assert plan(_cum([75600]), _cum([512]), 40, 256) == (4, 0, 0)               # cross-attention
    assert plan(_cum([512, 1152, 4095, 9450]), _cum([4096, 9216, 32760, 75600]), 40, 256) == (8, 0, 0)
    # the same launch on 200 compute units: 384 items leave 184 for a second
    # round, more than half of it, so nothing is split and 8 waves run it
    assert plan(_cum([4096]), _cum([4096]), 24, 200) == (8, 0, 0)
    try:
        B.debug_attention_split(2)
        assert plan(_cum([4096]), _cum([4096]), 24, 256) == (8, 2, 128)         # forced split: 8 waves
        B.debug_attention_split(1)
        assert plan(_cum([75600]), _cum([75600]), 40, 256) == (8, 0, 0)
        B.debug_attention_split(0)
        B.debug_attention_shape(4)
        assert plan(_cum([75600]), _cum([75600]), 40, 256) == (4, 0, 0)
        B.debug_attention_shape(8)
        assert plan(_cum([4096]), _cum([4096]), 24, 256) == (8, 2, 128)
        assert plan(_cum([100]), _cum([77]), 2, 256) == (8, 0, 0)
    finally:
        B.debug_attention_split(0)
        B.debug_attention_shape(0)


def test_attention_plan_rejects_bad_arguments():
    L = _lib()
    cu = (ctypes.c_int32 * 2)(0, 100)
    bad_cu = (ctypes.c_int32 * 2)(5, 100)
    out = [ctypes.c_int() for _ in range(3)]
    refs = [ctypes.byref(x) for x in out]
    assert L.dit_debug_attention_plan(cu, cu, 1, 2, 256, *refs) == B.DIT_OK
    assert L.dit_debug_attention_plan(bad_cu, cu, 1, 2, 256, *refs) == B.DIT_ERR_INVALID_ARG
    assert L.dit_debug_attention_plan(cu, cu, 0, 2, 256, *refs) == B.DIT_ERR_INVALID_ARG
    assert L.dit_debug_attention_plan(cu, cu, 1, 0, 256, *refs) == B.DIT_ERR_INVALID_ARG
    assert L.dit_debug_attention_plan(cu, cu, 1, 2, 0, *refs) == B.DIT_ERR_INVALID_ARG
    assert b"compute_units" in L.dit_last_error()
    assert L.dit_debug_attention_plan(cu, cu, 1, 2, 256, None, refs[1], refs[2]) == B.DIT_ERR_INVALID_ARG


def test_norm_kernels_reject_bad_arguments():
    L = _lib()
    S = ctypes.c_void_p(0)
    cu, pcu = _cu([0, 4])
    assert L.dit_adaln_modulate(P, P, P, 3, pcu, 1, 64, 1e-6, P, B.DIT_BF16, S) == B.DIT_ERR_INVALID_ARG
    assert L.dit_adaln_modulate(P, P, P, 64, pcu, 1, 60, 1e-6, P, B.DIT_BF16, S) == B.DIT_ERR_INVALID_ARG
    assert L.dit_adaln_modulate(P, P, P, 64, pcu, 1, 16384, 1e-6, P, B.DIT_BF16, S) == B.DIT_ERR_UNSUPPORTED
    assert L.dit_adaln_modulate(P, P, P, 64, pcu, 1, 64, 0.0, P, B.DIT_BF16, S) == B.DIT_ERR_INVALID_ARG
    assert L.dit_layer_norm_affine(P, None, P, 4, 64, 1e-6, P, B.DIT_BF16, S) == B.DIT_ERR_INVALID_ARG
    sec = (ctypes.c_int * 3)(44, 42, 40)
    psec = ctypes.cast(sec, ctypes.POINTER(ctypes.c_int32))
    assert L.dit_qk_norm_rope(P, P, 256, 4, 2, 128, P, P, 1e-6, psec, 1e4, None, B.DIT_BF16, S) == B.DIT_ERR_INVALID_ARG
    assert b"sum to" in L.dit_last_error()
    sec = (ctypes.c_int * 3)(43, 43, 42)
    psec = ctypes.cast(sec, ctypes.POINTER(ctypes.c_int32))
    assert L.dit_qk_norm_rope(P, P, 256, 4, 2, 128, P, P, 1e-6, psec, 1e4, None, B.DIT_BF16, S) == B.DIT_ERR_INVALID_ARG
    assert L.dit_qk_norm_rope(P, P, 256, 4, 2, 96, P, P, 1e-6, None, 1e4, None, B.DIT_BF16, S) == B.DIT_ERR_UNSUPPORTED
    assert L.dit_gated_residual(P, P, None, P, 2, pcu, 1, 64, P, B.DIT_BF16, S) == B.DIT_ERR_INVALID_ARG
    assert L.dit_gated_residual(P, P, None, P, 64, pcu, 1, 8200, P, B.DIT_BF16, S) == B.DIT_ERR_UNSUPPORTED
    assert L.dit_gated_residual(P, P, None, P, 64, pcu, 1, 4100, P, B.DIT_F32, S) == B.DIT_ERR_UNSUPPORTED


def _block_structs(dtype=B.DIT_BF16, hidden=256, heads=2, head_dim=128, sections=(0, 64, 64)):
    cfg = B.BlockConfig(hidden, heads, head_dim, 512, hidden, sections, dtype)
    w = B.CWeights()
    for n in B.WEIGHT_FIELDS:
        setattr(w, n, 0x10000)
    vl = B.Varlen([0, 16, 40], [0, 8, 20], [(1, 4, 4), (1, 4, 6)])
    return cfg, w, vl


def test_block_validation_and_workspace():
    L = _lib()
    S = ctypes.c_void_p(0)
    cfg, w, vl = _block_structs()
    need = L.dit_block_workspace_size(ctypes.byref(cfg.c), ctypes.byref(vl.c))
    assert need > 0 and need % 256 == 0
    # workspace too small, misaligned, missing
    r = L.dit_block_forward(ctypes.byref(cfg.c), ctypes.byref(w), ctypes.byref(vl.c), P, P, None, P, P,
                            ctypes.c_void_p(0x100000), need - 256, S)
    assert r == B.DIT_ERR_WORKSPACE
    r = L.dit_block_forward(ctypes.byref(cfg.c), ctypes.byref(w), ctypes.byref(vl.c), P, P, None, P, P,
                            ctypes.c_void_p(0x100010), need, S)
    assert r == B.DIT_ERR_WORKSPACE
    # a weight missing
    w.w_up = None
    r = L.dit_block_forward(ctypes.byref(cfg.c), ctypes.byref(w), ctypes.byref(vl.c), P, P, None, P, P, P, need, S)
    assert r == B.DIT_ERR_INVALID_ARG and b"w_up" in L.dit_last_error()
    # with a precomputed modulation the block's timestep MLP and adaLN weights are not needed
    w.w_up = P.value
    w.w_t1 = w.w_ada = None
    r = L.dit_block_forward(ctypes.byref(cfg.c), ctypes.byref(w), ctypes.byref(vl.c), P, P, None, P, P, P, need, S)
    assert r == B.DIT_ERR_INVALID_ARG and b"w_t1" in L.dit_last_error()
    r = L.dit_block_forward(ctypes.byref(cfg.c), ctypes.byref(w), ctypes.byref(vl.c), P, None, P, P, P, None, need, S)
    assert r == B.DIT_ERR_WORKSPACE, L.dit_last_error()
    w.w_up = None
    # bad configs
    for kw, code in [(dict(head_dim=64, heads=4, sections=(0, 32, 32)), B.DIT_ERR_UNSUPPORTED),
                     (dict(sections=(0, 64, 62)), B.DIT_ERR_INVALID_ARG),
                     (dict(hidden=250), B.DIT_ERR_INVALID_ARG)]:
        cfg2, w2, vl2 = _block_structs(**kw)
        r = L.dit_block_forward(ctypes.byref(cfg2.c), ctypes.byref(w2), ctypes.byref(vl2.c), P, P, None, P, P, P, 1 << 40,
                                S)
        assert r == code, (kw, r, L.dit_last_error())
        assert L.dit_block_workspace_size(ctypes.byref(cfg2.c), ctypes.byref(vl2.c)) == 0
    # rows of a request that do not fit its grid
    cfg, w, vl = _block_structs()
    vl = B.Varlen([0, 17, 40], [0, 8, 20], [(1, 4, 4), (1, 4, 6)])
    r = L.dit_block_forward(ctypes.byref(cfg.c), ctypes.byref(w), ctypes.byref(vl.c), P, P, None, P, P, P, 1 << 40, S)
    assert r == B.DIT_ERR_INVALID_ARG and b"exceed its grid" in L.dit_last_error()


# ---------------------------------------------------------------- the denoising step


def _step_args(grids=((3, 4, 6), (1, 6, 10)), rows=None, C=16, patch=(1, 2, 2), n_blocks=2, dtype=None,
               pos_offset=None):
    dtype = B.DIT_BF16 if dtype is None else dtype
    bc = B.BlockConfig(256, 2, 128, 1024, 256, (44, 42, 42), dtype)
    cfg = B.ModelConfig(bc, n_blocks, C, patch)
    rows = rows or [f * h * w for f, h, w in grids]
    cu = np.cumsum([0] + list(rows))
    vl = B.Varlen(cu, [40 * i for i in range(len(rows) + 1)], list(grids), pos_offset)
    blk = B.CWeights()
    for n in B.WEIGHT_FIELDS:
        setattr(blk, n, P.value)
    w = B.ModelWeights({}, [blk] * max(n_blocks, 1))
    for n in B.MODEL_FIELDS:
        setattr(w.c, n, P.value)
    return cfg, vl, w


def _step_call(cfg, vl, w, ws=None, ws_bytes=0, latent=P, kv=P):
    L = _lib()
    return L.dit_denoise_step(ctypes.byref(cfg.c), ctypes.byref(w.c), ctypes.byref(vl.c), latent, P, P, kv, P, ws,
                              ws_bytes, ctypes.c_void_p(0))


def test_denoise_step_sizes():
    L = _lib()
    cfg, vl, w = _step_args()
    assert L.dit_text_kv_elems(ctypes.byref(cfg.c), ctypes.byref(vl.c)) == 2 * 80 * 2 * 256
    need = L.dit_denoise_workspace_size(ctypes.byref(cfg.c), ctypes.byref(vl.c))
    blk = L.dit_block_workspace_size(ctypes.byref(cfg.block.c), ctypes.byref(vl.c))
    assert need > 0 and blk > 0
    # x and the patch tokens on top of a block workspace without text keys/values
    assert need >= 132 * 256 * 2 + 132 * 64 * 2
    cfg2, vl2, _ = _step_args(rows=[72, 59])
    assert L.dit_denoise_workspace_size(ctypes.byref(cfg2.c), ctypes.byref(vl2.c)) == 0


def test_denoise_step_rejects_bad_arguments():
    L = _lib()
    cfg, vl, w = _step_args()
    # valid arguments up to the workspace: fails on the workspace, launches nothing
    assert _step_call(cfg, vl, w) == B.DIT_ERR_WORKSPACE
    assert _step_call(cfg, vl, w, ws=P, ws_bytes=1024) == B.DIT_ERR_WORKSPACE
    assert _step_call(cfg, vl, w, latent=None) == B.DIT_ERR_INVALID_ARG
    assert _step_call(cfg, vl, w, kv=P_MIS) == B.DIT_ERR_INVALID_ARG
    cfg2, vl2, w2 = _step_args(rows=[72, 59])
    assert _step_call(cfg2, vl2, w2) == B.DIT_ERR_INVALID_ARG
    assert b"whole grid" in L.dit_last_error()
    cfg2, vl2, w2 = _step_args(pos_offset=[0, 4])
    assert _step_call(cfg2, vl2, w2) == B.DIT_ERR_INVALID_ARG
    assert b"pos_offset" in L.dit_last_error()
    cfg2, vl2, w2 = _step_args(C=3)
    assert _step_call(cfg2, vl2, w2) == B.DIT_ERR_UNSUPPORTED
    cfg2, vl2, w2 = _step_args(C=3, patch=(1, 1, 1), grids=((3, 8, 12), (1, 12, 20)), dtype=B.DIT_F32)
    assert _step_call(cfg2, vl2, w2) == B.DIT_ERR_UNSUPPORTED
    cfg2, vl2, w2 = _step_args(patch=(1, 0, 2))
    assert _step_call(cfg2, vl2, w2) == B.DIT_ERR_INVALID_ARG
    cfg2, vl2, w2 = _step_args(n_blocks=0)
    assert _step_call(cfg2, vl2, w2) == B.DIT_ERR_INVALID_ARG
    w.c.w_out = None
    assert _step_call(cfg, vl, w) == B.DIT_ERR_INVALID_ARG
    assert b"w_out" in L.dit_last_error()
    cfg, vl, w = _step_args()
    w.blocks[1].w_qkv = None
    assert _step_call(cfg, vl, w) == B.DIT_ERR_INVALID_ARG
    assert b"block 1" in L.dit_last_error() and b"w_qkv" in L.dit_last_error()
    cfg, vl, w = _step_args()
    w.blocks[0].w_t1 = None     # the blocks' own timestep MLP is not read by the step
    assert _step_call(cfg, vl, w) == B.DIT_ERR_WORKSPACE


def test_text_kv_and_latent_stages_reject_bad_arguments():
    L = _lib()
    S = ctypes.c_void_p(0)
    cfg, vl, w = _step_args()
    assert L.dit_text_kv(ctypes.byref(cfg.c), ctypes.byref(w.c), ctypes.byref(vl.c), None, P, S) == \
        B.DIT_ERR_INVALID_ARG
    w.blocks[1].w_ckv = None
    assert L.dit_text_kv(ctypes.byref(cfg.c), ctypes.byref(w.c), ctypes.byref(vl.c), P, P, S) == \
        B.DIT_ERR_INVALID_ARG
    assert b"block 1" in L.dit_last_error()
    cfg2, vl2, _ = _step_args(rows=[72, 61])
    assert L.dit_patchify(ctypes.byref(cfg2.c), ctypes.byref(vl2.c), P, P, S) == B.DIT_ERR_INVALID_ARG
    assert L.dit_unpatchify_euler(ctypes.byref(cfg.c), ctypes.byref(vl.c), P, P, None, P, S) == \
        B.DIT_ERR_INVALID_ARG
    assert L.dit_patchify(ctypes.byref(cfg.c), ctypes.byref(vl.c), P_MIS, P, S) == B.DIT_ERR_INVALID_ARG


def test_attention_rejects_too_many_work_items():
    """2^30 query rows x 64 heads is more 256-row work items than the kernel
    numbers (2^27): rejected on the host, nothing launched."""
    L = _lib()
    cu, pcu = _cu([0, 1 << 30])
    st = L.dit_attention_varlen(P, P, P, ctypes.c_void_p(1 << 46), 64 * 128, 64 * 128, 64 * 128, 64 * 128, pcu,
                                pcu, 1, 64, 128, 0.1, B.DIT_BF16, ctypes.c_void_p(0))
    assert st == B.DIT_ERR_UNSUPPORTED and b"work items" in L.dit_last_error(), L.dit_last_error()


def test_block_seams_take_timesteps_or_modulation():
    """Both seams take the conditioning as dit_block_forward does: t (the
    block's timestep MLP and adaLN weights are read) or a precomputed mod
    (those weights are not read).  Every call stops at the workspace check,
    after the arguments it depends on have been accepted."""
    L = _lib()
    S = ctypes.c_void_p(0)
    cfg, w, vl = _block_structs()
    need = L.dit_block_workspace_size(ctypes.byref(cfg.c), ctypes.byref(vl.c))
    pre = lambda w, t, mod: L.dit_block_pre_attention(ctypes.byref(cfg.c), ctypes.byref(w), ctypes.byref(vl.c), P, t,
                                                       mod, P, None, need, S)
    post = lambda w, t, mod: L.dit_block_post_attention(ctypes.byref(cfg.c), ctypes.byref(w), ctypes.byref(vl.c), P,
                                                         P, P, t, mod, P, None, need, S)
    assert pre(w, P, P) == B.DIT_ERR_WORKSPACE
    assert post(w, None, P) == B.DIT_ERR_WORKSPACE
    assert post(w, P, None) == B.DIT_ERR_WORKSPACE
    assert post(w, None, None) == B.DIT_ERR_INVALID_ARG and b"t is NULL" in L.dit_last_error()
    assert pre(w, None, None) == B.DIT_ERR_INVALID_ARG and b"mod is NULL" in L.dit_last_error()
    for missing in ("w_t1", "b_t2", "w_ada"):
        cfg, w, vl = _block_structs()
        setattr(w, missing, None)
        # from t: the conditioning weights are needed
        assert pre(w, P, P) == B.DIT_ERR_INVALID_ARG and missing.encode() in L.dit_last_error()
        assert post(w, P, None) == B.DIT_ERR_INVALID_ARG and missing.encode() in L.dit_last_error()
        # from mod: they are not read
        assert pre(w, None, P) == B.DIT_ERR_WORKSPACE, L.dit_last_error()
        assert post(w, None, P) == B.DIT_ERR_WORKSPACE, L.dit_last_error()


def test_noalloc_modulation_rejects_before_any_device_call():
    """The no-workspace conditioning validates like dit_timestep_modulation and
    rejects a scratch need over its static array on the host."""
    L = _lib()
    S = ctypes.c_void_p(0)
    cfg, w, _ = _block_structs()
    f = lambda cfg, n, t=P, mod=P: L.dit_timestep_modulation_noalloc(ctypes.byref(cfg.c), ctypes.byref(w), n, t, mod, S)
    assert f(cfg, 0) == B.DIT_ERR_INVALID_ARG
    assert f(cfg, 65) == B.DIT_ERR_INVALID_ARG
    assert f(cfg, 1, t=None) == B.DIT_ERR_INVALID_ARG and b"t is NULL" in L.dit_last_error()
    assert f(cfg, 1, mod=P_MIS) == B.DIT_ERR_INVALID_ARG
    w.w_ada = None
    assert f(cfg, 1) == B.DIT_ERR_INVALID_ARG and b"w_ada" in L.dit_last_error()
    w.w_ada = P.value
    # F = 32768, D = 8192, 64 requests: (F + 2D) * 64 * 4 = 12 MiB > 8 MiB
    big = B.BlockConfig(8192, 64, 128, 8192, 32768, (0, 64, 64), B.DIT_BF16)
    assert f(big, 64) == B.DIT_ERR_UNSUPPORTED and b"static array" in L.dit_last_error()
