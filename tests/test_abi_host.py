"""Host-only checks of the C ABI (no GPU needed): the library loads, exports
every function include/quads.h declares, and rejects invalid arguments with
the documented status codes before touching the GPU."""

import ctypes
import os
import re
import subprocess
import sys

import pytest

from paper_2607_15810_amd import quads as Q

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "quads.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][\w]*\s*\*?\s*([a-z_][a-z0-9_]*)\s*\(", src,
                       flags=re.M)
    return sorted(set(n for n in names if n not in ("if", "defined")))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(Q.LIB_PATH):
        pytest.fail("libquads.so is not built (python -m paper_2607_15810_amd.build)")
    return Q.lib()


def test_header_declares_the_seven_calls():
    names = declared_functions()
    for n in ["nvfp4_quantize_act", "nvfp4_quantize_weight", "moe_route_permute",
              "moe_w4a4_grouped_gemm", "rac_select_channels", "rac_residual_gemm",
              "moe_unpermute_combine"]:
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", Q.LIB_PATH], capture_output=True,
                         text=True).stdout
    exported = set(l.split()[-1] for l in out.splitlines() if " T " in l)
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, missing
    for n in declared_functions():
        assert n in Q.SIGNATURES, f"binding lacks {n}"
    # nothing else leaks out of the library
    assert exported == set(declared_functions())


def test_status_strings(lib):
    assert Q.status_string(0) == "ok"
    for st in range(-7, 0):
        assert Q.status_string(st) not in ("ok", "unknown status")
    assert lib.qd_version() >= 1


def _nv(groups, rows, cols, ptr=16):
    return Q.NVFP4(ptr, ptr, ptr, groups, rows, cols)


FAKE = 1 << 20            # an aligned, never-dereferenced address


def test_quantize_act_validation(lib):
    nv = _nv(1, 4, 32, FAKE)
    ws = lib.nvfp4_quantize_act_workspace(4, 32)
    r = lambda *a: Q.raw("nvfp4_quantize_act", *a)
    assert r(FAKE, 0, 4, 30, None, 0, ctypes.byref(_nv(1, 4, 30, FAKE)), None, None, FAKE, ws,
             None) == Q.QD_ERR_SHAPE
    assert r(FAKE, 7, 4, 32, None, 0, ctypes.byref(nv), None, None, FAKE, ws, None) == Q.QD_ERR_DTYPE
    assert r(None, 0, 4, 32, None, 0, ctypes.byref(nv), None, None, FAKE, ws, None) == Q.QD_ERR_NULL
    assert r(FAKE + 2, 0, 4, 32, None, 0, ctypes.byref(nv), None, None, FAKE, ws,
             None) == Q.QD_ERR_ALIGN
    assert r(FAKE, 0, 4, 32, None, 0, ctypes.byref(nv), None, None, FAKE, ws - 1,
             None) == Q.QD_ERR_WORKSPACE
    assert r(FAKE, 0, 4, 32, None, 0, ctypes.byref(_nv(1, 5, 32, FAKE)), None, None, FAKE, ws,
             None) == Q.QD_ERR_SHAPE
    # RAC statistics need an internally computed amax and bf16 input
    assert r(FAKE, 0, 4, 32, FAKE, 1, ctypes.byref(nv), FAKE, FAKE, FAKE, ws,
             None) == Q.QD_ERR_UNSUPPORTED
    assert r(FAKE, 1, 4, 32, None, 0, ctypes.byref(nv), FAKE, FAKE, FAKE, ws,
             None) == Q.QD_ERR_UNSUPPORTED
    # zero rows: a no-op that touches nothing
    assert r(None, 0, 0, 32, None, 0, ctypes.byref(_nv(1, 0, 32, 0)), None, None, FAKE, ws,
             None) == Q.QD_OK


def test_route_validation(lib):
    ws = lib.moe_route_permute_workspace(8, 16, 4)
    r = lambda *a: Q.raw("moe_route_permute", *a)
    args = [FAKE] * 6
    assert r(FAKE, 8, 16, 0, 1, *args[:5], FAKE, ws, None) == Q.QD_ERR_SHAPE     # k = 0
    assert r(FAKE, 8, 16, 17, 1, *args[:5], FAKE, ws, None) == Q.QD_ERR_SHAPE    # k > E
    assert r(FAKE, 8, 2000, 4, 1, *args[:5], FAKE, ws, None) == Q.QD_ERR_SHAPE   # E > 1024
    assert r(None, 8, 16, 4, 1, *args[:5], FAKE, ws, None) == Q.QD_ERR_NULL
    assert r(FAKE, 8, 16, 4, 1, *args[:5], FAKE, 8, None) == Q.QD_ERR_WORKSPACE


def test_gemm_validation(lib):
    a = _nv(1, 16, 256, FAKE)
    w = _nv(4, 128, 256, FAKE)
    # (a, row_token, offsets, E, rows, w, rq, sel, Ks, rq_sel, epilogue, out, amax, stream)
    r = lambda *x: Q.raw("moe_w4a4_grouped_gemm", *x)
    assert r(ctypes.byref(a), None, FAKE, 4, 16, ctypes.byref(w), None, None, 0, None, 5, FAKE,
             None, None) == Q.QD_ERR_DTYPE
    assert r(ctypes.byref(a), None, None, 4, 16, ctypes.byref(w), None, None, 0, None, 0, FAKE,
             None, None) == Q.QD_ERR_SHAPE          # E > 1 needs offsets
    w_badk = _nv(4, 128, 128, FAKE)
    assert r(ctypes.byref(a), None, FAKE, 4, 16, ctypes.byref(w_badk), None, None, 0, None, 0,
             FAKE, None, None) == Q.QD_ERR_SHAPE
    w_odd = _nv(4, 40, 256, FAKE)                  # SwiGLU needs N % 32 == 0
    assert r(ctypes.byref(a), FAKE, FAKE, 4, 16, ctypes.byref(w_odd), None, None, 0, None, 1,
             FAKE, None, None) == Q.QD_ERR_SHAPE
    rq = _nv(1, 16, 256, FAKE)
    assert r(ctypes.byref(a), FAKE, FAKE, 4, 16, ctypes.byref(w), ctypes.byref(rq), None, 4,
             None, 0, FAKE, None, None) == Q.QD_ERR_NULL     # residual without channel list
    assert r(ctypes.byref(a), FAKE, FAKE, 4, 16, ctypes.byref(w), None, FAKE, 4, None, 0,
             FAKE, None, None) == Q.QD_ERR_NULL     # K_s > 0 without the residual
    assert r(ctypes.byref(a), FAKE, FAKE, 4, 16, ctypes.byref(w), None, None, 0, None, 0,
             FAKE + 8, None, None) == Q.QD_ERR_ALIGN
    # many rows per expert: the tiled kernel needs the compact residual
    a_big = _nv(1, 4096, 256, FAKE)
    rq_big = _nv(1, 4096, 256, FAKE)
    w_big = _nv(4, 256, 256, FAKE)
    assert r(ctypes.byref(a_big), FAKE, FAKE, 4, 8192, ctypes.byref(w_big), ctypes.byref(rq_big),
             FAKE, 8, None, 1, FAKE, None, None) == Q.QD_ERR_NULL
    assert r(ctypes.byref(a_big), FAKE, FAKE, 4, 8192, ctypes.byref(w_big), ctypes.byref(rq_big),
             FAKE, 8, FAKE + 8, 1, FAKE, None, None) == Q.QD_ERR_ALIGN
    assert lib.moe_w4a4_grouped_gemm_amax_count(64, 256, 256, 4, 8, 1) > 0
    # the layer sizes its partial buffer with the same count the kernel writes
    assert lib.moe_w4a4_grouped_gemm_amax_count(8192, 256, 256, 4, 8, 1) % 8 == 0


def test_gather_selected_validation(lib):
    rq = _nv(1, 8, 64, FAKE)
    r = lambda *x: Q.raw("rac_gather_selected", *x)
    assert lib.rac_selected_width(0) == 0 and lib.rac_selected_width(1) == 16
    assert lib.rac_selected_width(64) == 64 and lib.rac_selected_width(65) == 80
    assert r(ctypes.byref(rq), FAKE, 65, FAKE, None) == Q.QD_ERR_SHAPE     # K_s > K
    assert r(ctypes.byref(rq), None, 4, FAKE, None) == Q.QD_ERR_NULL
    assert r(ctypes.byref(rq), FAKE, 4, FAKE + 8, None) == Q.QD_ERR_ALIGN
    assert r(ctypes.byref(rq), None, 0, FAKE, None) == Q.QD_OK            # nothing to gather


def test_select_and_combine_validation(lib):
    xq = _nv(1, 8, 64, FAKE)
    rq = _nv(1, 8, 64, FAKE)
    ws = lib.rac_select_channels_workspace(8, 64)
    r = lambda *x: Q.raw("rac_select_channels", *x)
    assert r(FAKE, ctypes.byref(xq), 65, FAKE, FAKE, 1, FAKE, ctypes.byref(rq), FAKE, ws,
             None) == Q.QD_ERR_SHAPE                 # K_s > K
    assert r(FAKE, ctypes.byref(xq), 4, FAKE, FAKE, 1, None, ctypes.byref(rq), FAKE, ws,
             None) == Q.QD_ERR_NULL
    assert r(FAKE, ctypes.byref(xq), 4, FAKE, FAKE, 1, FAKE, ctypes.byref(rq), FAKE, 0,
             None) == Q.QD_ERR_WORKSPACE
    c = lambda *x: Q.raw("moe_unpermute_combine", *x)
    assert c(FAKE, FAKE, FAKE, 4, 2, 12, FAKE, None) == Q.QD_ERR_SHAPE     # H % 8
    assert c(FAKE, FAKE, FAKE, 4, 33, 16, FAKE, None) == Q.QD_ERR_SHAPE    # k > 32
    assert c(None, None, None, 0, 2, 16, None, None) == Q.QD_OK           # empty batch


def test_layer_workspace_and_views(lib):
    n = lib.qd_moe_layer_workspace(256, 2048, 128, 8, 768)
    assert n > 256 * 8 * 2048 * 2             # holds z
    off = (ctypes.c_int64 * len(Q.VIEW_NAMES))()
    assert Q.raw("qd_moe_layer_views", 256, 2048, 128, 8, 768, off) == Q.QD_OK
    o = list(off)
    assert o == sorted(o) and len(set(o)) == len(o)
    assert all(v % 256 == 0 for v in o) and o[-1] < n
    # channel counts outside [0, H] (W13 site) and [0, I] (W2 site)
    F = 1 << 20
    w13 = Q.NVFP4(F, F, F, 4, 128, 256)
    w2 = Q.NVFP4(F, F, F, 4, 256, 64)
    f = lambda Ks, Ks2: Q.raw("qd_moe_layer_forward", F, F, 16, 256, 4, 2, 64, Ks, Ks2, 1,
                              ctypes.byref(w13), ctypes.byref(w2), F, F, 1 << 30, None)
    assert f(257, 0) == Q.QD_ERR_SHAPE
    assert f(8, 65) == Q.QD_ERR_SHAPE
    assert f(8, -1) == Q.QD_ERR_SHAPE


def test_injected_launch_failure():
    """QD_FAULT_INJECT=launch makes every launching call return QD_ERR_HIP
    after argument checks (run in a subprocess so the env is isolated)."""
    code = (
        "import ctypes\n"
        "from paper_2607_15810_amd import quads as Q\n"
        "L = Q.lib()\n"
        "F = 1 << 20\n"
        "nv = Q.NVFP4(F, F, F, 1, 4, 32)\n"
        "ws = L.nvfp4_quantize_act_workspace(4, 32)\n"
        "st = Q.raw('nvfp4_quantize_act', F, 0, 4, 32, None, 0, ctypes.byref(nv), None, None, F, ws, None)\n"
        "print(st)\n")
    env = dict(os.environ, QD_FAULT_INJECT="launch")
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env,
                         cwd=ROOT, timeout=120)
    assert out.returncode == 0, out.stderr
    assert int(out.stdout.strip().splitlines()[-1]) == Q.QD_ERR_HIP


def test_frag_scales_validation(lib):
    assert lib.nvfp4_frag_scales_bytes(2, 32, 512) == 2 * 32 * 32
    assert lib.nvfp4_frag_scales_bytes(2, 40, 512) == 0        # rows % 16
    assert lib.nvfp4_frag_scales_bytes(2, 32, 384) == 0        # cols % 256
    assert lib.nvfp4_frag_scales_bytes(0, 32, 512) == 0
    r = lib.nvfp4_pack_frag_scales
    assert r(None, FAKE, None) == Q.QD_ERR_NULL
    assert r(ctypes.byref(_nv(2, 32, 512, FAKE)), None, None) == Q.QD_ERR_NULL
    assert r(ctypes.byref(_nv(2, 40, 512, FAKE)), FAKE, None) == Q.QD_ERR_SHAPE
    assert r(ctypes.byref(_nv(2, 32, 384, FAKE)), FAKE, None) == Q.QD_ERR_SHAPE
    assert r(ctypes.byref(_nv(2, 32, 512, FAKE)), FAKE + 4, None) == Q.QD_ERR_ALIGN


def test_gemm_rejects_misaligned_frag_scales(lib):
    a = _nv(1, 16, 256, FAKE)
    w = _nv(4, 128, 256, FAKE)
    w.scales_frag = FAKE + 8
    offs = FAKE
    st = lib.moe_w4a4_grouped_gemm(ctypes.byref(a), None, offs, 4, 16, ctypes.byref(w), None,
                                   None, 0, None, 0, FAKE, None, None)
    assert st == Q.QD_ERR_ALIGN


def test_mxfp4_validation(lib):
    q = lib.mxfp4_quantize_rows
    assert q(FAKE, 0, 4, 40, FAKE, FAKE, None) == Q.QD_ERR_SHAPE       # cols % 32
    assert q(FAKE, 7, 4, 64, FAKE, FAKE, None) == Q.QD_ERR_DTYPE
    assert q(None, 0, 4, 64, FAKE, FAKE, None) == Q.QD_ERR_NULL
    assert q(FAKE + 2, 0, 4, 64, FAKE, FAKE, None) == Q.QD_ERR_ALIGN
    assert q(None, 0, 0, 64, None, None, None) == Q.QD_OK              # empty: nothing to do
    g = lib.moe_mxfp4_grouped_gemm
    args = lambda K, N, ws=FAKE: (FAKE, FAKE, 64, None, FAKE, 4, 64, FAKE, ws, N, K, 0, FAKE, None)
    assert g(*args(192, 256)) == Q.QD_ERR_UNSUPPORTED                  # K % 128
    assert g(*args(256, 200)) == Q.QD_ERR_UNSUPPORTED                  # N % 128
    assert g(*args(256, 256, FAKE + 2)) == Q.QD_ERR_ALIGN              # scales 4-byte aligned
    assert g(None, FAKE, 64, None, FAKE, 4, 64, FAKE, FAKE, 256, 256, 0, FAKE, None) == Q.QD_ERR_NULL
    assert g(FAKE, FAKE, 64, None, FAKE, 4, 64, FAKE, FAKE, 256, 256, 9, FAKE, None) == Q.QD_ERR_DTYPE
    lw = lib.qd_mxfp4_moe_layer_workspace
    assert lw(16, 256, 4, 2, 256) > 0
    f = lib.qd_mxfp4_moe_layer_forward
    assert f(FAKE, FAKE, 16, 256, 4, 2, 256, 1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 16,
             None) == Q.QD_ERR_WORKSPACE


def test_w4a16_validation(lib):
    F = 1 << 20
    w = Q.NVFP4(F, F, F, 2, 64, 128)          # E = 2 groups of [64][128]
    g = lambda *a: Q.raw("moe_w4a16_grouped_gemm", *a)
    assert g(F, 16, None, F, 2, 16, None, 0, F, None) == Q.QD_ERR_NULL           # no weights
    assert g(F, 16, None, F, 2, 16, ctypes.byref(w), 7, F, None) == Q.QD_ERR_DTYPE
    assert g(F, 16, None, None, 2, 16, ctypes.byref(w), 0, F, None) == Q.QD_ERR_SHAPE  # E > 1, no offsets
    assert g(F, 8, None, F, 2, 16, ctypes.byref(w), 0, F, None) == Q.QD_ERR_SHAPE  # rows > a_rows
    assert g(F, 16, None, F, 1025, 16, ctypes.byref(w), 0, F, None) == Q.QD_ERR_SHAPE
    w_bad_k = Q.NVFP4(F, F, F, 2, 64, 96)     # K % 64
    assert g(F, 16, None, F, 2, 16, ctypes.byref(w_bad_k), 0, F, None) == Q.QD_ERR_SHAPE
    w_bad_n = Q.NVFP4(F, F, F, 2, 48, 128)    # N % 32
    assert g(F, 16, None, F, 2, 16, ctypes.byref(w_bad_n), 0, F, None) == Q.QD_ERR_SHAPE
    assert g(F + 2, 16, None, F, 2, 16, ctypes.byref(w), 0, F, None) == Q.QD_ERR_ALIGN
    assert g(None, 0, None, F, 2, 0, ctypes.byref(w), 0, None, None) == Q.QD_OK   # no rows



def test_per_expert_validation(lib):
    """Per-expert RAC sets: argument checks before any launch."""
    xq = _nv(1, 8, 256, FAKE)
    rq = _nv(1, 8, 256, FAKE)
    ws = lib.rac_select_channels_per_expert_workspace(8, 256, 4)
    assert ws > 0
    r = lambda *x: Q.raw("rac_select_channels_per_expert", *x)
    # (x, xq, Ks, row_token, offsets, E, rows, scores_pe, ramax, sel_pe, rq, rq_rows, ws, ws_bytes, stream)
    assert r(FAKE, ctypes.byref(xq), 257, FAKE, FAKE, 4, 16, FAKE, FAKE, FAKE, ctypes.byref(rq),
             FAKE, FAKE, ws, None) == Q.QD_ERR_SHAPE          # K_s > K
    assert r(FAKE, ctypes.byref(xq), 4, None, FAKE, 4, 16, FAKE, FAKE, FAKE, ctypes.byref(rq),
             FAKE, FAKE, ws, None) == Q.QD_ERR_NULL           # no routing
    assert r(FAKE, ctypes.byref(xq), 4, FAKE, FAKE, 4, 16, FAKE, FAKE, None, ctypes.byref(rq),
             FAKE, FAKE, ws, None) == Q.QD_ERR_NULL           # K_s > 0 without the sets
    assert r(FAKE, ctypes.byref(xq), 4, FAKE, FAKE, 4, 16, FAKE, FAKE, FAKE, ctypes.byref(rq),
             FAKE, FAKE, 8, None) == Q.QD_ERR_WORKSPACE
    assert r(FAKE, ctypes.byref(xq), 4, FAKE, FAKE, 4, 16, FAKE, FAKE, FAKE, ctypes.byref(rq),
             FAKE + 8, FAKE, ws, None) == Q.QD_ERR_ALIGN
    a = _nv(1, 64, 256, FAKE)
    rq = _nv(1, 64, 256, FAKE)
    w = _nv(4, 256, 256, FAKE)
    g = lambda *x: Q.raw("moe_w4a4_grouped_gemm_per_expert", *x)
    # (a, row_token, offsets, E, rows, w, rq, sel_pe, Ks, rq_rows, epilogue, out, amax, stream)
    assert g(ctypes.byref(a), FAKE, FAKE, 4, 128, ctypes.byref(w), ctypes.byref(rq), FAKE, 0,
             FAKE, 1, FAKE, None, None) == Q.QD_ERR_SHAPE       # K_s >= 1
    assert g(ctypes.byref(a), FAKE, FAKE, 4, 128, ctypes.byref(w), ctypes.byref(rq), None, 4,
             FAKE, 1, FAKE, None, None) == Q.QD_ERR_NULL
    w_n = _nv(4, 80, 256, FAKE)                    # N not a multiple of 128: no tile kernel
    assert g(ctypes.byref(a), FAKE, FAKE, 4, 128, ctypes.byref(w_n), ctypes.byref(rq), FAKE, 4,
             FAKE, 0, FAKE, None, None) == Q.QD_ERR_UNSUPPORTED
    assert lib.moe_w4a4_grouped_gemm_per_expert_amax_count(128, 256, 256, 4, 4, 1) > 0
    assert lib.moe_w4a4_grouped_gemm_per_expert_amax_count(128, 80, 256, 4, 4, 1) == 0
    assert lib.qd_moe_layer_per_expert_workspace(64, 256, 4, 2, 128, 8) > 0
    lw = lambda *x: Q.raw("qd_moe_layer_forward_per_expert", *x)
    w13 = _nv(4, 256, 256, FAKE)
    w2 = _nv(4, 256, 128, FAKE)
    assert lw(FAKE, FAKE, 64, 256, 4, 2, 128, 0, 1, ctypes.byref(w13), ctypes.byref(w2), FAKE,
              FAKE, 1 << 30, None) == Q.QD_ERR_SHAPE           # K_s >= 1
    assert lw(FAKE, FAKE, 64, 256, 4, 2, 128, 8, 1, ctypes.byref(w13), ctypes.byref(w2), FAKE,
              FAKE, 16, None) == Q.QD_ERR_WORKSPACE
    assert lw(None, None, 0, 256, 4, 2, 128, 8, 1, ctypes.byref(w13), ctypes.byref(w2), None,
              None, 0, None) == Q.QD_OK                       # empty batch


def test_block_validation(lib):
    """The block entry point (RMSNorm + router folded ahead of the layer):
    argument checks before any launch, and its workspace and views."""
    T, H, E, k, I = 64, 256, 4, 2, 128
    n = lib.qd_moe_block_workspace(T, H, E, k, I)
    assert n > lib.qd_moe_layer_workspace(T, H, E, k, I) + T * H * 2
    off = (ctypes.c_int64 * (len(Q.VIEW_NAMES) + 2))()
    assert lib.qd_moe_block_views(T, H, E, k, I, off) == Q.QD_OK
    lo = (ctypes.c_int64 * len(Q.VIEW_NAMES))()
    assert lib.qd_moe_layer_views(T, H, E, k, I, lo) == Q.QD_OK
    assert list(off)[:len(Q.VIEW_NAMES)] == list(lo)
    nv = len(Q.VIEW_NAMES)
    assert off[nv] >= lib.qd_moe_layer_workspace(T, H, E, k, I)
    assert off[nv + 1] >= off[nv] + T * H * 2 and off[nv + 1] + T * E * 4 <= n
    w13 = _nv(E, 2 * I, H, FAKE)
    w2 = _nv(E, H, I, FAKE)
    b = lambda *x: Q.raw("qd_moe_block_forward", *x)
    # (h, gamma, eps, w_router, T, H, E, k, I, Ks, Ks2, renorm, w13, w2, y, ws, ws_bytes, stream)
    assert b(FAKE, FAKE, ctypes.c_float(1e-6), None, T, H, E, k, I, 8, 0, 1, ctypes.byref(w13),
             ctypes.byref(w2), FAKE, FAKE, n, None) == Q.QD_ERR_NULL     # no router
    assert b(FAKE, FAKE, ctypes.c_float(-1.0), FAKE, T, H, E, k, I, 8, 0, 1, ctypes.byref(w13),
             ctypes.byref(w2), FAKE, FAKE, n, None) == Q.QD_ERR_SHAPE    # eps < 0
    assert b(FAKE, FAKE, ctypes.c_float(float("inf")), FAKE, T, H, E, k, I, 8, 0, 1,
             ctypes.byref(w13), ctypes.byref(w2), FAKE, FAKE, n, None) == Q.QD_ERR_SHAPE
    assert b(FAKE, FAKE, ctypes.c_float(1e-6), FAKE, T, H, E, k, I, 8, 0, 1, ctypes.byref(w13),
             ctypes.byref(w2), FAKE, FAKE, n - 16, None) == Q.QD_ERR_WORKSPACE
    assert b(FAKE + 8, FAKE, ctypes.c_float(1e-6), FAKE, T, H, E, k, I, 8, 0, 1,
             ctypes.byref(w13), ctypes.byref(w2), FAKE, FAKE, n, None) == Q.QD_ERR_ALIGN
    w13b = _nv(300, 2 * I, H, FAKE)
    w2b = _nv(300, H, I, FAKE)
    assert b(FAKE, FAKE, ctypes.c_float(1e-6), FAKE, T, H, 300, k, I, 8, 0, 1,
             ctypes.byref(w13b), ctypes.byref(w2b), FAKE, FAKE, 1 << 40,
             None) == Q.QD_ERR_UNSUPPORTED                               # E > 256
    w13w = _nv(E, 2 * I, 9216, FAKE)
    w2w = _nv(E, 9216, I, FAKE)
    assert b(FAKE, FAKE, ctypes.c_float(1e-6), FAKE, T, 9216, E, k, I, 8, 0, 1,
             ctypes.byref(w13w), ctypes.byref(w2w), FAKE, FAKE, 1 << 40,
             None) == Q.QD_ERR_UNSUPPORTED                               # rows past LDS
    assert b(None, None, ctypes.c_float(1e-6), None, 0, H, E, k, I, 8, 0, 1, ctypes.byref(w13),
             ctypes.byref(w2), None, None, 0, None) == Q.QD_OK          # empty batch
