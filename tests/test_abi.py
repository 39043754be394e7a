"""Host-only checks of the C ABI: the library loads, exports every entry point
declared in include/moe.h, and rejects bad arguments before touching the GPU
(every call below returns from host-side validation; no HIP call is made)."""
import ctypes
import os
import re

import pytest

from tests.conftest import ROOT

HEADER = os.path.join(ROOT, "include", "moe.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def m():
    from paper_2609_15627_amd import moe
    return moe


def test_header_declares_the_four_layer_calls():
    names = declared_functions()
    for n in ("moe_route_topk", "moe_permute", "moe_fp4_grouped_gemm", "moe_combine_fixed_order"):
        assert n in names


def test_library_exports_every_declared_symbol(m):
    lib = ctypes.CDLL(m.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_covers_every_declared_symbol(m):
    assert set(declared_functions()) <= set(m._SIGNATURES)


def test_status_strings(m):
    for s in range(5):
        assert m.lib.moe_status_string(s)
    assert m.lib.moe_last_variant() == m.VARIANT_NONE


FAKE = ctypes.c_void_p(0x1000)   # never dereferenced: validation fails first
NUL = ctypes.c_void_p(0)


@pytest.mark.parametrize("args", [
    (FAKE, -1, 8, 2, 0, FAKE, FAKE, NUL),          # T < 0
    (FAKE, 4, 0, 1, 0, FAKE, FAKE, NUL),           # E < 1
    (FAKE, 4, 8, 9, 0, FAKE, FAKE, NUL),           # k > E
    (FAKE, 4, 8, 0, 0, FAKE, FAKE, NUL),           # k < 1
    (FAKE, 4, 8, 2, 2, FAKE, FAKE, NUL),           # n_shared not 0/1
    (FAKE, 4, 2048, 2, 0, FAKE, FAKE, NUL),        # E > MOE_MAX_EXPERTS
    (FAKE, 4, 64, 33, 0, FAKE, FAKE, NUL),         # k_total > 32
    (NUL, 4, 8, 2, 0, FAKE, FAKE, NUL),            # null logits
    (FAKE, 4, 8, 2, 0, NUL, FAKE, NUL),            # null ids
])
def test_route_rejects(m, args):
    assert m.lib.moe_route_topk(*args) == m.MOE_ERR_INVALID_ARG


def test_permute_rejects(m):
    L = m.lib
    assert L.moe_permute(FAKE, -1, 8, 2, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, NUL) == 1
    assert L.moe_permute(FAKE, 4, 0, 2, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, NUL) == 1
    assert L.moe_permute(FAKE, 4, 4096, 2, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, NUL) == 1
    assert L.moe_permute(FAKE, 4, 8, 0, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, NUL) == 1
    assert L.moe_permute(FAKE, 4, 8, 2, NUL, FAKE, FAKE, FAKE, FAKE, 1 << 20, NUL) == 1
    # large inputs need a workspace
    assert L.moe_permute(FAKE, 4096, 8, 2, FAKE, FAKE, FAKE, FAKE, NUL, 0, NUL) == m.MOE_ERR_WORKSPACE
    need = m.moe_permute_workspace_bytes(4096, 8, 2)
    assert L.moe_permute(FAKE, 4096, 8, 2, FAKE, FAKE, FAKE, FAKE, FAKE, need - 1, NUL) == 3


def test_gemm_rejects(m):
    L = m.lib
    base = dict(T=8, H=256, I=128, NE=4, kt=2, f=0)

    def call(ws_bytes=1 << 30, ws=FAKE, **kw):
        a = dict(base, **kw)
        return L.moe_fp4_grouped_gemm(FAKE, a["T"], a["H"], a["I"], a["NE"], a["kt"], FAKE, FAKE,
                                      FAKE, FAKE, FAKE, FAKE, a["f"], FAKE, ws, ws_bytes, NUL)
    assert call(H=200) == 1            # H % 128
    assert call(I=96) == 1             # I % 128
    assert call(T=-1) == 1
    assert call(NE=0) == 1
    assert call(kt=40) == 1
    assert call(f=7) == 1
    assert call(ws=NUL) == m.MOE_ERR_WORKSPACE
    assert call(f=1, ws=NUL) == m.MOE_ERR_WORKSPACE   # MXFP6 goes as far as the workspace check
    # MXFP6 blocks sit in 32-byte slots in the workspace: as many code bytes as MXFP8
    assert m.moe_fp4_grouped_gemm_workspace_layout(8, 256, 128, 4, 2, "e2m3") == \
        m.moe_fp4_grouped_gemm_workspace_layout(8, 256, 128, 4, 2, "e4m3")
    need = m.moe_fp4_grouped_gemm_workspace_bytes(8, 256, 128, 4, 2, "e4m3")
    assert need > 0 and call(ws_bytes=need - 1) == m.MOE_ERR_WORKSPACE
    assert m.moe_fp4_grouped_gemm_workspace_bytes(8, 200, 128, 4, 2) == 0


def test_workspace_layout_is_ordered_and_sized(m):
    for fmt in ("e4m3", "e2m1"):
        off = m.moe_fp4_grouped_gemm_workspace_layout(64, 4096, 2048, 257, 9, fmt)
        assert off == sorted(off) and all(o % 256 == 0 for o in off)
        bits = m.ACT_BITS[fmt]
        assert off[1] - off[0] >= 64 * 4096 * bits // 8
        assert off[3] - off[2] >= 64 * 9 * 2048 * bits // 8
        assert off[5] == m.moe_fp4_grouped_gemm_workspace_bytes(64, 4096, 2048, 257, 9, fmt)


def test_combine_quant_logits_reject(m):
    L = m.lib
    assert L.moe_combine_fixed_order(FAKE, FAKE, 4, 100, 2, FAKE, NUL) == 1   # H % 8
    assert L.moe_combine_fixed_order(FAKE, FAKE, 4, 128, 0, FAKE, NUL) == 1
    assert L.moe_combine_fixed_order(NUL, FAKE, 4, 128, 2, FAKE, NUL) == 1
    assert L.moe_quantize_act(FAKE, 4, 100, 0, FAKE, FAKE, NUL) == 1          # K % 32
    assert L.moe_quantize_act(FAKE, 4, 128, 9, FAKE, FAKE, NUL) == 1          # format
    assert L.moe_router_logits(FAKE, FAKE, 4, 100, 8, FAKE, NUL) == 1         # H % 8
    assert L.moe_router_logits(FAKE, FAKE, 4, 128, 0, FAKE, NUL) == 1
    assert L.moe_probe_scaled_mfma(NUL, FAKE, 0, FAKE, FAKE, FAKE, NUL) == 1


def test_route_ex_and_router_reject(m):
    L = m.lib
    ref = ctypes.byref

    def opts(score=0, ng=1, tg=1):
        return m._RouteOpts(score, None, ng, tg, 1, 1.0)
    ok = opts()
    assert L.moe_route_topk_ex(FAKE, 4, 8, 2, 0, None, FAKE, FAKE, NUL) == 1    # opts NULL
    assert L.moe_route_topk_ex(FAKE, 4, 8, 2, 0, ref(opts(score=2)), FAKE, FAKE, NUL) == 1
    assert L.moe_route_topk_ex(FAKE, 4, 8, 2, 0, ref(opts(ng=3)), FAKE, FAKE, NUL) == 1  # 3 !| 8
    assert L.moe_route_topk_ex(FAKE, 4, 8, 2, 0, ref(opts(ng=0)), FAKE, FAKE, NUL) == 1
    assert L.moe_route_topk_ex(FAKE, 4, 8, 2, 0, ref(opts(ng=4, tg=5)), FAKE, FAKE, NUL) == 1
    # k larger than the experts of the kept groups (1 group of 2)
    assert L.moe_route_topk_ex(FAKE, 4, 8, 3, 0, ref(opts(ng=4, tg=1)), FAKE, FAKE, NUL) == 1
    assert L.moe_route_topk_ex(NUL, 4, 8, 2, 0, ref(ok), FAKE, FAKE, NUL) == 1     # null logits
    assert L.moe_router_topk(FAKE, FAKE, 4, 100, 8, 2, 0, None, NUL, FAKE, FAKE, NUL) == 1  # H % 128
    assert L.moe_router_topk(FAKE, FAKE, 4, 128, 8, 9, 0, None, NUL, FAKE, FAKE, NUL) == 1  # k > E
    assert L.moe_router_topk(FAKE, FAKE, 4, 128, 1025, 8, 0, None, NUL, FAKE, FAKE, NUL) == 1  # E
    assert L.moe_router_topk(NUL, FAKE, 4, 128, 8, 2, 0, None, NUL, FAKE, FAKE, NUL) == 1   # null x


def test_gemm_stages_combine_and_formats_reject(m):
    L = m.lib

    def stages(st, f=0, ws=FAKE):
        return L.moe_fp4_grouped_gemm_stages(FAKE, 8, 256, 128, 4, 2, FAKE, FAKE, FAKE, FAKE, FAKE,
                                             FAKE, f, FAKE, ws, 1 << 30, st, NUL)
    assert stages(0) == 1 and stages(8) == 1          # stage mask outside 1..7
    assert stages(7, f=9) == 1                        # format
    assert stages(7, ws=NUL) == m.MOE_ERR_WORKSPACE

    def comb(f=0, T=8, H=256, topk_w=FAKE, out=FAKE):
        return L.moe_fp4_grouped_gemm_combine(FAKE, T, H, 128, 4, 2, FAKE, FAKE, FAKE, FAKE, FAKE,
                                              FAKE, f, topk_w, out, FAKE, 1 << 30, 7, NUL)
    assert comb(H=200) == 1
    assert comb(topk_w=NUL) == 1 and comb(out=NUL) == 1
    assert comb(f=1) == m.MOE_ERR_UNSUPPORTED          # MXFP6
    assert L.moe_fp4_grouped_gemm_combine_supported(8, 200, 128, 4, 2, 0) == 0
    assert L.moe_fp4_grouped_gemm_combine_supported(8, 256, 128, 4, 2, 1) == 0
    assert L.moe_fp4_grouped_gemm_combine_supported(8, 256, 128, 4, 2, 3) == 0   # BF16 contract
    # the BF16 contract has no standalone activation quantisation
    assert L.moe_quantize_act(FAKE, 4, 128, m.ACT_FORMATS["bf16"], FAKE, FAKE, NUL) == 1
    # BF16 workspace: no x codes, no scales
    off = m.moe_fp4_grouped_gemm_workspace_layout(64, 4096, 2048, 257, 9, "bf16")
    assert off[0] == off[1] == off[2] and off[3] == off[4]
    assert off[3] - off[2] >= 64 * 9 * 2048 * 2


def test_gemm_rejects_shapes_past_32_bit_offsets(m):
    """x of 4 GiB (2^20 tokens x 4096 FP8 codes) is refused before anything
    is enqueued; one token fewer still passes the check (then fails on the
    fake workspace size instead)."""
    L = m.lib

    def call(T, f=0):
        return L.moe_fp4_grouped_gemm(FAKE, T, 4096, 128, 4, 1, FAKE, FAKE, FAKE, FAKE, FAKE,
                                      FAKE, f, FAKE, FAKE, 16, NUL)
    assert call(1 << 20) == m.MOE_ERR_UNSUPPORTED
    assert call((1 << 20) - 1) == m.MOE_ERR_WORKSPACE
    assert call(1 << 19, f=m.ACT_FORMATS["bf16"]) == m.MOE_ERR_UNSUPPORTED   # 2 bytes an element


def test_noalloc_gemm_rejects_before_touching_the_gpu(m):
    """The allocation-free grouped GEMM validates like moe_fp4_grouped_gemm and
    refuses shapes whose workspace exceeds its static scratch, before any HIP
    call (so these run without a GPU)."""
    L = m.lib

    def call(T, H=4096, I=2048, NE=257, kt=9, f=0, x=FAKE):
        return L.moe_fp4_grouped_gemm_noalloc(x, T, H, I, NE, kt, FAKE, FAKE, FAKE, FAKE, FAKE,
                                              FAKE, f, FAKE, NUL)
    need = m.moe_fp4_grouped_gemm_workspace_bytes
    big = next(T for T in range(1000, 4000, 8) if need(T, 4096, 2048, 257, 9) > m.NOALLOC_SCRATCH_BYTES)
    assert need(big - 8, 4096, 2048, 257, 9) <= m.NOALLOC_SCRATCH_BYTES < need(big, 4096, 2048, 257, 9)
    assert call(big) == m.MOE_ERR_WORKSPACE
    assert call(8192) == m.MOE_ERR_WORKSPACE
    assert call(64, H=200) == m.MOE_ERR_INVALID_ARG                  # H % 128
    assert call(64, f=9) == m.MOE_ERR_INVALID_ARG                    # format
    assert call(64, x=NUL) == m.MOE_ERR_INVALID_ARG                  # null pointer
    assert call(0) == m.MOE_OK                                       # empty batch: nothing enqueued


def test_set_tiled_rows_validation(m):
    """The row-tile control takes 0, 128 or 256 and rejects anything else
    (host only)."""
    L = m.lib
    try:
        for bad in (-1, 1, 64, 192, 512):
            assert L.moe_set_tiled_rows(bad) == 1
        for ok in (128, 256, 0):
            assert L.moe_set_tiled_rows(ok) == 0
    finally:
        L.moe_set_tiled_rows(0)


def test_pack_fp4_weights_validation(m):
    """The weight packing call rejects shapes outside its layout and
    overlapping or misaligned buffers on the host."""
    L = m.lib
    buf = ctypes.create_string_buffer(64 * 1024 + 16)
    base = (ctypes.addressof(buf) + 15) // 16 * 16
    src, dst = ctypes.c_void_p(base), ctypes.c_void_p(base + 32 * 1024)
    assert L.moe_pack_fp4_weights(src, dst, 0, 128, NUL) == 0        # nothing to do
    assert L.moe_pack_fp4_weights(src, dst, 15, 128, NUL) == 1       # rows % 16
    assert L.moe_pack_fp4_weights(src, dst, 16, 96, NUL) == 1        # K % 128
    assert L.moe_pack_fp4_weights(src, dst, -16, 128, NUL) == 1
    assert L.moe_pack_fp4_weights(src, src, 16, 128, NUL) == 1       # in place
    assert L.moe_pack_fp4_weights(src, ctypes.c_void_p(base + 512), 16, 128, NUL) == 1  # overlap
    assert L.moe_pack_fp4_weights(ctypes.c_void_p(base + 4), dst, 16, 128, NUL) == 1    # alignment
    assert L.moe_pack_fp4_weights(None, dst, 16, 128, NUL) == 1
