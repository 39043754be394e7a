"""Python binding of libmoe.so (include/moe.h): argument marshalling only.

Every function takes and returns torch tensors on the GPU; torch provides the
device memory and the stream, every step of the layer runs in the library's
HIP kernels. The library must be built (``__graft_entry__.build()`` or
``python -m paper_2609_15627_amd._build``); importing this module without it
raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmoe.so")

MOE_OK, MOE_ERR_INVALID_ARG, MOE_ERR_UNSUPPORTED, MOE_ERR_WORKSPACE, MOE_ERR_LAUNCH = range(5)
ACT_FORMATS = {"e4m3": 0, "e2m3": 1, "e2m1": 2, "bf16": 3}
ACT_BITS = {"e4m3": 8, "e2m3": 6, "e2m1": 4, "bf16": 16}
VARIANT_NONE, VARIANT_STREAM, VARIANT_TILED, VARIANT_BF16, VARIANT_MIXED = 0, 1, 2, 3, 4
VARIANT_BF16_STREAM = 5
VARIANT_SHORT = 6
WS_REGIONS = 6

_P = ctypes.c_void_p
_I = ctypes.c_int
_SZ = ctypes.c_size_t

_SIGNATURES = {
    "moe_router_logits": (_I, [_P, _P, _I, _I, _I, _P, _P]),
    "moe_route_topk": (_I, [_P, _I, _I, _I, _I, _P, _P, _P]),
    "moe_route_topk_ex": (_I, [_P, _I, _I, _I, _I, _P, _P, _P, _P]),
    "moe_router_topk": (_I, [_P, _P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P]),
    "moe_permute_workspace_bytes": (_SZ, [_I, _I, _I]),
    "moe_permute": (_I, [_P, _I, _I, _I, _P, _P, _P, _P, _P, _SZ, _P]),
    "moe_quantize_act": (_I, [_P, _I, _I, _I, _P, _P, _P]),
    "moe_pack_fp4_weights": (_I, [_P, _P, ctypes.c_long, _I, _P]),
    "moe_set_tiled_rows": (_I, [_I]),
    "moe_fp4_grouped_gemm_workspace_bytes": (_SZ, [_I, _I, _I, _I, _I, _I]),
    "moe_fp4_grouped_gemm_workspace_layout": (_I, [_I, _I, _I, _I, _I, _I, ctypes.POINTER(_SZ)]),
    "moe_fp4_grouped_gemm": (_I, [_P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _I, _P, _P,
                                  _SZ, _P]),
    "moe_fp4_grouped_gemm_stages": (_I, [_P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _I, _P,
                                         _P, _SZ, _I, _P]),
    "moe_fp4_grouped_gemm_noalloc": (_I, [_P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _I, _P,
                                          _P]),
    "moe_fp4_grouped_gemm_combine_supported": (_I, [_I, _I, _I, _I, _I, _I]),
    "moe_fp4_grouped_gemm_combine": (_I, [_P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _I, _P,
                                          _P, _P, _SZ, _I, _P]),
    "moe_combine_fixed_order": (_I, [_P, _P, _I, _I, _I, _P, _P]),
    "moe_status_string": (ctypes.c_char_p, [_I]),
    "moe_last_variant": (_I, []),
    "moe_probe_scaled_mfma": (_I, [_P, _P, _I, _P, _P, _P, _P]),
}


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is missing: build the HIP library first "
                          "(python -m paper_2609_15627_amd._build)")
    lib = ctypes.CDLL(_LIB_PATH)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype, fn.argtypes = res, args
    return lib


lib = _load()
LIB_PATH = _LIB_PATH


class MoeError(RuntimeError):
    def __init__(self, status, what):
        super().__init__(f"{what}: {lib.moe_status_string(status).decode()} (status {status})")
        self.status = status


def _check(status, what):
    if status != MOE_OK:
        raise MoeError(status, what)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _need(t, dtype, shape, name):
    if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous() or not t.is_cuda:
        raise ValueError(f"{name}: expected contiguous {dtype} {tuple(shape)} on the GPU, got "
                         f"{t.dtype} {tuple(t.shape)} on {t.device}")


def _u16(t):
    """bf16 tensors are passed as their bit patterns."""
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t


def moe_router_logits(x, w_router, logits=None, stream=None):
    """logits [T, E] fp32 = x [T, H] bf16 . w_router [E, H] bf16 ^T."""
    T, H = x.shape
    E = w_router.shape[0]
    _need(x, torch.bfloat16, (T, H), "x")
    _need(w_router, torch.bfloat16, (E, H), "w_router")
    if logits is None:
        logits = torch.empty((T, E), dtype=torch.float32, device=x.device)
    _need(logits, torch.float32, (T, E), "logits")
    _check(lib.moe_router_logits(_ptr(x), _ptr(w_router), T, H, E, _ptr(logits), _stream(stream)),
           "moe_router_logits")
    return logits


class _RouteOpts(ctypes.Structure):
    _fields_ = [("score", ctypes.c_int), ("bias", ctypes.c_void_p), ("n_group", ctypes.c_int),
                ("topk_group", ctypes.c_int), ("renorm", ctypes.c_int), ("scale", ctypes.c_float)]


def moe_route_topk(logits, k, n_shared=0, topk_ids=None, topk_w=None, stream=None,
                   score="softmax", bias=None, n_group=1, topk_group=1, renorm=True, scale=1.0):
    """Top-k routing. With the default options this is ``moe_route_topk``;
    otherwise ``moe_route_topk_ex`` (score "softmax" | "sigmoid", selection
    bias fp32 [E], group-limited selection, renormalisation, scaling)."""
    T, E = logits.shape
    kt = k + n_shared
    _need(logits, torch.float32, (T, E), "logits")
    if topk_ids is None:
        topk_ids = torch.empty((T, kt), dtype=torch.int32, device=logits.device)
    if topk_w is None:
        topk_w = torch.empty((T, kt), dtype=torch.float32, device=logits.device)
    _need(topk_ids, torch.int32, (T, kt), "topk_ids")
    _need(topk_w, torch.float32, (T, kt), "topk_w")
    default = (score == "softmax" and bias is None and n_group == 1 and bool(renorm)
               and scale == 1.0)
    if default:
        _check(lib.moe_route_topk(_ptr(logits), T, E, k, n_shared, _ptr(topk_ids), _ptr(topk_w),
                                  _stream(stream)), "moe_route_topk")
        return topk_ids, topk_w
    if score not in ("softmax", "sigmoid"):
        raise ValueError(f"score: {score!r}")
    if bias is not None:
        _need(bias, torch.float32, (E,), "bias")
    opts = _RouteOpts(1 if score == "sigmoid" else 0, None if bias is None else bias.data_ptr(),
                      n_group, topk_group, 1 if renorm else 0, scale)
    _check(lib.moe_route_topk_ex(_ptr(logits), T, E, k, n_shared, ctypes.byref(opts),
                                 _ptr(topk_ids), _ptr(topk_w), _stream(stream)),
           "moe_route_topk_ex")
    return topk_ids, topk_w


def moe_router_topk(x, w_router, k, n_shared=0, logits=None, topk_ids=None, topk_w=None,
                    stream=None, score="softmax", bias=None, n_group=1, topk_group=1,
                    renorm=True, scale=1.0, want_logits=False):
    """Fused router projection + routing (any E <= 1024). Returns (ids, w) or, with
    ``want_logits``, (ids, w, logits)."""
    T, H = x.shape
    E = w_router.shape[0]
    kt = k + n_shared
    _need(x, torch.bfloat16, (T, H), "x")
    _need(w_router, torch.bfloat16, (E, H), "w_router")
    if want_logits and logits is None:
        logits = torch.empty((T, E), dtype=torch.float32, device=x.device)
    if logits is not None:
        _need(logits, torch.float32, (T, E), "logits")
    if topk_ids is None:
        topk_ids = torch.empty((T, kt), dtype=torch.int32, device=x.device)
    if topk_w is None:
        topk_w = torch.empty((T, kt), dtype=torch.float32, device=x.device)
    _need(topk_ids, torch.int32, (T, kt), "topk_ids")
    _need(topk_w, torch.float32, (T, kt), "topk_w")
    if score not in ("softmax", "sigmoid"):
        raise ValueError(f"score: {score!r}")
    if bias is not None:
        _need(bias, torch.float32, (E,), "bias")
    opts = _RouteOpts(1 if score == "sigmoid" else 0, None if bias is None else bias.data_ptr(),
                      n_group, topk_group, 1 if renorm else 0, scale)
    _check(lib.moe_router_topk(_ptr(x), _ptr(w_router), T, H, E, k, n_shared,
                               ctypes.byref(opts), _ptr(logits), _ptr(topk_ids), _ptr(topk_w),
                               _stream(stream)), "moe_router_topk")
    return (topk_ids, topk_w, logits) if want_logits else (topk_ids, topk_w)


def moe_permute_workspace_bytes(T, n_experts_total, k_total):
    return lib.moe_permute_workspace_bytes(T, n_experts_total, k_total)


def moe_permute(topk_ids, n_experts_total, out=None, ws=None, stream=None):
    """Returns (counts, offsets, sorted, pos) int32 tensors."""
    T, kt = topk_ids.shape
    _need(topk_ids, torch.int32, (T, kt), "topk_ids")
    dev = topk_ids.device
    if out is None:
        out = (torch.empty(n_experts_total, dtype=torch.int32, device=dev),
               torch.empty(n_experts_total + 1, dtype=torch.int32, device=dev),
               torch.empty(T * kt, dtype=torch.int32, device=dev),
               torch.empty(T * kt, dtype=torch.int32, device=dev))
    counts, offsets, srt, pos = out
    nb = moe_permute_workspace_bytes(T, n_experts_total, kt)
    if ws is None:
        ws = torch.empty(max(nb, 256), dtype=torch.uint8, device=dev)
    _check(lib.moe_permute(_ptr(topk_ids), T, n_experts_total, kt, _ptr(counts), _ptr(offsets),
                           _ptr(srt), _ptr(pos), _ptr(ws), ws.numel(), _stream(stream)),
           "moe_permute")
    return counts, offsets, srt, pos


def act_code_bytes(K, fmt):
    """Bytes of K activation codes as moe_quantize_act packs them."""
    return K * ACT_BITS[fmt] // 8


def ws_code_bytes(K, fmt):
    """Bytes of K activation codes in the grouped GEMM's workspace (an e2m3
    block of 24 bytes sits in a 32-byte slot there)."""
    return K if fmt == "e2m3" else act_code_bytes(K, fmt)


def moe_quantize_act(x, fmt="e4m3", codes=None, scales=None, stream=None):
    rows, K = x.shape
    _need(x, torch.bfloat16, (rows, K), "x")
    if codes is None:
        codes = torch.empty((rows, act_code_bytes(K, fmt)), dtype=torch.uint8, device=x.device)
    if scales is None:
        scales = torch.empty((rows, K // 32), dtype=torch.uint8, device=x.device)
    _check(lib.moe_quantize_act(_ptr(x), rows, K, ACT_FORMATS[fmt], _ptr(codes), _ptr(scales),
                                _stream(stream)), "moe_quantize_act")
    return codes, scales


def set_tiled_rows(rows):
    """Row-tile size of the LDS-tiled geometry: 128, 256, or 0 for the
    automatic choice (``moe_set_tiled_rows``; process-wide, same bits)."""
    _check(lib.moe_set_tiled_rows(int(rows)), "moe_set_tiled_rows")


def moe_pack_fp4_weights(w, out=None, stream=None):
    """FP4 code matrix (uint8, last dimension K/2, any leading dimensions:
    e.g. W13 [NE, 2I, H/2]) into the grouped GEMM's block layout; returns a
    tensor of the same shape."""
    if w.dtype != torch.uint8 or not w.is_cuda or not w.is_contiguous():
        raise ValueError("w: contiguous uint8 tensor on the GPU expected")
    kbytes = w.shape[-1]
    rows = w.numel() // kbytes if kbytes else 0
    if out is None:
        out = torch.empty_like(w)
    elif out.shape != w.shape or out.dtype != torch.uint8 or not out.is_contiguous():
        raise ValueError("out: contiguous uint8 tensor of w's shape expected")
    _check(lib.moe_pack_fp4_weights(_ptr(w), _ptr(out), rows, 2 * kbytes, _stream(stream)),
           "moe_pack_fp4_weights")
    return out


def pack_expert_weights(weights, stream=None):
    """(w13, w13_s, w2, w2_s) with row-major codes -> the same tuple with both
    code tensors in the block layout the grouped GEMM reads (the scales are
    unchanged). Done once, when the weights are loaded."""
    w13, w13_s, w2, w2_s = weights
    return (moe_pack_fp4_weights(w13, stream=stream), w13_s,
            moe_pack_fp4_weights(w2, stream=stream), w2_s)


def moe_fp4_grouped_gemm_workspace_bytes(T, H, I, n_experts_total, k_total, fmt="e4m3"):
    return lib.moe_fp4_grouped_gemm_workspace_bytes(T, H, I, n_experts_total, k_total,
                                                    ACT_FORMATS[fmt])


def moe_fp4_grouped_gemm_workspace_layout(T, H, I, n_experts_total, k_total, fmt="e4m3"):
    arr = (_SZ * WS_REGIONS)()
    _check(lib.moe_fp4_grouped_gemm_workspace_layout(T, H, I, n_experts_total, k_total,
                                                     ACT_FORMATS[fmt], arr),
           "moe_fp4_grouped_gemm_workspace_layout")
    return list(arr)


def moe_fp4_grouped_gemm(x, offsets, sorted_, w13, w13_s, w2, w2_s, k_total, fmt="e4m3",
                         partials=None, ws=None, stream=None, stages=7):
    """stages: 7 runs the whole call; other masks call moe_fp4_grouped_gemm_stages."""
    T, H = x.shape
    NE, two_i, _ = w13.shape
    I = two_i // 2
    _need(x, torch.bfloat16, (T, H), "x")
    _need(offsets, torch.int32, (NE + 1,), "offsets")
    _need(sorted_, torch.int32, (T * k_total,), "sorted")
    _need(w13, torch.uint8, (NE, 2 * I, H // 2), "w13")
    _need(w13_s, torch.uint8, (NE, 2 * I, H // 32), "w13_s")
    _need(w2, torch.uint8, (NE, H, I // 2), "w2")
    _need(w2_s, torch.uint8, (NE, H, I // 32), "w2_s")
    if partials is None:
        partials = torch.empty((T * k_total, H), dtype=torch.float32, device=x.device)
    _need(partials, torch.float32, (T * k_total, H), "partials")
    if ws is None:
        ws = torch.empty(max(moe_fp4_grouped_gemm_workspace_bytes(T, H, I, NE, k_total, fmt), 256),
                         dtype=torch.uint8, device=x.device)
    args = (_ptr(x), T, H, I, NE, k_total, _ptr(offsets), _ptr(sorted_), _ptr(w13), _ptr(w13_s),
            _ptr(w2), _ptr(w2_s), ACT_FORMATS[fmt], _ptr(partials), _ptr(ws), ws.numel())
    if stages == 7:
        _check(lib.moe_fp4_grouped_gemm(*args, _stream(stream)), "moe_fp4_grouped_gemm")
    else:
        _check(lib.moe_fp4_grouped_gemm_stages(*args, stages, _stream(stream)),
               "moe_fp4_grouped_gemm_stages")
    return partials


NOALLOC_SCRATCH_BYTES = 32 << 20  # MOE_NOALLOC_SCRATCH_BYTES


def moe_fp4_grouped_gemm_noalloc(x, offsets, sorted_, w13, w13_s, w2, w2_s, k_total, partials,
                                 fmt="e4m3", stream=None):
    """moe_fp4_grouped_gemm with the library's static scratch as its workspace:
    nothing is allocated (``partials`` must be given)."""
    T, H = x.shape
    NE, two_i, _ = w13.shape
    I = two_i // 2
    _need(x, torch.bfloat16, (T, H), "x")
    _need(offsets, torch.int32, (NE + 1,), "offsets")
    _need(sorted_, torch.int32, (T * k_total,), "sorted")
    _need(w13, torch.uint8, (NE, 2 * I, H // 2), "w13")
    _need(w13_s, torch.uint8, (NE, 2 * I, H // 32), "w13_s")
    _need(w2, torch.uint8, (NE, H, I // 2), "w2")
    _need(w2_s, torch.uint8, (NE, H, I // 32), "w2_s")
    _need(partials, torch.float32, (T * k_total, H), "partials")
    _check(lib.moe_fp4_grouped_gemm_noalloc(
        _ptr(x), T, H, I, NE, k_total, _ptr(offsets), _ptr(sorted_), _ptr(w13), _ptr(w13_s),
        _ptr(w2), _ptr(w2_s), ACT_FORMATS[fmt], _ptr(partials), _stream(stream)),
        "moe_fp4_grouped_gemm_noalloc")
    return partials


def moe_fp4_grouped_gemm_combine_supported(T, H, I, n_experts_total, k_total, fmt="e4m3"):
    """True when the down projection can run fused with the combine."""
    return bool(lib.moe_fp4_grouped_gemm_combine_supported(T, H, I, n_experts_total, k_total,
                                                           ACT_FORMATS[fmt]))


def moe_fp4_grouped_gemm_combine(x, offsets, sorted_, w13, w13_s, w2, w2_s, topk_w, fmt="e4m3",
                                 out=None, ws=None, stream=None, stages=7):
    """The grouped GEMM with its down projection fused with the fixed-order
    combine: writes out [T, H] bf16 directly (bit-identical to
    moe_fp4_grouped_gemm + moe_combine_fixed_order)."""
    T, H = x.shape
    NE, two_i, _ = w13.shape
    I = two_i // 2
    k_total = topk_w.shape[1]
    _need(x, torch.bfloat16, (T, H), "x")
    _need(offsets, torch.int32, (NE + 1,), "offsets")
    _need(sorted_, torch.int32, (T * k_total,), "sorted")
    _need(w13, torch.uint8, (NE, 2 * I, H // 2), "w13")
    _need(w13_s, torch.uint8, (NE, 2 * I, H // 32), "w13_s")
    _need(w2, torch.uint8, (NE, H, I // 2), "w2")
    _need(w2_s, torch.uint8, (NE, H, I // 32), "w2_s")
    _need(topk_w, torch.float32, (T, k_total), "topk_w")
    if out is None:
        out = torch.empty((T, H), dtype=torch.bfloat16, device=x.device)
    _need(out, torch.bfloat16, (T, H), "out")
    if ws is None:
        ws = torch.empty(max(moe_fp4_grouped_gemm_workspace_bytes(T, H, I, NE, k_total, fmt), 256),
                         dtype=torch.uint8, device=x.device)
    _check(lib.moe_fp4_grouped_gemm_combine(
        _ptr(x), T, H, I, NE, k_total, _ptr(offsets), _ptr(sorted_), _ptr(w13), _ptr(w13_s),
        _ptr(w2), _ptr(w2_s), ACT_FORMATS[fmt], _ptr(topk_w), _ptr(out), _ptr(ws), ws.numel(),
        stages, _stream(stream)), "moe_fp4_grouped_gemm_combine")
    return out


def moe_combine_fixed_order(partials, topk_w, out=None, stream=None):
    T, kt = topk_w.shape
    H = partials.shape[1]
    _need(partials, torch.float32, (T * kt, H), "partials")
    _need(topk_w, torch.float32, (T, kt), "topk_w")
    if out is None:
        out = torch.empty((T, H), dtype=torch.bfloat16, device=partials.device)
    _need(out, torch.bfloat16, (T, H), "out")
    _check(lib.moe_combine_fixed_order(_ptr(partials), _ptr(topk_w), T, H, kt, _ptr(out),
                                       _stream(stream)), "moe_combine_fixed_order")
    return out


def moe_last_variant():
    return lib.moe_last_variant()


def moe_probe_scaled_mfma(a, sa, b, sb, fmt="e4m3", d=None, stream=None):
    if d is None:
        d = torch.empty((16, 16), dtype=torch.float32, device=a.device)
    _check(lib.moe_probe_scaled_mfma(_ptr(a), _ptr(sa), ACT_FORMATS[fmt], _ptr(b), _ptr(sb),
                                     _ptr(d), _stream(stream)), "moe_probe_scaled_mfma")
    return d


class MoELayer:
    """One routed-MoE layer forward through the four library calls.

    Owns the intermediate buffers and workspaces (torch allocations made once
    at construction); ``forward`` enqueues only library kernels.
    """

    def __init__(self, T, H, E, k, I, n_shared=0, fmt="e4m3", device="cuda", fused=False):
        """fused: run the down projection fused with the combine (same bits
        as the two calls; raises MoeError when the dims do not allow it).
        None picks it whenever the library supports the dims. Off by default:
        at decode size the two-kernel path measured faster."""
        self.T, self.H, self.E, self.k, self.I, self.S = T, H, E, k, I, n_shared
        self.NE, self.kt = E + n_shared, k + n_shared
        self.fmt = fmt
        ok = moe_fp4_grouped_gemm_combine_supported(T, H, I, self.NE, self.kt, fmt)
        if fused and not ok:
            raise MoeError(MOE_ERR_UNSUPPORTED, "fused down + combine for these dims")
        self.fused = ok if fused is None else bool(fused)
        dev = torch.device(device)
        A = T * self.kt
        self.logits = torch.empty((T, E), dtype=torch.float32, device=dev)
        self.ids = torch.empty((T, self.kt), dtype=torch.int32, device=dev)
        self.w = torch.empty((T, self.kt), dtype=torch.float32, device=dev)
        self.perm = (torch.empty(self.NE, dtype=torch.int32, device=dev),
                     torch.empty(self.NE + 1, dtype=torch.int32, device=dev),
                     torch.empty(A, dtype=torch.int32, device=dev),
                     torch.empty(A, dtype=torch.int32, device=dev))
        self.perm_ws = torch.empty(max(moe_permute_workspace_bytes(T, self.NE, self.kt), 256),
                                   dtype=torch.uint8, device=dev)
        self.partials = None if self.fused else torch.empty((A, H), dtype=torch.float32, device=dev)
        self.gemm_ws = torch.empty(
            max(moe_fp4_grouped_gemm_workspace_bytes(T, H, I, self.NE, self.kt, fmt), 256),
            dtype=torch.uint8, device=dev)
        self.out = torch.empty((T, H), dtype=torch.bfloat16, device=dev)

    def workspace_view(self, region):
        """uint8 view of a grouped-GEMM workspace region (0..3, see include/moe.h)."""
        off = moe_fp4_grouped_gemm_workspace_layout(self.T, self.H, self.I, self.NE, self.kt,
                                                    self.fmt)
        return self.gemm_ws[off[region]:off[region + 1]]

    def forward(self, x, weights, logits=None, w_router=None, stream=None, events=None):
        """Enqueue the layer. ``weights``: (w13, w13_s, w2, w2_s) with the codes in
        the block layout (``pack_expert_weights``). ``events``: optional list of 7 torch.cuda.Event
        recorded between the steps (route, permute, quantise, gate/up, down,
        combine) for per-step timing; with the fused path "down" is the fused
        down projection + combine and "combine" is empty."""
        w13, w13_s, w2, w2_s = weights
        ev = (lambda i: events[i].record(stream)) if events else (lambda i: None)
        ev(0)
        if logits is None:
            logits = moe_router_logits(x, w_router, self.logits, stream=stream)
        moe_route_topk(logits, self.k, self.S, self.ids, self.w, stream=stream)
        ev(1)
        counts, offsets, srt, pos = moe_permute(self.ids, self.NE, out=self.perm, ws=self.perm_ws,
                                                stream=stream)
        ev(2)
        if self.fused:
            g = (x, offsets, srt, w13, w13_s, w2, w2_s, self.w, self.fmt)
            if events:
                for i, st in enumerate((1, 2, 4)):
                    moe_fp4_grouped_gemm_combine(*g, out=self.out, ws=self.gemm_ws, stream=stream,
                                                 stages=st)
                    ev(3 + i)
            else:
                moe_fp4_grouped_gemm_combine(*g, out=self.out, ws=self.gemm_ws, stream=stream)
            ev(6)
            return self.out
        g = (x, offsets, srt, w13, w13_s, w2, w2_s, self.kt, self.fmt)
        if events:
            for i, st in enumerate((1, 2, 4)):
                moe_fp4_grouped_gemm(*g, partials=self.partials, ws=self.gemm_ws, stream=stream,
                                     stages=st)
                ev(3 + i)
        else:
            moe_fp4_grouped_gemm(*g, partials=self.partials, ws=self.gemm_ws, stream=stream)
        out = moe_combine_fixed_order(self.partials, self.w, out=self.out, stream=stream)
        ev(6)
        return out

    def capture(self, x, weights, logits=None, w_router=None):
        """Record one ``forward`` into a HIP graph, so that a decode step is one
        graph launch instead of six kernel launches. The graph reads x, the
        weights and the logits from the tensors given here (copy new inputs
        into them before a replay) and writes ``self.out``. Every kernel of
        the layer clears what it needs itself (no memset nodes) and the
        persistent GEMM's work queue is left at zero by each launch, so
        replays are independent."""
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):  # first call outside the graph: lazy host state
            self.forward(x, weights, logits=logits, w_router=w_router)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            self.forward(x, weights, logits=logits, w_router=w_router)
        return self.out

    def replay(self):
        """Re-run the captured forward on the current stream; returns ``self.out``."""
        self.graph.replay()
        return self.out
