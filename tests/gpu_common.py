"""Shared helpers of the GPU parity tests: upload seeded inputs, run the
library's layer forward, compare with the oracle."""
from __future__ import annotations

import functools
import sys

import numpy as np
import torch

import synth


def log(msg):
    """Name the case on stdout before each GPU step (flushed)."""
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


def to_dev_u8(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def to_dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def bf16_bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def bf16_to_f64(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def pack_fp4_ref(w):
    """The block layout of moe_pack_fp4_weights written out in numpy: a
    [rows, K/2] code matrix as groups of 16 rows, each group's bytes ordered
    by 64-byte K piece, then row, then byte."""
    w = np.ascontiguousarray(w, np.uint8)
    rows, kb = w.shape
    return w.reshape(rows // 16, 16, kb // 64, 64).transpose(0, 2, 1, 3).reshape(rows, kb)


def dev_expert_weights(ws):
    """Row-major numpy (w13, w13_s, w2, w2_s) -> device tensors with the codes
    in the grouped GEMM's block layout (moe_pack_fp4_weights; scales as they
    are)."""
    from paper_2609_15627_amd import moe
    return moe.pack_expert_weights(tuple(to_dev_u8(a) for a in ws))


@functools.lru_cache(maxsize=2)
def _stacked_weights(H, I, NE, seed):
    cfg = synth.LayerConfig("w", 1, H, NE, 1, I, 0, "normal", seed)
    return synth.gen_all_experts(cfg)


@functools.lru_cache(maxsize=1)
def _dev_weights(H, I, NE, seed):
    return dev_expert_weights(_stacked_weights(H, I, NE, seed))


def drop_caches():
    _dev_weights.cache_clear()
    _stacked_weights.cache_clear()
    torch.cuda.empty_cache()


def dev_weights(cfg, share=True):
    """Device weights of a config (codes in the block layout). Routed experts
    depend only on (H, I, e, seed), so configs with equal dims share one
    upload (the shared expert is index E); a block-layout tensor sliced to
    its first NE experts is the block layout of those experts."""
    if not share:
        return dev_expert_weights(synth.gen_all_experts(cfg))
    ne_max = 257 if (cfg.H, cfg.I) == (4096, 2048) else cfg.NE
    full = _dev_weights(cfg.H, cfg.I, ne_max, cfg.seed)
    if cfg.NE == ne_max:
        return full
    return tuple(a[:cfg.NE] for a in full)


def ws_codes(b, fmt):
    """Workspace activation code bytes [rows, n] -> one code per element: e2m1
    packs two per byte (low nibble first); e2m3 holds each 32-element block's
    24 bytes (code j at bits 6j) in a 32-byte slot; e4m3 one per byte."""
    b = np.asarray(b, np.uint8)
    if fmt == "e4m3":
        return b
    if fmt == "e2m1":
        out = np.empty(b.shape[:-1] + (2 * b.shape[-1],), np.uint8)
        out[..., 0::2], out[..., 1::2] = b & 15, b >> 4
        return out
    slots = b.reshape(b.shape[0], -1, 32)[:, :, :24]
    bits = np.unpackbits(slots, axis=-1, bitorder="little").reshape(b.shape[0], -1, 32, 6)
    return (bits * (1 << np.arange(6))).sum(-1).reshape(b.shape[0], -1).astype(np.uint8)


def rowrel(y, ref):
    """max over rows of max|y - ref| / max|ref| (row-wise infinity-norm relative error)."""
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.abs(ref).max(axis=1)
    den = np.where(den == 0, 1.0, den)
    return float((np.abs(y - ref).max(axis=1) / den).max())


def metrics(y, ref):
    """The paper's kernel-level metrics: max abs error, relative L2, cosine."""
    y = np.asarray(y, np.float64).ravel()
    ref = np.asarray(ref, np.float64).ravel()
    d = y - ref
    return dict(max_abs=float(np.abs(d).max()), rel_l2=float(np.linalg.norm(d) / np.linalg.norm(ref)),
                cosine=float(y @ ref / (np.linalg.norm(y) * np.linalg.norm(ref))),
                rowrel=rowrel(y.reshape(1, -1), ref.reshape(1, -1)))
