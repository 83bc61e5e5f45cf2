"""Seeded synthetic inputs for the MoE-layer workloads.

This module only draws random numbers and rounds them to the storage type; it
holds none of the method's arithmetic, so both the oracle tests and the HIP
path may take their inputs from it.

Every tensor has its own NumPy PCG64 stream keyed by
(seed, workload id, layer, tensor id, index), so one expert's weights can be
drawn without drawing the others.

Recipe (stand-in for the paper's real model weights and datasets, which are
not available): weights ~ N(0, 0.02); hidden states ~ N(0, 1); per-slot
confidence ~ U(0, 1); expert popularity p_k proportional to k^-1.1 over a
seeded permutation of the experts; residency = the R most popular experts
(the tiny layer: the first R of a seeded permutation); routing skew, where
enabled, is a logit bias ln p_e. bf16 tensors are drawn in fp32 and rounded to
bf16 with round-to-nearest-even; both sides see the identical bf16 values.
"""
from __future__ import annotations

import zlib
from typing import List, Optional, Tuple

import numpy as np

from .workloads import DTYPE_BF16, DTYPE_F32, WFMT_MXFP4, Workload

WEIGHT_STD = 0.02

T_X, T_WG, T_POP, T_CONF, T_W13, T_W2, T_W13S, T_W2S, T_LA, T_LB, T_RES, T_SG = range(1, 13)


def _wid(wl: Workload) -> int:
    # Shape-level identity so that e.g. the three DSV2 decode batch sizes share weights.
    s = wl.shape
    return zlib.crc32(repr((s.d, s.n_experts, s.top_k, s.inter, s.shared_inter, s.lore_rank, s.dtype)).encode())


def rng(*key: int) -> np.random.Generator:
    return np.random.default_rng([int(k) & 0xFFFFFFFF for k in key])


def f32_to_bf16_bits(a: np.ndarray, overwrite: bool = False) -> np.ndarray:
    """Round fp32 to bf16 (round to nearest, ties to even); returns uint16 bits.
    overwrite=True lets the (float32, contiguous) input serve as scratch."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32) if overwrite else a.view(np.uint32).copy()
    bias = u >> np.uint32(16)
    bias &= np.uint32(1)
    bias += np.uint32(0x7FFF)
    u += bias
    u >>= np.uint32(16)
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def to_storage(a32: np.ndarray, dtype: int, overwrite: bool = False) -> np.ndarray:
    """fp32 draw -> storage array (float32, or uint16 bf16 bits)."""
    if dtype == DTYPE_BF16:
        return f32_to_bf16_bits(a32, overwrite=overwrite)
    return np.ascontiguousarray(a32, dtype=np.float32)


def as_f32(a: np.ndarray, dtype: int) -> np.ndarray:
    """Storage array -> float32 values (exact)."""
    return bf16_bits_to_f32(a) if dtype == DTYPE_BF16 else np.asarray(a, dtype=np.float32)


def _normal(key: Tuple[int, ...], shape, std: float, dtype: int) -> np.ndarray:
    a = rng(*key).standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return to_storage(a, dtype, overwrite=True)


def _key(wl: Workload, layer: int, tensor: int, index: int = 0) -> Tuple[int, ...]:
    return (wl.seed, _wid(wl), layer, tensor, index)


def gen_x(wl: Workload, layer: int = 0, step: int = 0, tokens: Optional[int] = None) -> np.ndarray:
    """Hidden states x[T][d] ~ N(0, 1)."""
    T = wl.tokens if tokens is None else tokens
    return _normal((wl.seed, _wid(wl), layer, T_X, step, T), (T, wl.shape.d), 1.0, wl.shape.dtype)


def gen_router(wl: Workload, layer: int = 0) -> np.ndarray:
    """Router weight W_g[N][d] ~ N(0, 0.02)."""
    s = wl.shape
    return _normal(_key(wl, layer, T_WG), (s.n_experts, s.d), WEIGHT_STD, s.dtype)


def popularity(wl: Workload, layer: int = 0) -> np.ndarray:
    """Zipf(s) popularity p[e]: rank k (1-based) has weight k^-s; ranks are
    assigned to experts by a seeded permutation."""
    N = wl.shape.n_experts
    order = rng(*_key(wl, layer, T_POP)).permutation(N)  # order[k-1] = expert of rank k
    w = np.arange(1, N + 1, dtype=np.float64) ** (-wl.zipf_s)
    w /= w.sum()
    p = np.empty(N, dtype=np.float64)
    p[order] = w
    return p


def gen_bias(wl: Workload, layer: int = 0) -> Optional[np.ndarray]:
    """Routing-skew logit bias b_e = ln p_e (fp32), or None when disabled."""
    if not wl.skew:
        return None
    return np.log(popularity(wl, layer)).astype(np.float32)


def resident_experts(wl: Workload, layer: int = 0) -> List[int]:
    """Ids of the R experts resident in the GPU cache (ascending)."""
    N, R = wl.shape.n_experts, wl.resident
    if R >= N:
        return list(range(N))
    if wl.shape.dtype == DTYPE_F32 and N <= 8:
        sel = rng(*_key(wl, layer, T_RES)).permutation(N)[:R]
    else:
        p = popularity(wl, layer)
        sel = np.argsort(-p, kind="stable")[:R]
    return sorted(int(e) for e in sel)


def gen_conf(wl: Workload, layer: int = 0, step: int = 0, tokens: Optional[int] = None) -> np.ndarray:
    """Per-slot routing confidence conf[T][K] ~ U(0, 1), fp32."""
    T = wl.tokens if tokens is None else tokens
    return rng(wl.seed, _wid(wl), layer, T_CONF, step, T).random((T, wl.shape.top_k), dtype=np.float32)


# FP4 E2M1 magnitudes by code 0..7 (OCP Microscaling formats v1.0); the sign is bit 3.
E2M1_MAGNITUDES = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def quantize_mxfp4(a: np.ndarray) -> np.ndarray:
    """A [rows][K] fp32 matrix (K a multiple of 32) -> one MXFP4 byte blob: rows*K/2 bytes of
    E2M1 codes (element 2i in the low nibble of byte i), then rows*K/32 E8M0 block scales.

    Per block of 32 the shared exponent is floor(log2(max |a|)) - 2 (2 = the largest E2M1
    exponent); elements a / 2^exponent go to the nearest E2M1 value, ties to the even code,
    saturating at 6.  An all-zero block gets scale 2^0."""
    rows, K = a.shape
    assert K % 32 == 0
    blk = np.asarray(a, np.float64).reshape(rows, K // 32, 32)
    amax = np.abs(blk).max(axis=2)
    ex = np.zeros(amax.shape, np.int64)
    nz = amax > 0
    ex[nz] = np.floor(np.log2(amax[nz])).astype(np.int64) - 2
    ex = np.clip(ex, -127, 127)
    q = (np.abs(blk) / np.ldexp(1.0, ex)[:, :, None]).reshape(-1)
    mids = (E2M1_MAGNITUDES[1:] + E2M1_MAGNITUDES[:-1]) / 2  # decision points between codes
    code = np.searchsorted(mids, q, side="left")  # q at a midpoint takes the lower code here
    at_mid = (code < 7) & (q == mids[np.minimum(code, 6)])
    code = np.where(at_mid & (code % 2 == 1), code + 1, code)  # ties to the even code
    sign = (blk.reshape(-1) < 0) & (code > 0)
    codes = (code | np.where(sign, 8, 0)).astype(np.uint8).reshape(rows, K)
    packed = (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)
    scales = (ex + 127).astype(np.uint8)
    return np.concatenate([packed.reshape(-1), scales.reshape(-1)])


def mxfp4_bytes(rows: int, K: int) -> int:
    return rows * K // 2 + rows * K // 32


def gen_expert(wl: Workload, layer: int, e: int) -> Tuple[np.ndarray, np.ndarray]:
    """Routed expert e: w13[2I][d] (rows 0..I-1 gate W1, rows I..2I-1 up W3), w2[d][I] in the
    storage dtype, or as MXFP4 blobs (quantize_mxfp4 of the same draws) when wl.wfmt is MXFP4."""
    s = wl.shape
    if wl.wfmt == WFMT_MXFP4:
        w13 = rng(*_key(wl, layer, T_W13, e)).standard_normal(size=(2 * s.inter, s.d), dtype=np.float32)
        w2 = rng(*_key(wl, layer, T_W2, e)).standard_normal(size=(s.d, s.inter), dtype=np.float32)
        return quantize_mxfp4(w13 * np.float32(WEIGHT_STD)), quantize_mxfp4(w2 * np.float32(WEIGHT_STD))
    w13 = _normal(_key(wl, layer, T_W13, e), (2 * s.inter, s.d), WEIGHT_STD, s.dtype)
    w2 = _normal(_key(wl, layer, T_W2, e), (s.d, s.inter), WEIGHT_STD, s.dtype)
    return w13, w2


def gen_shared(wl: Workload, layer: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """Shared block: w13s[2 I_s][d], w2s[d][I_s]."""
    s = wl.shape
    w13 = _normal(_key(wl, layer, T_W13S), (2 * s.shared_inter, s.d), WEIGHT_STD, s.dtype)
    w2 = _normal(_key(wl, layer, T_W2S), (s.d, s.shared_inter), WEIGHT_STD, s.dtype)
    return w13, w2


def gen_shared_gate(wl: Workload, layer: int = 0) -> Optional[np.ndarray]:
    """Gate row w_sg[d] ~ N(0, 0.02) of a gated shared block, or None when ungated."""
    if not wl.shared_gate:
        return None
    return _normal(_key(wl, layer, T_SG), (wl.shape.d,), WEIGHT_STD, wl.shape.dtype)


def gen_lore(wl: Workload, layer: int, e: int) -> Tuple[np.ndarray, np.ndarray]:
    """LoRE factors of expert e: A[r][d], B[d][r] ~ N(0, 0.02)."""
    s = wl.shape
    A = _normal(_key(wl, layer, T_LA, e), (s.lore_rank, s.d), WEIGHT_STD, s.dtype)
    B = _normal(_key(wl, layer, T_LB, e), (s.d, s.lore_rank), WEIGHT_STD, s.dtype)
    return A, B
