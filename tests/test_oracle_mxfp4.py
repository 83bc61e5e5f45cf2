"""Pins for MXFP4 routed-expert weights (OCP Microscaling formats v1.0: FP4 E2M1 elements,
one E8M0 power-of-two scale per 32 consecutive elements of a row), the quantised variant
of the expert weights (the paper runs Qwen2-57B-A14B with 5-bit k-quant weights; its
format is not given, so this library uses the MI355X-native MX format).

References: the E2M1 and E8M0 value tables of the MX specification written out as
numbers, blobs packed here from matrices whose values are known exactly, torch fp64
for the SwiGLU and the dense MoE on those known matrices, and quantiser round trips,
midpoints and saturation worked by hand.
"""
import numpy as np
import pytest
import torch

from paper_2608_21240_amd import synth, workloads as W
from test_oracle_layer import f64, t_swiglu

# the sixteen E2M1 codes by value, from the MX specification's element table
E2M1_VALUES = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0, -0.0, -0.5, -1.0, -1.5, -2.0, -3.0, -4.0, -6.0]


def pack(codes, scales):
    """codes [rows][K] (0..15), scales [rows][K/32] (E8M0 bytes) -> blob (low nibble first)."""
    codes = np.asarray(codes, np.uint8)
    packed = codes[:, 0::2] | (codes[:, 1::2] << 4)
    return np.concatenate([packed.reshape(-1), np.asarray(scales, np.uint8).reshape(-1)]).astype(np.uint8)


def known_matrix(rng, rows, K, lo=-6, hi=2):
    """A random matrix of MXFP4-representable values with its codes and scales."""
    codes = rng.integers(0, 16, size=(rows, K))
    ex = rng.integers(lo, hi, size=(rows, K // 32))
    vals = np.array(E2M1_VALUES)[codes] * np.ldexp(1.0, np.repeat(ex, 32, axis=1))
    return vals, pack(codes, ex + 127)


def test_element_table_and_scales(orc):
    rows, K = 2, 64
    codes = np.tile(np.arange(16), (rows, K // 16))
    for s, mult in ((127, 1.0), (130, 8.0), (120, 2.0 ** -7), (0, 2.0 ** -127)):
        blob = pack(codes, np.full((rows, K // 32), s))
        for c in range(16):
            v = orc.mxfp4_elem(blob, rows, K, 1, c)
            assert v == E2M1_VALUES[c] * mult, (s, c, v)
    nan_blob = pack(codes, np.full((rows, K // 32), 255))
    assert np.isnan(orc.mxfp4_elem(nan_blob, rows, K, 0, 3))


def test_nibble_order_and_scale_per_block(orc):
    rows, K = 1, 64
    codes = np.zeros((rows, K), np.int64)
    codes[0, 0], codes[0, 1], codes[0, 33] = 2, 7, 5  # 1.0 (low nibble), 6.0 (high nibble), 3.0
    blob = pack(codes, [[127, 129]])  # scales 1 and 4
    assert blob[0] == 0x72
    assert orc.mxfp4_elem(blob, rows, K, 0, 0) == 1.0
    assert orc.mxfp4_elem(blob, rows, K, 0, 1) == 6.0
    assert orc.mxfp4_elem(blob, rows, K, 0, 33) == 12.0
    assert orc.mxfp4_elem(blob, rows, K, 0, 32) == 0.0


def test_quantizer_round_trip_of_representable_values():
    # every block leads with 6.0 (code 7) so the quantiser picks the exponent the matrix
    # was built with; the other codes are random
    r = np.random.default_rng(1)
    codes = r.integers(0, 16, size=(6, 96)); codes[:, ::32] = 7
    ex = r.integers(-6, 2, size=(6, 3))
    vals = np.array(E2M1_VALUES)[codes] * np.ldexp(1.0, np.repeat(ex, 32, axis=1))
    q = synth.quantize_mxfp4(vals.astype(np.float32))
    # -0 codes (8) come back as +0 (code 0): compare values, then bytes where no -0 occurs
    back = np.array([[float(np.array(E2M1_VALUES)[c]) for c in row] for row in codes])
    exp_codes = np.where(codes == 8, 0, codes)
    assert np.array_equal(q, pack(exp_codes, ex + 127))
    assert np.allclose(back * np.ldexp(1.0, np.repeat(ex, 32, axis=1)), vals)


def test_quantizer_rounding_and_saturation():
    # one block with max 6 (exponent 0): midpoints go to the even code, beyond 6 saturates
    x = np.zeros((1, 32), np.float32)
    x[0, :10] = [6.0, 0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, -2.6, 0.2]
    q = synth.quantize_mxfp4(x)
    codes = np.empty(32, np.int64)
    codes[0::2], codes[1::2] = q[:16] & 15, q[:16] >> 4
    assert q[16] == 127  # 2^0
    # 6 -> 7; 0.25 -> 0 (codes 0|1, even 0); 0.75 -> 1.0 (codes 1|2 -> 2); 1.25 -> 1.0 (2|3 -> 2);
    # 1.75 -> 2.0 (3|4 -> 4); 2.5 -> 2.0 (4|5 -> 4); 3.5 -> 4.0 (5|6 -> 6); 5.0 -> 4.0 (6|7 -> 6);
    # -2.6 -> -3.0 (code 13); 0.2 -> 0
    assert codes[:10].tolist() == [7, 0, 2, 2, 4, 4, 6, 6, 13, 0]
    # the shared exponent: block max 13 -> floor(log2 13) - 2 = 1, so 13 / 2 = 6.5 saturates to 6
    y = np.zeros((1, 32), np.float32)
    y[0, 0], y[0, 1] = 13.0, -1.0
    qy = synth.quantize_mxfp4(y)
    assert qy[16] == 128 and (qy[0] & 15) == 7 and (qy[0] >> 4) == 9  # 6 * 2 = 12, -0.5 * 2 = -1


def test_mxfp4_swiglu_matches_torch_on_known_weights(orc):
    r = np.random.default_rng(2)
    d, I = 64, 32
    w13, b13 = known_matrix(r, 2 * I, d)
    w2, b2 = known_matrix(r, d, I)
    x = r.standard_normal(d)
    y = orc.swiglu(d, I, orc.MXFP4, b13, b2, x)
    ref = t_swiglu(torch.from_numpy(x[None]), torch.from_numpy(w13), torch.from_numpy(w2), I)[0].numpy()
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-14)


def test_all_resident_mxfp4_layer_is_the_dense_moe(orc):
    # bf16 activations, router and shared block; MXFP4 routed experts with known values
    r = np.random.default_rng(3)
    d, N, K, I, Is, T = 64, 6, 2, 32, 32, 5
    shape = W.MoEShape(d=d, n_experts=N, top_k=K, inter=I, shared_inter=Is, lore_rank=4, dtype=W.DTYPE_BF16)
    bf = lambda a: synth.to_storage(a.astype(np.float32), W.DTYPE_BF16)
    x = bf(r.standard_normal((T, d)))
    wg = bf(r.standard_normal((N, d)) * 0.3)
    w13s, w2s = bf(r.standard_normal((2 * Is, d)) * 0.2), bf(r.standard_normal((d, Is)) * 0.2)
    mats = [(known_matrix(r, 2 * I, d), known_matrix(r, d, I)) for _ in range(N)]
    w13 = [m[0][1] for m in mats]; w2 = [m[1][1] for m in mats]
    lA = [bf(r.standard_normal((4, d)) * 0.1) for _ in range(N)]
    lB = [bf(r.standard_normal((d, 4)) * 0.1) for _ in range(N)]
    cfg = orc.make_cfg(shape, wfmt=orc.MXFP4)
    res = orc.layer(cfg, x, wg, None, np.ones(N, np.int32), r.random((T, K)).astype(np.float32), w13, w2, w13s, w2s,
                    lA, lB)
    xt = f64(x, W.DTYPE_BF16)
    ref = t_swiglu(xt, f64(w13s, W.DTYPE_BF16), f64(w2s, W.DTYPE_BF16), Is)
    for t in range(T):
        for k in range(K):
            e = int(res["idx"][t, k])
            ref[t] += float(res["g"][t, k]) * t_swiglu(xt[t:t + 1], torch.from_numpy(mats[e][0][0]),
                                                       torch.from_numpy(mats[e][1][0]), I)[0]
    assert np.allclose(res["out"], ref.numpy(), rtol=1e-11, atol=1e-12)
    # the exact CPU path reads the same MXFP4 weights
    cls = np.full((T, K), 2, np.uint8)
    resid = orc.exact_residual(cfg, x, res["idx"], res["g"], cls, w13, w2)
    assert np.allclose(resid + res["y_shared"], ref.numpy(), rtol=1e-11, atol=1e-12)
