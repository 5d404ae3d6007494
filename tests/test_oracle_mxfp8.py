"""Pins of the oracle's MX-FP8 dispatch payload (Section 1, the precision
lever on b_x in Eq. 1): E4M3 element encoding, the E8M0 block scale, the
block quantiser and the dispatch of encoded rows.  CPU only."""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O


def _torch_e4m3(v):
    """The library's fp32 -> float8_e4m3fn conversion (round to nearest even)."""
    return torch.as_tensor(np.asarray(v, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_encode_matches_library_on_every_code_and_midpoint():
    pos = np.arange(0x7F, dtype=np.uint8)                  # 0x00 .. 0x7E: every finite magnitude
    vals = O.e4m3_decode(pos)
    # the library decodes every finite code to the same value
    lib = torch.as_tensor(pos).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    np.testing.assert_array_equal(vals, lib)
    mids = (vals[:-1] + vals[1:]) / 2                      # exact ties between neighbours
    for v in (vals, -vals, mids, -mids, np.nextafter(mids, 0), np.nextafter(mids, 1e9)):
        v = v.astype(np.float32).astype(np.float64)        # values the library sees
        np.testing.assert_array_equal(O.e4m3_encode(v), _torch_e4m3(v))


def test_encode_matches_library_on_random_values():
    rng = np.random.default_rng(0)
    v = np.concatenate([rng.normal(size=20000) * 50, rng.normal(size=20000) * 1e-2,
                        rng.uniform(-464, 464, 20000)]).astype(np.float32).astype(np.float64)
    np.testing.assert_array_equal(O.e4m3_encode(v), _torch_e4m3(v))


def test_encode_handworked_codes_and_saturation():
    # OCP 8-bit floating point, E4M3: S.EEEE.MMM, bias 7
    table = [(448.0, 0x7E), (-448.0, 0xFE), (1.0, 0x38), (-2.0, 0xC0), (0.5, 0x30), (2.0 ** -6, 0x08),
             (2.0 ** -9, 0x01), (7 * 2.0 ** -9, 0x07), (256.0, 0x78), (240.0, 0x77), (0.0, 0x00),
             (-0.0, 0x80), (1.0625, 0x38), (1.1875, 0x3A), (2.0 ** -10, 0x00), (1.5 * 2.0 ** -10, 0x01)]
    for v, c in table:
        assert int(O.e4m3_encode(np.array([v]))[0]) == c, v
    # beyond the largest finite value: saturate (the library would give NaN)
    np.testing.assert_array_equal(O.e4m3_encode([465.0, 511.9, 1e30, -600.0]), [0x7E, 0x7E, 0x7E, 0xFE])
    with pytest.raises(ValueError):
        O.e4m3_encode([np.inf])
    with pytest.raises(ValueError):
        O.e4m3_decode([0x7F])


def test_decode_encode_round_trip_all_codes():
    codes = np.array([c for c in range(256) if c & 0x7F != 0x7F], np.uint8)
    assert codes.size == 254
    np.testing.assert_array_equal(O.e4m3_encode(O.e4m3_decode(codes)), codes)
    v = O.e4m3_decode(codes[codes < 0x80])
    assert np.all(np.diff(v) > 0)                          # codes ordered like their values
    assert v.max() == 448.0 and v[1] == 2.0 ** -9


def test_shared_exponent_closed_forms():
    amax = np.array([1.0, 1.9, 2.0, 448.0, 511.0, 512.0, 2.0 ** -6, 3.0e38, 0.0, 2.0 ** -130])
    want = [-8, -8, -7, 0, 0, 1, -14, 127 - 8, -127, -127]
    np.testing.assert_array_equal(O.mx_shared_exponent(amax), want)


def _bound(x, X):
    """Per-element error bound of one MX-FP8 element at scale X: half an E4M3
    ulp (2^-4 relative in the normal range, 2^-10 X below it) or the clip to
    448 X for the block maximum."""
    a = np.abs(x)
    return np.maximum(np.maximum(2.0 ** -4 * a, 2.0 ** -10 * X), a - 448 * X)


def test_quantize_error_bound_and_maximum():
    rng = np.random.default_rng(1)
    x = O.round_bf16(rng.normal(size=(64, 256)) * np.exp(rng.normal(size=(64, 1)) * 4))
    codes, scales = O.mxfp8_quantize(x)
    deq = O.mxfp8_dequantize(codes, scales)
    X = np.repeat(np.ldexp(1.0, scales.astype(np.int64) - 127), 32, axis=1)
    assert np.all(np.abs(deq - x) <= _bound(x, X))
    # the block maximum lands in [256, 512) before rounding: its code's exponent field is 15
    blk = np.abs(x).reshape(64, 8, 32)
    top = np.argmax(blk, axis=2)
    cb = codes.reshape(64, 8, 32)
    e_field = (np.take_along_axis(cb, top[:, :, None], 2)[:, :, 0] & 0x78) >> 3
    assert np.all(e_field == 15)


def test_quantize_power_of_two_equivariance_and_block_independence():
    rng = np.random.default_rng(2)
    x = O.round_bf16(rng.normal(size=(8, 128)))
    c0, s0 = O.mxfp8_quantize(x)
    for j in (-20, -3, 5, 30):
        c1, s1 = O.mxfp8_quantize(x * 2.0 ** j)
        np.testing.assert_array_equal(c1, c0)
        np.testing.assert_array_equal(s1.astype(int), s0.astype(int) + j)
    y = x.copy()
    y[:, 40] *= 64.0                                        # element of block 1 only
    c2, s2 = O.mxfp8_quantize(y)
    keep = np.ones(128, bool)
    keep[32:64] = False
    np.testing.assert_array_equal(c2[:, keep], c0[:, keep])
    np.testing.assert_array_equal(np.delete(s2, 1, axis=1), np.delete(s0, 1, axis=1))


def test_encoded_values_round_trip_exactly():
    # values that are already E4M3 times a power of two with the block
    # maximum in [256, 448] survive quantisation exactly
    rng = np.random.default_rng(3)
    codes = rng.integers(0, 0x7F, size=(16, 64)).astype(np.uint8)
    codes[:, ::32] = 0x78 + rng.integers(0, 7, size=(16, 2))   # block max in [256, 448]
    sign = (rng.integers(0, 2, size=codes.shape) << 7).astype(np.uint8)
    codes = codes | sign
    s = rng.integers(-30, 30, size=(16, 2))
    x = O.e4m3_decode(codes) * np.repeat(np.ldexp(1.0, s), 32, axis=1)
    c, sc = O.mxfp8_quantize(x)
    np.testing.assert_array_equal(O.mxfp8_dequantize(c, sc), x)


def test_zero_block_and_shape_rules():
    x = np.zeros((2, 64))
    x[1, 33] = 3.0
    c, s = O.mxfp8_quantize(x)
    assert np.all(s[0] == 0) and s[1, 0] == 0 and s[1, 1] == 127 + 1 - 8
    assert np.all(O.mxfp8_dequantize(c, s) == x)
    with pytest.raises(ValueError):
        O.mxfp8_quantize(np.zeros((1, 48)))


def test_dispatch_mxfp8_rows_and_payload():
    rng = np.random.default_rng(4)
    S, D, E, K = 40, 96, 6, 3
    x = O.round_bf16(rng.normal(size=(S, D)))
    logits = rng.normal(size=(S, E)).astype(np.float32)
    idx, p = O.route(logits, K)
    _, _, _, inv = O.expert_permutation(idx, E)
    cd, sc, pd = O.dispatch_mxfp8(x, p, inv, K)
    c, s = O.mxfp8_quantize(x)
    for t in range(S):
        for k in range(K):
            pos = inv[t * K + k]
            np.testing.assert_array_equal(cd[pos], c[t])
            np.testing.assert_array_equal(sc[pos], s[t])
            assert pd[pos] == p[t, k]
    # Eq. 1 with b_x = 1 + 1/32: the bench workload's dispatch payload
    assert O.mx_payload_bytes(8192, 6, 2048) == 8192 * 6 * (2048 + 64 + 4) == 104_005_632
    assert O.mx_payload_bytes(8192, 6, 2048) / O.dispatch_payload_bytes(8192, 6, 2048) < 0.52


def test_layer_with_mxfp8_payload_reads_decoded_rows():
    rng = np.random.default_rng(5)
    S, D, E, K, F = 24, 64, 4, 2, 32
    x = O.round_bf16(rng.normal(size=(S, D)))
    Wr = rng.normal(size=(D, E)) / 8
    W1 = rng.normal(size=(E, D, F)) / 8
    W2 = rng.normal(size=(E, F, D)) / 6
    f = O.layer_fwd(x, Wr, W1, W2, K, payload="mxfp8", round_payload=False)
    xq, xs = O.mxfp8_quantize(x)
    g = O.layer_fwd(O.mxfp8_dequantize(xq, xs), Wr, W1, W2, K, logits=O.router_logits(x, Wr),
                    round_payload=False)
    np.testing.assert_allclose(f["y"], g["y"], rtol=0, atol=1e-12)
    with pytest.raises(ValueError):
        O.layer_fwd(x, Wr, W1, W2, K, payload="fp4")
