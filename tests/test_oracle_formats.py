"""Pins of the oracle's storage-format decoders (exhaustive code tables)."""
import numpy as np
import torch

from oracle.formats import bf16_to_f64, e4m3fn_to_f64, f64_to_e4m3fn, quantise_e4m3fn


def test_e4m3fn_all_codes_match_torch():
    codes = np.arange(256, dtype=np.uint8)
    ours = e4m3fn_to_f64(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).double().numpy()
    nan = np.isnan(ref)
    assert (np.isnan(ours) == nan).all()
    assert np.array_equal(ours[~nan], ref[~nan])
    # sign of zero
    assert np.signbit(ours[0x80]) and not np.signbit(ours[0x00])


def test_e4m3fn_spec_values():
    v = e4m3fn_to_f64(np.array([0x7E, 0xFE, 0x01, 0x07, 0x08, 0x38, 0xB8, 0x7F, 0xFF, 0x00], np.uint8))
    assert v[0] == 448.0 and v[1] == -448.0            # largest finite magnitude
    assert v[2] == 2.0 ** -9                           # smallest subnormal
    assert v[3] == 7 * 2.0 ** -9                       # largest subnormal
    assert v[4] == 2.0 ** -6                           # smallest normal
    assert v[5] == 1.0 and v[6] == -1.0                # bias 7
    assert np.isnan(v[7]) and np.isnan(v[8])           # S.1111.111 is NaN
    assert v[9] == 0.0
    # exactly 2 NaN codes and no infinities in the whole table
    all_v = e4m3fn_to_f64(np.arange(256, dtype=np.uint8))
    assert np.isnan(all_v).sum() == 2 and not np.isinf(all_v).any()


def test_bf16_all_patterns_match_torch():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ours = bf16_to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()
    nan = np.isnan(ref)
    assert (np.isnan(ours) == nan).all()
    assert np.array_equal(ours[~nan], ref[~nan])
    assert bf16_to_f64(np.array([0x3F80, 0xC000, 0x7F80], np.uint16)).tolist() == [1.0, -2.0, np.inf]


def test_e4m3fn_encode_round_trips_every_code():
    codes = np.array([c for c in range(256) if c & 0x7F != 0x7F], np.uint8)
    assert np.array_equal(f64_to_e4m3fn(e4m3fn_to_f64(codes)), codes)


def test_e4m3fn_encode_midpoints_go_to_the_even_code():
    vals = e4m3fn_to_f64(np.arange(0x7F, dtype=np.uint8))
    mid = (vals[:-1] + vals[1:]) / 2                     # exact in fp64
    got = f64_to_e4m3fn(mid).astype(int)
    lo = np.arange(0x7E)
    assert np.array_equal(got, np.where(lo % 2 == 0, lo, lo + 1))
    # just off the midpoint: the nearer neighbour
    eps = np.abs(mid) * 2.0 ** -30
    assert np.array_equal(f64_to_e4m3fn(mid - eps).astype(int), lo)
    assert np.array_equal(f64_to_e4m3fn(mid + eps).astype(int), lo + 1)
    assert np.array_equal(f64_to_e4m3fn(-mid).astype(int), got | 0x80)


def test_e4m3fn_encode_saturates_and_keeps_the_sign_of_zero():
    big = np.array([448.0, 449.0, 464.0, 480.0, 1e30, -1e30, -464.0])
    assert f64_to_e4m3fn(big).tolist() == [0x7E, 0x7E, 0x7E, 0x7E, 0x7E, 0xFE, 0xFE]
    # subnormals step by 2^-9: 2^-10 and 3 * 2^-10 are ties (to codes 0 and 2)
    assert f64_to_e4m3fn(np.array([0.0, -0.0, 2.0 ** -11, 2.0 ** -10, 3 * 2.0 ** -11, 3 * 2.0 ** -10])).tolist() \
        == [0x00, 0x80, 0x00, 0x00, 0x01, 0x02]


def test_e4m3fn_encode_matches_torch_in_range():
    """torch's float8_e4m3fn cast rounds to nearest even (it does not saturate,
    so only values inside the finite range are compared)."""
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * s for s in (2.0 ** -8, 0.05, 1.0, 30.0, 120.0)])
    x = x[np.abs(x) < 440].astype(np.float32)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(f64_to_e4m3fn(x.astype(np.float64)), ref)


def test_quantise_rounds_the_quotient_to_fp32_first():
    # y = x / s in fp32 (IEEE division): with a power-of-two scale the quotient is exact
    x = np.array([1.0, -3.5, 0.0078125, 5.25])
    assert quantise_e4m3fn(x, 2.0 ** -6).tolist() == f64_to_e4m3fn(x * 64).tolist()
    # s = fp32(1 / 1.1875): the exact quotient 1 / s lies just below the
    # midpoint 1.1875 of 1.125 (0x39) and 1.25 (0x3A); fp32 division rounds it
    # onto the midpoint, which goes to the even code 0x3A
    s = float(np.float32(1 / 1.1875))
    assert 1 / s < 1.1875 and f64_to_e4m3fn(np.array([1 / s])).tolist() == [0x39]
    assert float(np.float32(1.0) / np.float32(s)) == 1.1875
    assert quantise_e4m3fn(np.array([1.0]), s).tolist() == [0x3A]
