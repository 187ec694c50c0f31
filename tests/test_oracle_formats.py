"""Pins of the oracle's storage-format decoders (exhaustive code tables)."""
import numpy as np
import torch

from oracle.formats import bf16_to_f64, e4m3fn_to_f64


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
