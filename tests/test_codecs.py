"""Pins for the oracle's element decoders (CPU only).

Every one of the 256 e4m3 codes and 65536 bf16 patterns is checked against
torch's own float8_e4m3fn / bfloat16 conversions (a library routine) and
against anchor values fixed by the OCP 8-bit float format (E4M3: bias 7,
largest finite 448, smallest subnormal 2^-9, S.1111.111 the only NaN).
"""
import math

import numpy as np
import torch

import oracle


def test_e4m3_all_codes_match_torch():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    for c in range(256):
        got = oracle.e4m3_to_double(c)
        if math.isnan(ref[c]):
            assert math.isnan(got), c
        else:
            assert got == ref[c] and math.copysign(1, got) == math.copysign(1, ref[c]), c


def test_e4m3_anchor_values():
    anchors = {0x00: 0.0, 0x01: 2.0 ** -9, 0x07: 7 * 2.0 ** -9, 0x08: 2.0 ** -6,
               0x38: 1.0, 0x39: 1.125, 0x40: 2.0, 0x7E: 448.0, 0xFE: -448.0,
               0xB8: -1.0, 0x77: 240.0, 0x78: 256.0}
    for code, val in anchors.items():
        assert oracle.e4m3_to_double(code) == val, hex(code)
    assert math.isnan(oracle.e4m3_to_double(0x7F))
    assert math.isnan(oracle.e4m3_to_double(0xFF))
    assert math.copysign(1.0, oracle.e4m3_to_double(0x80)) == -1.0
    finite = [oracle.e4m3_to_double(c) for c in range(256)
              if c not in (0x7F, 0xFF)]
    assert max(finite) == 448.0 and min(finite) == -448.0


def test_bf16_all_patterns_match_torch():
    bits = np.arange(65536, dtype=np.uint16)
    ref = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(
        torch.float64).numpy()
    # the oracle decodes one value per call; sample every pattern class densely
    for b in list(range(0, 65536, 97)) + [0x0000, 0x8000, 0x3F80, 0x7F7F, 0x0001,
                                          0x7F80, 0xFF80, 0x7FC0]:
        got = oracle.bf16_to_double(b)
        if math.isnan(ref[b]):
            assert math.isnan(got)
        else:
            assert got == ref[b], hex(b)
