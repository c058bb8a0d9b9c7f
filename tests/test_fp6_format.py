"""CPU checks of the FP6 (e2m3) code format the FP6 MFMA route uses (no GPU needed).

The route is exact only if every INT4 code is an e2m3 value and the test-side decoder
reads the padded layout as the format defines it: both are checked here against the
format's definition (OCP Microscaling Formats: sign, 2 exponent bits with bias 1, 3
mantissa bits, exponent 0 subnormal)."""
import numpy as np

from gpu_util import E2M3_TABLE, decode_fp6_rows, e2m3_value


def test_e2m3_value_table():
    # the normal and subnormal ranges of the definition
    assert e2m3_value(0b0_00_000) == 0.0
    assert e2m3_value(0b0_00_001) == 0.125
    assert e2m3_value(0b0_00_111) == 0.875
    assert e2m3_value(0b0_01_000) == 1.0
    assert e2m3_value(0b0_11_111) == 7.5
    assert e2m3_value(0b1_10_100) == -3.0
    assert len(set(E2M3_TABLE[:32])) == 32  # 32 distinct magnitudes


def test_every_int4_code_is_exact_in_e2m3():
    """Every code |q| <= 7 is exactly one e2m3 value of each sign (and 0 twice)."""
    for q in range(-7, 8):
        hits = [f for f in range(64) if E2M3_TABLE[f] == q]
        assert len(hits) == (2 if q == 0 else 1), (q, hits)


def test_products_and_sums_exact_in_fp32():
    """Products of two codes and their sums over K <= 2^18 stay integers below 2^24: an
    fp32 accumulator adds them exactly in any order."""
    q = np.arange(-7, 8, dtype=np.float32)
    prods = np.outer(q, q).astype(np.float32)
    assert np.array_equal(prods, np.outer(q.astype(np.int64), q.astype(np.int64)))
    assert 49 * 11008 < 2 ** 24


def _encode(codes):
    """Reference packer from the definition: code q -> the e2m3 field of value q."""
    field = {int(E2M3_TABLE[f]): f for f in range(64) if E2M3_TABLE[f] == int(E2M3_TABLE[f]) and f != 32}
    R, K = codes.shape
    out = np.zeros((R, K), dtype=np.uint8)
    for r in range(R):
        for g in range(K // 32):
            v = 0
            for i in range(32):
                v |= field[int(codes[r, 32 * g + i])] << (6 * i)
            out[r, 32 * g:32 * g + 24] = np.frombuffer(v.to_bytes(24, "little"), dtype=np.uint8)
    return out


def test_decoder_round_trip():
    rng = np.random.default_rng(0)
    codes = rng.integers(-7, 8, size=(5, 128))
    assert np.array_equal(decode_fp6_rows(_encode(codes)), codes.astype(np.float64))
