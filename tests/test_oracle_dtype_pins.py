"""Pins for the oracle's bfloat16 and fp8 (e4m3) entries (CPU only).

bfloat16 is the upper half of an IEEE binary32, so its decoder is checked
against torch's bfloat16 -> float64 conversion (a library routine) on all
65,536 bit patterns; the operator on bfloat16 inputs is checked against the
binary16 entry on inputs that both formats represent exactly (the two
entries then see identical values and must agree to rounding of fp64).  The
e4m3 decoder is checked against torch.float8_e4m3fn on all 256 codes, and
since every finite e4m3 value is exact in binary16 the fp8 entry must agree
with the binary16 entry on the widened values."""
import numpy as np
import torch

from paper_2505_08098_amd import workloads as W


def test_bf16_decoder_matches_torch_on_every_pattern(oracle):
    bits = np.arange(65536, dtype=np.uint16)
    got = oracle.widen_bf16(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    assert oracle.bf16_to_double(0x3F80) == 1.0
    assert oracle.bf16_to_double(0xC000) == -2.0
    assert oracle.bf16_to_double(0x0001) == 2.0 ** -133


def test_bf16_entry_equals_f16_entry_on_common_values(oracle):
    """Multiples of 1/32 in [-4, 4] have at most 8 significant bits: exact in
    binary16 and in bfloat16."""
    rng = np.random.default_rng(21)
    N, d = 90, 32
    rp, ci = W.random_csr(rng, N, max_deg=20, empty_frac=0.1, dup_frac=0.2)
    vals = [rng.integers(-128, 129, size=(N, d)) / 32.0 for _ in range(3)]
    f16 = [v.astype(np.float16) for v in vals]
    b16 = [W.to_bf16_bits(v.astype(np.float32)) for v in vals]
    for v, b in zip(vals, b16):
        assert np.array_equal(oracle.widen_bf16(b), v)
    O1, l1 = oracle.attention_f64(rp, ci, *f16, 0.3, want_lse=True)
    O2, l2 = oracle.attention_bf16_f64(rp, ci, *b16, 0.3, want_lse=True)
    np.testing.assert_allclose(O2, O1, rtol=0, atol=1e-13)
    fin = np.isfinite(l1)
    assert np.array_equal(fin, np.isfinite(l2))
    np.testing.assert_allclose(l2[fin], l1[fin], rtol=0, atol=1e-13)


def test_bf16_generator_rounds_to_nearest_even():
    x = np.array([1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -3.0e38, 1e-40],
                 dtype=np.float32)
    b = W.to_bf16_bits(x)
    # ties go to the even neighbour: 1 + 2^-8 -> 1, 1 + 3*2^-8 -> 1 + 2^-6
    assert b[0] == 0x3F80 and b[1] == 0x3F80 and b[2] == 0x3F82
    assert b[3] == 0xFF62 and b[4] != 0


def test_e4m3_decoder_matches_torch_on_every_byte(oracle):
    """OCP e4m3 (torch.float8_e4m3fn, a library routine) on all 256 codes."""
    b = np.arange(256, dtype=np.uint8)
    got = oracle.widen_e4m3(b)
    ref = torch.from_numpy(b).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert nan.sum() == 2 and np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    assert oracle.e4m3_to_double(0x7E) == 448.0 and oracle.e4m3_to_double(0x01) == 2.0 ** -9


def test_e4m3_entry_equals_f16_entry(oracle):
    """Every finite e4m3 value is exact in binary16, so the fp8 entry must
    agree with the fp16 entry on the same values, for any inputs."""
    rng = np.random.default_rng(22)
    N, d = 80, 32
    rp, ci = W.random_csr(rng, N, max_deg=25, empty_frac=0.1, dup_frac=0.2)
    X = [W.to_e4m3_bits(3 * rng.standard_normal((N, d), dtype=np.float32)) for _ in range(3)]
    H = [oracle.widen_e4m3(x).astype(np.float16) for x in X]
    for x, h in zip(X, H):
        assert np.array_equal(h.astype(np.float64), oracle.widen_e4m3(x))
    O1, l1 = oracle.attention_f64(rp, ci, *H, 0.4, want_lse=True)
    O2, l2 = oracle.attention_e4m3_f64(rp, ci, *X, 0.4, want_lse=True)
    np.testing.assert_allclose(O2, O1, rtol=0, atol=1e-13)
    fin = np.isfinite(l1)
    np.testing.assert_allclose(l2[fin], l1[fin], rtol=0, atol=1e-13)
