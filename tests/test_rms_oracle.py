"""Pins of the RMSNorm + FP8 quantization oracle: the E4M3 encoder against
the format's definition and the library's float8_e4m3fn conversion, and the
normalization against closed forms and invariants."""
import numpy as np
import pytest

from oracle import mathref
from oracle.mathref import E4M3_MAX, e4m3fn_decode, e4m3fn_encode, rmsnorm_fp8_rows
from workloads import rmsnorm_program, rmsnorm_worklist
from workloads.tensors import bf16_to_f32, rmsnorm_inputs, to_bf16_bits

torch = pytest.importorskip("torch")


def _finite_codes():
    c = np.arange(256, dtype=np.uint8)
    return c[(c & 0x7F) != 0x7F]


def test_e4m3_decode_matches_format_definition():
    """Exponent bias 7, three mantissa bits, subnormals m/8 * 2^-6, largest
    finite 448 = 1.75 * 2^8, smallest subnormal 2^-9."""
    c = _finite_codes()
    v = e4m3fn_decode(c)
    ref = torch.from_numpy(c).view(torch.float8_e4m3fn).double().numpy()
    assert np.array_equal(v, ref)
    assert v.max() == E4M3_MAX == 1.75 * 2 ** 8
    assert np.min(np.abs(v[v != 0])) == 2.0 ** -9


def test_e4m3_encode_round_trip_and_ties_to_even():
    c = _finite_codes()
    c = c[c != 0x80]                         # -0 encodes as 0x80 only from -0.0
    v = e4m3fn_decode(c)
    assert np.array_equal(e4m3fn_encode(v), c)
    # midpoints between neighbours round to the even mantissa
    pos = np.sort(e4m3fn_decode(c[c < 0x80]))
    mids = (pos[:-1] + pos[1:]) / 2
    got = e4m3fn_encode(mids)
    lo, hi = e4m3fn_encode(pos[:-1]), e4m3fn_encode(pos[1:])
    want = np.where(lo % 2 == 0, lo, hi)
    assert np.array_equal(got, want)
    assert np.array_equal(e4m3fn_encode(-mids), want | 0x80)
    # values between 448 and 464 saturate to 448
    assert np.all(e4m3fn_encode(np.array([448.0, 450.0, 463.9])) == 0x7E)


def test_e4m3_encode_matches_library_conversion():
    rng = np.random.default_rng(7)
    x = (rng.standard_normal(200000) * rng.choice([1e-4, 1e-2, 1.0, 30.0, 200.0], 200000)).clip(-460, 460)
    x = x.astype(np.float32)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(e4m3fn_encode(x.astype(np.float64)), ref)


def test_rmsnorm_constant_row_closed_form():
    """A row of one value c with gamma = 1: y = c / sqrt(c^2 + eps) everywhere,
    every code is the largest magnitude and s = |y| / 448."""
    h, eps = 1024, 1e-6
    g = to_bf16_bits(np.ones(h, np.float32))
    for c in (0.5, -3.0, 2.0 ** -10):
        x = to_bf16_bits(np.full((1, h), c, np.float32))
        codes, s, t = rmsnorm_fp8_rows(x, g, eps, [0])
        cb = float(bf16_to_f32(x[0, :1])[0])
        y = cb / np.sqrt(cb * cb + eps)
        assert np.all(codes == (0xFE if c < 0 else 0x7E))
        assert s[0] == pytest.approx(abs(y) / 448.0, rel=1e-14)


def test_rmsnorm_zero_row():
    h = 1024
    codes, s, _ = rmsnorm_fp8_rows(np.zeros((1, h), np.uint16), to_bf16_bits(np.ones(h, np.float32)), 1e-6, [0])
    assert s[0] == 1.0 and not codes.any()


def test_rmsnorm_invariants():
    """With gamma = 1 and eps = 0 the normalized row has mean square 1; each
    nonzero row reaches the largest code; dequantized values are within half
    an E4M3 step of y."""
    ri = rmsnorm_inputs(seed=3, t=16, h=2048)
    ones = to_bf16_bits(np.ones(2048, np.float32))
    codes, s, t = rmsnorm_fp8_rows(ri.x, ones, 0.0, range(16))
    y = t * s[:, None]
    assert np.allclose(np.mean(y * y, axis=1), 1.0, rtol=1e-12)
    codes, s, t = rmsnorm_fp8_rows(ri.x, ri.gamma, 1e-6, range(16))
    assert np.all(np.max(codes & 0x7F, axis=1) == 0x7E)
    dq = e4m3fn_decode(codes) * s[:, None]
    y = t * s[:, None]
    step = np.where(np.abs(t) >= 2.0 ** -6, np.abs(t) * 2.0 ** -4, 2.0 ** -10) * s[:, None]
    assert np.all(np.abs(dq - y) <= step * (1 + 1e-12))


def test_rmsnorm_rows_match_direct_definition():
    """The row function against the formula written out on a small matrix."""
    ri = rmsnorm_inputs(seed=1, t=8, h=1024)
    x = bf16_to_f32(ri.x).astype(np.float64)
    g = bf16_to_f32(ri.gamma).astype(np.float64)
    y = x / np.sqrt((x ** 2).mean(axis=1, keepdims=True) + 1e-6) * g
    s = np.abs(y).max(axis=1) / 448.0
    codes, s2, _ = mathref.rmsnorm_fp8_rows(ri.x, ri.gamma, 1e-6, range(8))
    assert np.allclose(s2, s, rtol=1e-14)
    ref = torch.from_numpy((y / s[:, None]).astype(np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    amb = mathref.e4m3fn_ambiguous(y / s[:, None])
    assert np.array_equal(codes[~amb], ref[~amb])


def test_rmsnorm_worklist_covers_rows_once():
    for t, n_wg in ((32768, 768), (100, 7), (12, 20), (64, 3)):
        base, tt = rmsnorm_worklist(t, n_wg)
        seen = np.zeros(t, np.int64)
        for w in range(n_wg):
            n = int(tt.per_wg[w][1][0])
            seen[base[w]:base[w] + n] += 1
        assert np.all(seen == 1), (t, n_wg)
        trips = [int(tt.per_wg[w][1][0]) for w in range(n_wg)]
        assert max(trips) - min(trips) <= 1


def test_rmsnorm_program_offsets():
    """Double buffering: offsets {0, 2} on the row loop, four waits."""
    p = rmsnorm_program(64, 1024)
    assert sorted({k for _, _, k in p.deps}) == [0, 2]
