"""Pins for oracle.casts: format definitions, hand-worked rounding cases and
torch's own conversions (an implementation the oracle does not use)."""

import os

import numpy as np
import pytest
import torch

from oracle import casts

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip() if line.lstrip().startswith("#") else line.strip()
            if line:
                yield line.split()


def test_e4m3_value_table_matches_spec():
    for code, val in _rows("e4m3fn_values.txt"):
        c = int(code, 16)
        assert casts.e4m3_to_f64(np.array([c], dtype=np.uint8))[0] == float(val)
        if float(val) != 0.0:
            assert casts.f64_to_e4m3(np.array([float(val)]))[0] == c
    # every finite code round-trips and values ascend
    codes = np.arange(0x7F, dtype=np.uint8)
    v = casts.e4m3_to_f64(codes)
    assert np.all(np.diff(v) > 0) and v[-1] == 448.0
    assert np.array_equal(casts.f64_to_e4m3(v), codes)
    assert np.array_equal(casts.f64_to_e4m3(-v[1:]), codes[1:] | 0x80)


def test_hand_worked_rounding_cases():
    for kind, x, code, *_ in _rows("rounding_cases.txt"):
        u = np.array([int(x, 16)], dtype=np.uint32)
        if kind == "bf16":
            assert casts.f32_to_bf16(u)[0] == int(code, 16), x
        else:
            xv = u.view(np.float32).astype(np.float64)
            assert casts.f64_to_e4m3(xv)[0] == int(code, 16), x


def _torch_bf16(u32):
    return torch.from_numpy(u32.view(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _structured_f32():
    """Every upper half-word (sign, exponent, 7 high fraction bits) combined with
    the low half-words that decide rounding: zero, just below/at/above the
    halfway point, all ones, and random ones."""
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    rng = np.random.default_rng(1)
    lows = np.concatenate([np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF], dtype=np.uint32),
                           rng.integers(0, 1 << 16, 10, dtype=np.uint32)])
    u = (hi[:, None] | lows[None, :]).ravel()
    return u[(u & 0x7F800000) != 0x7F800000]


def test_f32_to_bf16_matches_torch_structured():
    u = _structured_f32()
    assert np.array_equal(casts.f32_to_bf16(u), _torch_bf16(u))


@pytest.mark.skipif(os.environ.get("WB_EXHAUSTIVE") != "1", reason="exhaustive sweep: set WB_EXHAUSTIVE=1")
def test_f32_to_bf16_matches_torch_exhaustive():
    step = 1 << 24
    for base in range(0, 1 << 32, step):
        u = np.arange(base, base + step, dtype=np.uint64).astype(np.uint32)
        u = u[(u & 0x7F800000) != 0x7F800000]
        assert np.array_equal(casts.f32_to_bf16(u), _torch_bf16(u)), hex(base)


def test_bf16_widening_is_exact():
    c = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    w = casts.bf16_to_f32(c)
    t = torch.from_numpy(c.view(np.int16)).view(torch.bfloat16).to(torch.float32).view(torch.int32).numpy().view(np.uint32)
    finite = (c & 0x7F80) != 0x7F80
    assert np.array_equal(w[finite], t[finite])


def _torch_e4m3(x_f32):
    return torch.from_numpy(x_f32).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_f64_to_e4m3_matches_torch():
    # every bf16 magnitude below 464, both signs, plus all exact midpoints of
    # neighbouring E4M3 values and one fp32 ulp either side of them
    c = np.arange(1 << 15, dtype=np.uint32).astype(np.uint16)
    x = casts.bf16_to_f32(c).view(np.float32)
    x = x[np.isfinite(x) & (x < 464)]
    v = casts.E4M3_VALUES
    mids = ((v[:-1] + v[1:]) / 2).astype(np.float32)
    near = np.concatenate([mids, np.nextafter(mids, np.float32(0)), np.nextafter(mids, np.float32(np.inf))])
    rng = np.random.default_rng(2)
    rnd = (rng.random(200000) * 460).astype(np.float32)
    allx = np.concatenate([x, near, rnd, np.float32(2.0) ** -np.arange(1, 40, dtype=np.float32)]).astype(np.float32)
    allx = np.concatenate([allx, -allx])
    assert np.array_equal(casts.f64_to_e4m3(allx.astype(np.float64)), _torch_e4m3(allx))


def test_quantize_block_matches_torch_formula():
    rng = np.random.default_rng(3)
    for trial in range(200):
        n = int(rng.integers(1, 300))
        scale = 10.0 ** rng.uniform(-30, 30)
        x = (rng.standard_normal(n) * scale).astype(np.float32)
        if trial % 17 == 0:
            x[:] = 0
        codes, s = casts.quantize_block(x)
        xt = torch.from_numpy(x)
        amax = xt.abs().max()
        st = (amax / torch.tensor(448.0)) if amax > 0 else torch.tensor(1.0)
        assert np.float32(s) == np.float32(st.item())
        qt = (xt / st).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        assert np.array_equal(codes, qt)


def test_quantize_invariants():
    rng = np.random.default_rng(4)
    for _ in range(100):
        x = (rng.standard_normal((128, 128)) * 10.0 ** rng.uniform(-20, 20)).astype(np.float32)
        codes, s = casts.quantize_block(x)
        a = np.abs(x)
        # the largest magnitude maps to +-448 exactly (s is a normal number here)
        k = np.argmax(a)
        assert codes.ravel()[k] & 0x7F == 0x7E
        # every code is the nearest E4M3 value to x/s (within half a step)
        q = casts.e4m3_to_f64(codes)
        xs = (x / np.float32(s)).astype(np.float64)
        assert np.all(np.abs(q - xs) <= np.abs(xs) * 2.0 ** -4 + 2.0 ** -10)
        # signs agree
        assert np.all((codes >> 7).astype(bool) == np.signbit(x))


def test_block_scale_zero_block():
    codes, s = casts.quantize_block(np.zeros(64, dtype=np.float32))
    assert s == np.float32(1.0) and not codes.any()
    codes, s = casts.quantize_block(-np.zeros(4, dtype=np.float32))
    assert s == np.float32(1.0) and np.all(codes == 0x80)


def test_quantize_matrix_partial_edges():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((130, 257)).astype(np.float32)
    codes, scales = casts.quantize_matrix(x, 128)
    assert scales.shape == (2, 3)
    # the 2x1 edge block at (1, 2) is quantised on its own
    c, s = casts.quantize_block(x[128:, 256:])
    assert scales[1, 2] == s and np.array_equal(codes[128:, 256:], c)


def test_quantize_divides_rather_than_multiplying_by_the_reciprocal():
    for xs, ams, by_div, by_rcp in _rows("fp8_division_cases.txt"):
        x = np.array([int(xs, 16)], dtype=np.uint32).view(np.float32)[0]
        amax = np.array([int(ams, 16)], dtype=np.uint32).view(np.float32)[0]
        block = np.array([x, amax], dtype=np.float32)
        codes, s = casts.quantize_block(block)
        assert codes[0] == int(by_div), (xs, ams)
        st = torch.tensor(amax) / torch.tensor(448.0)
        assert int((torch.tensor(x) / st).to(torch.float8_e4m3fn).view(torch.uint8)) == int(by_div)
        assert int((torch.tensor(x) * (1.0 / st)).to(torch.float8_e4m3fn).view(torch.uint8)) == int(by_rcp)
