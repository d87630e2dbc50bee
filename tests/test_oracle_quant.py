"""Pins for the oracle's 4-bit cache rows (the reading of the quantisation
experiments: per row, asymmetric 4-bit codes in groups of 32 channels, fp32
scale and offset; see the oracle header)."""
import numpy as np
import pytest


def _bf16(x):
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def _f(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _codes(c):
    """Unpack [n][d/2] bytes to [n][d] codes (channel 2j in the low nibble)."""
    lo, hi = c & 15, c >> 4
    return np.stack([lo, hi], axis=-1).reshape(c.shape[0], -1).astype(np.int32)


@pytest.mark.parametrize("d", [32, 64, 128])
def test_grid_rows_are_exact(orc, d):
    # Values already on a 16-level grid with a power-of-two step come back
    # bit for bit, with the grid index as the code.
    rng = np.random.default_rng(d)
    n = 20
    k = rng.integers(0, 16, (n, d))
    k[:, ::32] = 0
    k[:, 1::32] = 15  # every group spans the whole grid
    lo = rng.integers(-8, 8, (n, d // 32)).astype(np.float32) * 0.25
    step = np.float32(2.0) ** rng.integers(-6, 0, (n, d // 32)).astype(np.float32)
    x = np.repeat(lo, 32, axis=1) + k.astype(np.float32) * np.repeat(step, 32, axis=1)
    bits = _bf16(x)
    assert np.array_equal(_f(bits), x)  # the grid is bf16-representable
    codes, meta = orc.quant_rows(bits)
    np.testing.assert_array_equal(_codes(codes), k)
    np.testing.assert_array_equal(meta[..., 0], step)
    np.testing.assert_array_equal(meta[..., 1], lo)
    np.testing.assert_array_equal(orc.dequant_rows(codes, meta), bits)


def test_constant_group(orc):
    bits = np.full((3, 64), _bf16(np.float32(-2.75)), dtype=np.uint16)
    bits[1, 32:] = _bf16(np.float32(0.0))
    codes, meta = orc.quant_rows(bits)
    assert np.all(codes == 0) and np.all(meta[..., 0] == 0)
    np.testing.assert_array_equal(orc.dequant_rows(codes, meta), bits)


def test_signed_zero_offset(orc):
    # A group whose minimum is zero stores +0 as its offset whichever zero
    # (+0 or -0) comes first, so the stored bits depend only on the values.
    for first, second in ((0x8000, 0x0000), (0x0000, 0x8000), (0x8000, 0x8000)):
        x = np.full((1, 32), first, dtype=np.uint16)
        x[0, 1::2] = second
        x[0, 5] = _bf16(2.0)
        c, m = orc.quant_rows(x)
        assert m[0, 0, 1].view(np.uint32) == 0
        assert m[0, 0, 0] == np.float32(2.0) / np.float32(15.0)
        assert _codes(c)[0, 5] == 15 and np.all(np.delete(_codes(c)[0], 5) == 0)


def test_nibble_order(orc):
    # Channel 2j is the low nibble of byte j: a ramp 0..15 repeated.
    x = np.tile(np.arange(16, dtype=np.float32), 2)[None, :]
    codes, meta = orc.quant_rows(_bf16(x))
    assert meta[0, 0, 0] == 1.0 and meta[0, 0, 1] == 0.0
    assert codes[0, 0] == 0x10 and codes[0, 1] == 0x32 and codes[0, 7] == 0xFE


@pytest.mark.parametrize("scale", [0.01, 1.0, 40.0])
def test_error_bound_and_order(orc, scale):
    # |x - (code*scale + lo)| <= scale/2 (plus fp32 rounding), the group's
    # minimum maps to 0 and its maximum to 15, and codes never decrease with x.
    rng = np.random.default_rng(int(scale * 100))
    bits = _bf16(rng.standard_normal((50, 128)).astype(np.float32) * scale)
    x = _f(bits).astype(np.float64).reshape(50, 4, 32)
    codes, meta = orc.quant_rows(bits)
    c = _codes(codes).reshape(50, 4, 32)
    s, lo = meta[..., 0].astype(np.float64), meta[..., 1].astype(np.float64)
    rec = c * s[..., None] + lo[..., None]
    assert np.all(np.abs(x - rec) <= s[..., None] * (0.5 + 1e-5) + 1e-30)
    assert np.all(c[np.arange(50)[:, None], np.arange(4)[None, :], x.argmin(-1)] == 0)
    assert np.all(c[np.arange(50)[:, None], np.arange(4)[None, :], x.argmax(-1)] == 15)
    order = np.argsort(x, axis=-1, kind="stable")
    assert np.all(np.diff(np.take_along_axis(c, order, axis=-1), axis=-1) >= 0)
    # the bf16 read-back is within half a bf16 step of the fp32 value
    back = _f(orc.dequant_rows(codes, meta)).astype(np.float64).reshape(50, 4, 32)
    assert np.all(np.abs(back - rec) <= np.abs(rec) * 2.0 ** -8 + 1e-30)


def test_attention_over_grid_cache_is_unchanged(orc):
    # A cache whose rows are on the 4-bit grid attends identically after the
    # round trip (decode attention over the read-back rows).
    rng = np.random.default_rng(3)
    n, d = 48, 64
    k = rng.integers(0, 16, (n, d))
    k[:, ::32], k[:, 1::32] = 0, 15
    x = (k.astype(np.float32) - 7.0) * np.float32(0.125)
    K = _bf16(x)
    V = _bf16(x[::-1].copy())
    q = _bf16(rng.standard_normal(d).astype(np.float32))
    Kq = orc.dequant_rows(*orc.quant_rows(K))
    Vq = orc.dequant_rows(*orc.quant_rows(V))
    np.testing.assert_array_equal(Kq, K)
    np.testing.assert_array_equal(orc.attend(q, Kq, Vq, 0.125), orc.attend(q, K, V, 0.125))
