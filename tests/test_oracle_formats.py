"""Pins of the oracle's storage-format rounding against library routines and the
format definitions (binary16 via numpy, bfloat16 and E4M3FN via torch, E4M3FN
decode values from the OCP 8-bit floating point specification)."""
import numpy as np
import torch


def _boundary_f32_for_f16():
    """Every binary16 value, the midpoints to its neighbours, and one fp32 ulp on
    each side of those midpoints: exactly where a rounding mistake would show."""
    h = np.arange(0, 0x7c00, dtype=np.uint16).view(np.float16).astype(np.float64)
    mids = (h[:-1] + h[1:]) / 2
    pts = np.concatenate([h, mids, [65504.0, 65519.0, 65520.0, 65536.0, 1e6]])
    f = pts.astype(np.float32)
    up = np.nextafter(f, np.float32(np.inf))
    dn = np.nextafter(f, np.float32(0))
    allv = np.concatenate([f, up, dn])
    return np.concatenate([allv, -allv])


def test_f16_rounding_matches_numpy(O):
    x = _boundary_f32_for_f16()
    rng = np.random.default_rng(1)
    r = (rng.standard_normal(2_000_000) * np.exp(rng.uniform(-25, 12, 2_000_000))).astype(np.float32)
    x = np.concatenate([x, r, np.float32([np.inf, -np.inf, 0.0, -0.0])])
    ours = O.f32_to_f16_bits(x)
    with np.errstate(over="ignore"):             # values past the FP16 range round to infinity
        ref = x.astype(np.float16).view(np.uint16)
    assert np.array_equal(ours, ref)




def test_bf16_rounding_matches_torch(O):
    rng = np.random.default_rng(2)
    b = np.arange(0, 0x7f80, dtype=np.uint32) << 16
    v = b.view(np.float32).astype(np.float64)
    mids = ((v[:-1] + v[1:]) / 2).astype(np.float32)
    f = np.concatenate([b.view(np.float32), mids])
    f = np.concatenate([f, np.nextafter(f, np.float32(np.inf)), np.nextafter(f, np.float32(0))])
    r = (rng.standard_normal(2_000_000) * np.exp(rng.uniform(-80, 80, 2_000_000))).astype(np.float32)
    x = np.concatenate([f, -f, r])
    x = x[np.isfinite(x)]
    ours = O.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_e4m3_decode_known_values(O):
    """OCP E4M3FN: bias 7, 3 fraction bits, S.1111.111 = NaN, no infinities."""
    dec = O.e4m3_to_f32(np.arange(256, dtype=np.uint8))
    assert dec[0x7E] == 448.0 and dec[0xFE] == -448.0
    assert dec[0x38] == 1.0 and dec[0x08] == 2.0 ** -6 and dec[0x01] == 2.0 ** -9
    assert dec[0x07] == 7 * 2.0 ** -9 and dec[0x40] == 2.0 and dec[0x7D] == 416.0
    assert np.isnan(dec[0x7F]) and np.isnan(dec[0xFF])
    fin = dec[np.isfinite(dec)]
    assert len(fin) == 254 and len(np.unique(fin)) == 253   # +0 and -0 compare equal
    # matches torch's decoder of the same format
    ref = torch.from_numpy(np.arange(256, dtype=np.uint8)).view(torch.float8_e4m3fn).float().numpy()
    both = np.isfinite(ref)
    assert np.array_equal(dec[both], ref[both])


def test_e4m3_encode_matches_torch_and_argmin(O):
    dec = O.e4m3_to_f32(np.arange(256, dtype=np.uint8)).astype(np.float64)
    finite = np.isfinite(dec)
    pos = np.sort(np.unique(dec[finite & (dec >= 0)]))
    mids = (pos[:-1] + pos[1:]) / 2
    f = np.concatenate([pos, mids]).astype(np.float32)
    f = np.concatenate([f, np.nextafter(f, np.float32(np.inf)), np.nextafter(f, np.float32(0))])
    rng = np.random.default_rng(3)
    r = (rng.uniform(-1, 1, 300_000) * np.exp(rng.uniform(-9, 6.1, 300_000))).astype(np.float32)
    x = np.concatenate([f, -f, r])
    x = np.clip(x, -448, 448).astype(np.float32)
    ours = O.f32_to_e4m3(x)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(ours, ref)
    # brute force: nearest finite code, ties to the even (last fraction bit 0) code
    codes = np.arange(256)[finite & ~((np.arange(256) & 0x7F) == 0x7F)]
    vals = dec[codes]
    sub = x[:: 7][:20000].astype(np.float64)
    d = np.abs(sub[:, None] - vals[None, :])
    best = d.min(axis=1, keepdims=True)
    cand = d <= best
    got = O.f32_to_e4m3(sub.astype(np.float32))
    gv = dec[got]
    assert np.all(np.abs(sub - gv) <= best[:, 0])
    ties = cand.sum(axis=1) > 1
    # at an exact tie the chosen code has an even fraction (ignoring +-0 duplicates)
    tie_even = (got[ties] & 1) == 0
    assert np.all(tie_even | (np.abs(gv[ties]) == 0))


def test_e4m3_saturates(O):
    x = np.float32([448.0, 460.0, 1e4, -1e4, -464.0])
    got = O.f32_to_e4m3(x)
    assert list(got) == [0x7E, 0x7E, 0x7E, 0xFE, 0xFE]
