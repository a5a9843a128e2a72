"""Pins of the oracle's binary16 coding (the fp16 gradients and parameters of
mixed-precision training, ZeRO Sec. 3.1) against numpy's float16 conversions,
an independent library implementation of IEEE 754 binary16."""
import os

import numpy as np

import oracle


def test_decode_all_65536_patterns():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float32)
    got = np.array([oracle.f16_to_f32(int(b)) for b in bits], np.float32)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan].view(np.uint32), ref[~nan].view(np.uint32))  # -0.0 kept


def _encode_many(xs: np.ndarray) -> np.ndarray:
    return np.array([oracle.f32_to_f16(float(x)) for x in xs], np.uint16)


def _check_encode(xs: np.ndarray):
    xs = xs.astype(np.float32)
    with np.errstate(over="ignore"):
        ref = xs.astype(np.float16).view(np.uint16)
    got = _encode_many(xs)
    nan = np.isnan(xs)
    assert np.all((got[nan] & 0x7C00) == 0x7C00) and np.all((got[nan] & 0x03FF) != 0)
    bad = np.nonzero(got[~nan] != ref[~nan])[0]
    assert bad.size == 0, [(float(xs[~nan][i]), hex(int(got[~nan][i])), hex(int(ref[~nan][i]))) for i in bad[:5]]


def test_encode_ties_and_neighbours_of_every_binary16_value():
    # For every finite positive binary16 value: the value itself, the exact midpoint to the
    # next value (a tie), and the fp32 neighbours of that midpoint, in both signs.
    h = np.arange(0, 0x7C00, dtype=np.uint16)
    lo = h.view(np.float16).astype(np.float64)
    hi = (h + 1).view(np.float16).astype(np.float64)  # 0x7C00 is +inf for the last one
    mid = np.where(np.isfinite(hi), (lo + hi) / 2, 65520.0).astype(np.float32)  # exact in fp32
    below = np.nextafter(mid, np.float32(0))
    above = np.nextafter(mid, np.float32(np.inf))
    xs = np.concatenate([lo.astype(np.float32), mid, below, above])
    _check_encode(np.concatenate([xs, -xs]))


def test_encode_strided_sweep_of_fp32_patterns():
    # Every 65,537th fp32 bit pattern: all exponents, subnormals, huge values, NaNs.
    pats = np.arange(0, 1 << 32, 65537, dtype=np.uint64).astype(np.uint32)
    _check_encode(pats.view(np.float32))


def test_encode_special_values():
    xs = np.array([0.0, -0.0, np.inf, -np.inf, 65504.0, 65519.996, 65520.0, 1e-8, 2.0 ** -25,
                   2.0 ** -24, 3 * 2.0 ** -26, 2.0 ** -14, 2.0 ** -14 - 2.0 ** -25], np.float32)
    _check_encode(xs)
    assert oracle.f32_to_f16(float("nan")) & 0x7C00 == 0x7C00


def test_encode_exhaustive_over_all_fp32_patterns():
    # Every one of the 2^32 fp32 bit patterns, in parallel chunks, against torch's CPU
    # float->half conversion (round to nearest even; numpy's cast agrees with it and is
    # checked on a sample in test_encode_matches_numpy_on_a_sample); NaNs must stay NaN.
    from concurrent.futures import ThreadPoolExecutor
    import torch
    chunk = 1 << 26

    def check(c):
        bits = np.arange(chunk, dtype=np.uint32) + np.uint32(c * chunk)
        x = bits.view(np.float32)
        got = oracle.f32_to_f16_array(x)
        ref = torch.from_numpy(x).to(torch.float16).view(torch.int16).numpy().view(np.uint16)
        nan = np.isnan(x)
        bad = np.flatnonzero((got != ref) & ~nan)
        nan_ok = bool(np.all((got[nan] & 0x7C00) == 0x7C00) and np.all((got[nan] & 0x3FF) != 0))
        return bad.size, (int(bits[bad[0]]) if bad.size else None), nan_ok

    workers = max(1, min(8, len(os.sched_getaffinity(0))))
    with ThreadPoolExecutor(max_workers=workers) as ex:
        results = list(ex.map(check, range((1 << 32) // chunk)))
    assert sum(r[0] for r in results) == 0, [hex(r[1]) for r in results if r[1] is not None][:5]
    assert all(r[2] for r in results)


def test_encode_matches_numpy_on_a_sample():
    # numpy's own float16 cast as a second, independent reference on random patterns
    r = np.random.default_rng(21)
    bits = r.integers(0, 1 << 32, size=1 << 21, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    got = oracle.f32_to_f16_array(x)
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).view(np.uint16)
    keep = ~np.isnan(x)
    assert np.array_equal(got[keep], ref[keep])
