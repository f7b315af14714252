"""Pins the oracle's fp32 -> bf16 / fp16 / fp8-e4m3fn round-to-nearest-even
conversions (and the exact upcasts) to torch's CPU dtype conversions.

Every one of the 2^32 fp32 bit patterns is converted by both and compared
(the three formats in parallel threads, about a minute in all), plus every
bit pattern in the exponent windows where each format's subnormal / normal /
overflow rules change as a quick first failure. NaNs compare as a class
(both NaN), everything else bit for bit."""
import numpy as np
import pytest
import torch

TORCH = {"bf16": (torch.bfloat16, torch.uint16), "f16": (torch.float16, torch.uint16),
         "f8": (torch.float8_e4m3fn, torch.uint8)}

# exponent-field windows (biased fp32 exponent) with rule changes per format
WINDOWS = {"bf16": [(0, 2), (252, 256)],
           "f16": [(98, 115), (140, 144), (254, 256)],
           "f8": [(108, 123), (133, 137), (254, 256)]}


def _compare(oracle_mod, name, bits):
    x = bits.view(np.float32)
    ours = oracle_mod.from_f32(x, name)
    tdt, tview = TORCH[name]
    ref = torch.from_numpy(x).to(tdt).view(tview).numpy()
    diff = ours != ref
    if not diff.any():
        return
    # differing encodings are allowed only where both are NaNs
    back_ours = oracle_mod.to_f32(ours[diff], name)
    back_ref = oracle_mod.to_f32(ref[diff], name)
    bad = ~(np.isnan(back_ours) & np.isnan(back_ref))
    assert not bad.any(), (name, [hex(int(v)) for v in bits[diff][bad][:8]], ours[diff][bad][:8],
                           ref[diff][bad][:8])


def _chunks(lo, hi, step=1, chunk=1 << 25):
    for s in range(lo, hi, chunk * step):
        e = min(hi, s + chunk * step)
        yield np.arange(s, e, step, dtype=np.uint64).astype(np.uint32)


@pytest.mark.parametrize("name", ["bf16", "f16", "f8"])
def test_boundary_exponent_windows_exhaustive(oracle_mod, name):
    for e0, e1 in WINDOWS[name]:
        for sign in (0, 1):
            lo = (sign << 31) | (e0 << 23)
            hi = (sign << 31) | (e1 << 23)
            for bits in _chunks(lo, hi):
                _compare(oracle_mod, name, bits)


def test_all_fp32_patterns(oracle_mod):
    """All 2^32 fp32 patterns, each format in its own thread (the oracle's
    C loop and torch's conversion both run outside the interpreter lock)."""
    from concurrent.futures import ThreadPoolExecutor

    def sweep(name):
        for bits in _chunks(0, 1 << 32):
            _compare(oracle_mod, name, bits)
        return name

    with ThreadPoolExecutor(max_workers=3) as ex:
        assert sorted(ex.map(sweep, ["bf16", "f16", "f8"])) == ["bf16", "f16", "f8"]


@pytest.mark.parametrize("name,nbits", [("bf16", 16), ("f16", 16), ("f8", 8)])
def test_upcast_every_pattern(oracle_mod, name, nbits):
    """All 2^16 / 2^8 patterns upcast exactly like torch, and narrow back to
    themselves (NaNs as a class)."""
    h = np.arange(1 << nbits, dtype=np.uint16 if nbits == 16 else np.uint8)
    ours = oracle_mod.to_f32(h, name)
    tdt, tview = TORCH[name]
    ref = torch.from_numpy(h.view(np.int16 if nbits == 16 else np.int8)).view(tdt).float().numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan].view(np.uint32), ref[~nan].view(np.uint32))
    back = oracle_mod.from_f32(ours, name)
    assert np.array_equal(back[~nan], h[~nan])


def test_fp8_named_points(oracle_mod):
    """e4m3fn facts: max 448, min subnormal 2^-9, 464 is the tie that rounds
    down to 448, anything rounding past it is NaN, infinity is NaN; a NaN
    input gives the canonical NaN 0x7F whatever its sign."""
    cases = [(448.0, 0x7E), (464.0, 0x7E), (465.0, 0x7F), (480.0, 0x7F), (float("inf"), 0x7F),
             (-448.0, 0xFE), (-1000.0, 0xFF), (2.0**-9, 0x01), (2.0**-10, 0x00), (1.5 * 2.0**-10, 0x01),
             (2.0**-6, 0x08), (1.0, 0x38), (0.0, 0x00), (-0.0, 0x80), (float("nan"), 0x7F),
             (-float("nan"), 0x7F)]
    x = np.array([c[0] for c in cases], dtype=np.float32)
    got = oracle_mod.from_f32(x, "f8")
    assert [int(v) for v in got] == [c[1] for c in cases]


def test_fp16_bf16_named_points(oracle_mod):
    f16 = {65504.0: 0x7BFF, 65519.0: 0x7BFF, 65520.0: 0x7C00, 2.0**-24: 0x0001, 2.0**-25: 0x0000,
           1.5 * 2.0**-25: 0x0001, 2.0**-14: 0x0400, 1.0: 0x3C00, -2.0: 0xC000}
    got = oracle_mod.from_f32(np.array(list(f16), dtype=np.float32), "f16")
    assert [int(v) for v in got] == list(f16.values())
    bf = {1.0: 0x3F80, 1.00390625: 0x3F80, 1.01171875: 0x3F82, 3.3895313892515355e38: 0x7F7F,
          float("inf"): 0x7F80, -0.0: 0x8000}
    got = oracle_mod.from_f32(np.array(list(bf), dtype=np.float32), "bf16")
    assert [int(v) for v in got] == list(bf.values())
