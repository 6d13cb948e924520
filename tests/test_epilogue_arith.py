"""CPU checks of two arithmetic claims the large-tile GEMM1 epilogue relies on
(paper Section 3.1.1, stage (3): SwiGLU and the 1x128 re-quantisation).

The kernel's sequences are replayed here in numpy float32, with the
hardware's base-2 exponential and reciprocal modelled as correctly rounded
results perturbed by one ulp either way:

* the shared-divisor quotient (one correctly rounded reciprocal per block
  scale, then q = v y refined by its exact remainder) rounds exactly as the
  IEEE division v / scale does -- the codes must not depend on it;
* the SwiGLU's relative error stays inside the 8 u (u = 2^-24) that the
  intermediate's admissible set allows, and sigmoid is exactly 1 for g >= 17.

Fused multiply-adds are replayed in x87 extended precision (64-bit
significands), where the products of two float32 values and the sums used
here are exact before the final rounding to float32.
"""
import numpy as np

f32 = np.float32
LD = np.longdouble


def _fma(a, b, c):
    return (LD(a) * LD(b) + LD(c)).astype(f32)


def _divby(v, b):
    pre = np.where(b < f32(2.0 ** -100), f32(2.0 ** 64), f32(1.0)).astype(f32)
    bb = (b * pre).astype(f32)
    y = (f32(1.0) / bb).astype(f32)
    vv = (v * pre).astype(f32)
    q = (vv * y).astype(f32)
    return _fma(_fma(-q, bb, vv), y, q)


def test_shared_divisor_quotient_rounds_like_division():
    rng = np.random.default_rng(7)
    n = 400_000
    amax = (np.exp2(rng.uniform(-140, 60, n)) * rng.uniform(1, 2, n)).astype(f32)
    scale = (amax / f32(448.0)).astype(f32)
    v = (amax * rng.uniform(-1, 1, n)).astype(f32)
    # values at the block's largest magnitude and exact multiples of the scale
    v[:1000] = amax[:1000]
    v[1000:2000] = (scale[1000:2000] * f32(17.0)).astype(f32)
    with np.errstate(under="ignore"):
        got = _divby(v, scale)
        ref = (v / scale).astype(f32)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def _swiglu_fast(g, u, pe, pr):
    log2e = f32(float.fromhex("0x1.715476p+0"))
    log2e_lo = f32(float.fromhex("0x1.4ae0c0p-26"))
    ln2 = f32(float.fromhex("0x1.62e430p-1"))
    z = -g
    t = (z * log2e).astype(f32)
    tl = _fma(z, log2e_lo, _fma(z, log2e, -t))
    e = np.exp2(t.astype(np.float64)).astype(f32)
    if pe:
        e = np.nextafter(e, f32(np.inf) if pe > 0 else f32(-np.inf)).astype(f32)
    e = (e * _fma(tl, ln2, f32(1.0))).astype(f32)
    d = (f32(1.0) + e).astype(f32)
    s0 = (1.0 / d.astype(np.float64)).astype(f32)
    if pr:
        s0 = np.nextafter(s0, f32(np.inf) if pr > 0 else f32(-np.inf)).astype(f32)
    s = _fma(s0, _fma(-d, s0, f32(1.0)), s0)
    return ((g * s).astype(f32) * u).astype(f32), s


def test_fast_swiglu_within_admissible_error():
    rng = np.random.default_rng(8)
    g = np.concatenate([rng.uniform(-95, 95, 300_000), rng.uniform(-20, 20, 300_000),
                        rng.standard_normal(300_000) * 3]).astype(f32)
    u = rng.uniform(-4, 4, g.size).astype(f32)
    ref = g.astype(np.float64) / (1.0 + np.exp(-g.astype(np.float64))) * u.astype(np.float64)
    worst = 0.0
    with np.errstate(over="ignore", under="ignore", invalid="ignore"):
        for pe in (-1, 0, 1):
            for pr in (-1, 0, 1):
                y, _ = _swiglu_fast(g, u, pe, pr)
                ok = np.abs(ref) > 1e-30
                rel = np.abs(y.astype(np.float64)[ok] - ref[ok]) / np.abs(ref[ok])
                worst = max(worst, float(rel.max()) / 2.0 ** -24)
    assert worst <= 8.0, worst


def test_fast_sigmoid_exactly_one_from_17():
    g = np.arange(17, 200, 0.25, dtype=f32)
    with np.errstate(over="ignore", under="ignore"):
        for pe in (-1, 0, 1):
            _, s = _swiglu_fast(g, np.ones_like(g), pe, 0)
            assert (s == f32(1.0)).all()
