"""Rounding of float32 results to bfloat16 in the library's kernels, through
the C ABI: llep_combine sums a token's pair rows in float32 and rounds once,
so with gates of 1 and two bf16 rows whose float32 sum is exact, each output
element is that exact sum rounded to bfloat16 (the float32 sum starts from
+0, as a sum over k does, so -0 + -0 gives +0). The expected bits come from the
definition of round-to-nearest-even on the float32 bits u,
(u + 0x7fff + ((u >> 16) & 1)) >> 16, with NaNs kept NaN; the cases cover
ties both ways, carries into the exponent, overflow to infinity, subnormal
sums, signed zeros, infinities and NaNs."""

import numpy as np
import pytest

from gpu_util import device

pytestmark = pytest.mark.gpu

D = 64


@pytest.fixture(scope="module")
def dev():
    return device()


def _bf16_bits(f32: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(f32, np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def _pairs(rng, n):
    """n pairs of bf16 bit patterns (a, b) whose float32 sum is exact."""
    out = []
    # random finite values of either sign, b within 2^-15 .. 2^0 of a's
    # magnitude, so the 8-bit significands overlap in a 24-bit sum
    sa = rng.integers(0, 2, n)
    ea = rng.integers(1, 254, n)
    ma = rng.integers(0, 128, n)
    shift = rng.integers(0, 16, n)
    sb = np.where(rng.random(n) < 0.8, sa, 1 - sa)
    eb = np.clip(ea - shift, 1, 254)
    mb = rng.integers(0, 128, n)
    a = (sa << 15) | (ea << 7) | ma
    b = (sb << 15) | (eb << 7) | mb
    out += list(zip(a.tolist(), b.tolist()))

    def f(x):
        return int(np.float32(x).view(np.uint32) >> 16)

    one, ulp = f(1.0), 2.0 ** -7
    out += [
        (one, f(ulp / 2)),             # tie: 1 + half an ulp -> 1 (even)
        (f(1 + ulp), f(ulp / 2)),      # tie: 1 + 1.5 ulp -> 1 + 2 ulp (even)
        (one, f(ulp / 2 + ulp / 4)),   # above the tie -> 1 + ulp
        (f(-1.0), f(-ulp / 2)),        # negative tie -> -1
        (f(255 / 128), f(ulp / 2)),    # carry into the exponent -> 2
        (0x7F7F, 0x7F7F),              # max + max overflows float32 -> inf
        (0x7F7F, 0x7B00),              # rounds up past the largest bf16 -> inf
        (0x0001, 0x0001),              # smallest subnormals
        (0x007F, 0x0001),              # subnormal carry into the normal range
        (0x8000, 0x8000),              # 0 + -0 + -0 = +0
        (0x0000, 0x8000),              # +0 + -0 = +0
        (0x7F80, 0x3F80),              # inf + 1 = inf
        (0xFF80, 0x3F80),              # -inf + 1 = -inf
        (0x7FC0, 0x3F80),              # NaN stays NaN
        (0x7F80, 0xFF80),              # inf - inf = NaN
    ]
    return out


def test_combine_rounds_to_nearest_even(dev):
    import torch
    from paper_2601_17111_amd import binding as B
    rng = np.random.default_rng(11)
    pairs = _pairs(rng, 20000)
    n = len(pairs)
    T = (n + D - 1) // D
    a = np.zeros(T * D, np.uint16)
    b = np.zeros(T * D, np.uint16)
    a[:n] = [p[0] for p in pairs]
    b[:n] = [p[1] for p in pairs]
    # out_perm rows: token t's pair 0 is row t (values a), pair 1 row T + t (b)
    out_perm = np.concatenate([a.reshape(T, D), b.reshape(T, D)]).view(np.int16)
    pair_row = np.stack([np.arange(T), T + np.arange(T)], axis=1).astype(np.int32)
    params = B.make_params(T, 2, 1, 1, 2 * T)
    op = torch.from_numpy(out_perm).to(dev).view(torch.bfloat16)
    pr = torch.from_numpy(pair_row).to(dev)
    y = torch.empty((T, D), dtype=torch.bfloat16, device=dev)
    B.llep_combine(params, op, pr, None, y)
    torch.cuda.synchronize()
    got = y.cpu().view(torch.int16).numpy().reshape(-1).view(np.uint16)[:n]

    fa = (a[:n].astype(np.uint32) << 16).view(np.float32)
    fb = (b[:n].astype(np.uint32) << 16).view(np.float32)
    with np.errstate(over="ignore", invalid="ignore"):
        s = fa.astype(np.float64) + fb.astype(np.float64)
        s32 = ((np.float32(0.0) + fa) + fb).astype(np.float32)
    exact = np.isfinite(s) & (np.abs(s) <= np.finfo(np.float32).max)
    # the float32 sums are exact by construction, except the overflows
    assert np.array_equal(s32[exact].astype(np.float64), s[exact])
    want = _bf16_bits(s32)
    nan = np.isnan(s32)
    got_nan = ((got & 0x7F80) == 0x7F80) & ((got & 0x7F) != 0)
    assert np.array_equal(got_nan, nan)
    bad = np.nonzero((got != want) & ~nan)[0]
    assert bad.size == 0, [(hex(a[i]), hex(b[i]), hex(got[i]), hex(want[i])) for i in bad[:8]]
