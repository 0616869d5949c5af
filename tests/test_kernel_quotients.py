"""Host-side checks of the integer arithmetic the estimate kernels take from
floating point (CPU only: they restate the arithmetic with numpy and never
call a kernel).

* Quotients of GPU counts: n / d for d dividing n <= ARENA_MAX_GPU_COUNT (1024)
  is computed as rint(float(n) * rcp(float(d))) in fp32, where the hardware
  reciprocal is within one unit in the last place.  Checked here for every
  such (n, d) with the reciprocal perturbed by up to two units either way.
* Samples per microbatch: Bg / (dp m) as rint(Bg * r) in fp64, r a reciprocal
  estimate refined by one Newton step, with a product test deciding
  divisibility; checked for every divisor of a range of batch sizes with r
  perturbed by a few units.
* Node-divisor masks: bit d set iff d divides the node size, d <= 31, against
  the remainder test the kernels used before.
"""
import numpy as np
import pytest

MAX_COUNT = 1024    # ARENA_MAX_GPU_COUNT
MAX_NODE = 31       # ARENA_MAX_GPUS_PER_NODE


def _ulp_neighbours(x, k, dtype):
    """x moved by -k .. k units in the last place (same dtype)."""
    out = [dtype(x)]
    lo = hi = dtype(x)
    for _ in range(k):
        lo = np.nextafter(lo, dtype(-np.inf), dtype=dtype)
        hi = np.nextafter(hi, dtype(np.inf), dtype=dtype)
        out += [lo, hi]
    return out


def test_count_quotients_from_float_reciprocals():
    f32 = np.float32
    bad = []
    for d in range(1, MAX_COUNT + 1):
        for r in _ulp_neighbours(f32(1.0) / f32(d), 2, f32):
            n = np.arange(d, MAX_COUNT + 1, d, dtype=np.int64)       # every multiple of d
            q = np.rint(n.astype(f32) * r).astype(np.int64)          # fp32 product, then rounding
            if not np.array_equal(q, n // d):
                bad.append((d, float(r)))
    assert not bad, bad[:5]


def test_count_divisibility_from_float_quotient():
    # the kernels decide d | n by q * d == n for the rounded quotient q: an
    # integer q can only satisfy it when d divides n, whatever q is
    f32 = np.float32
    for d in range(1, 33):
        n = np.arange(1, MAX_COUNT + 1, dtype=np.int64)
        q = np.rint(n.astype(f32) * (f32(1.0) / f32(d))).astype(np.int64)
        assert np.array_equal(q * d == n, n % d == 0)


@pytest.mark.parametrize("batches", [range(1, 4097), [1 << 20, 3 << 18, 1536 * 1024, (1 << 24) - 48]])
def test_microbatch_samples_from_refined_reciprocal(batches):
    bad = []
    for bg in batches:
        divs = [d for d in range(1, min(bg, 4096) + 1) if bg % d == 0]
        for d in divs:
            x = float(d)
            r0 = 1.0 / x
            for r in _ulp_neighbours(r0, 3, np.float64):
                # one Newton step on the perturbed estimate, as the kernels refine it
                e = np.float64(1.0) - np.float64(x) * r
                rr = r + e * r
                q = float(np.rint(np.float64(bg) * rr))
                if q * x != float(bg) or q != bg // d:
                    bad.append((bg, d))
        if bad:
            break
    assert not bad, bad[:5]


def test_node_divisor_mask_matches_remainders():
    for gpn in range(1, MAX_NODE + 1):
        divs = 0
        for d in range(1, gpn + 1):
            if gpn % d == 0:
                divs |= 1 << d
        for grp in range(1, 4 * MAX_COUNT + 1):
            tiles = grp < 32 and bool((divs >> grp) & 1)
            assert tiles == (grp <= gpn and gpn % grp == 0), (gpn, grp)
