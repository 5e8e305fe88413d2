"""The allocation-free self-check (pictura_selftest_rcp_noalloc) against the
allocating one (pictura_selftest_rcp), through the C ABI: the same mismatch
counts on the same ranges, on calls in a row with shrinking ranges (the
counter lives in the library's fixed device array and keeps the last call's
value, so each call must clear it), and the same argument errors."""
import struct

import pytest

pytestmark = pytest.mark.gpu


def _bits(f):
    return struct.unpack("<I", struct.pack("<f", f))[0]


@pytest.fixture(scope="module")
def ctx():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    from paper_2607_26005_amd import pictura
    h = pictura.pictura_create(0)
    yield pictura, h
    pictura.pictura_destroy(h)


def test_noalloc_matches_allocating_selftest(ctx):
    pictura, h = ctx
    # subnormal arguments, where 1/x overflows to +inf but the hardware reciprocal
    # and its Newton step do not (a non-zero count), then the fast reciprocal's
    # exact range (a zero count); each range twice, the second call smaller
    cases = [(1, 1 << 21), (1, 1 << 19), (_bits(1.0), 1 << 22), (_bits(1.0), 1 << 18),
             (_bits(-3.0), 1 << 20), (_bits(-3.0), 1 << 16)]
    counts = []
    for lo, n in cases:
        want = pictura.pictura_selftest_rcp(h, lo, n)
        got = pictura.pictura_selftest_rcp_noalloc(h, lo, n)
        print(f"[noalloc] lo={lo:#x} n={n}: {got} (allocating: {want})", flush=True)
        assert got == want, (lo, n, got, want)
        counts.append(got)
    assert counts[0] > counts[1] > 0          # the second, smaller call starts from a cleared counter
    assert counts[2] == counts[3] == counts[4] == counts[5] == 0


def test_noalloc_argument_errors(ctx):
    pictura, h = ctx
    with pytest.raises(pictura.PicturaError) as e:
        pictura.pictura_selftest_rcp_noalloc(h, 0x7F7FFFFF, 2)   # past the largest finite float
    assert e.value.status == pictura.EINVAL
    # the context stays usable after the error
    assert pictura.pictura_selftest_rcp_noalloc(h, _bits(2.0), 1024) == 0
