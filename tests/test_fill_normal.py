"""The library's seeded normal generator (slw_fill_normal), used to draw the
weights of stacks too large to draw on the host.

The generator is Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel
random numbers: as easy as 1, 2, 3", SC 2011) followed by Box-Muller on
24-bit uniforms.  A plain Python Philox written from that definition is
pinned here against the known-answer vectors published with the method
(counter and key all zero, all ones, and the digits of pi); the GPU test
then checks the library's output, element by element, against it.
"""
import numpy as np
import pytest

from paper_2609_07883_amd import synth

M0, M1, W0, W1 = 0xD2511F53, 0xCD9E8D57, 0x9E3779B9, 0xBB67AE85
MASK = 0xFFFFFFFF


def philox4x32_10(ctr, key):
    c = [int(x) & MASK for x in ctr]
    k = [int(x) & MASK for x in key]
    for r in range(10):
        if r:
            k = [(k[0] + W0) & MASK, (k[1] + W1) & MASK]
        p0, p1 = M0 * c[0], M1 * c[2]
        c = [((p1 >> 32) ^ c[1] ^ k[0]) & MASK, p1 & MASK, ((p0 >> 32) ^ c[3] ^ k[1]) & MASK, p0 & MASK]
    return c


def normals(n, seed):
    """The first n standard normals of the stream keyed by seed (float64)."""
    out = np.empty(4 * ((n + 3) // 4))
    for t in range(len(out) // 4):
        w = philox4x32_10([t & MASK, t >> 32, 0, 0], [seed & MASK, seed >> 32])
        for p in range(2):
            u = ((w[2 * p] >> 8) + 0.5) * 2.0 ** -24
            v = (w[2 * p + 1] >> 8) * 2.0 ** -24
            r = np.sqrt(-2.0 * np.log(u))
            out[4 * t + 2 * p] = r * np.cos(2 * np.pi * v)
            out[4 * t + 2 * p + 1] = r * np.sin(2 * np.pi * v)
    return out[:n]


def test_philox_known_answer_vectors():
    assert philox4x32_10([0, 0, 0, 0], [0, 0]) == [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]
    assert philox4x32_10([MASK] * 4, [MASK] * 2) == [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]
    assert philox4x32_10([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0]) == \
        [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]


def test_reference_normals_are_standard():
    z = normals(40000, 12345)
    assert abs(z.mean()) < 0.02 and abs(z.std() - 1) < 0.02
    assert abs(np.mean(z[0::2] * z[1::2])) < 0.02      # the two halves of a Box-Muller pair are uncorrelated


@pytest.mark.gpu
def test_library_fill_matches_reference():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_07883_amd import api
    n, seed, mean, std = 10003, (7 << 32) | 99, 1.0, 0.02
    t = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    api.fill_normal(t.data_ptr(), n, seed, mean, std, torch.cuda.current_stream().cuda_stream)
    got = t.float().cpu().numpy().astype(np.float64)
    ref = synth.bf16_to_f64(synth.bf16_bits(mean + std * normals(n, seed)))
    # identical after rounding to bf16, but for values within a float32 ulp of a rounding boundary
    ulp = np.abs(ref) * 2.0 ** -7
    assert np.all(np.abs(got - ref) <= ulp)
    assert np.mean(got == ref) > 0.999
