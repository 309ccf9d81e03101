"""The host-side page copies that install and read cached K/V
(runtime.write_pages / read_pages) against the pool layout written out with
tensor indexing, on CPU tensors: bit-exact, with the other tokens of a page
the rows cover in part left as they were.

Pool layout of one layer: K [blocks][Hkv][hd/32][16][32], V
[blocks][Hkv][hd][16]; token t of block b holds K row (h, d) at
[b][h][d / 32][t][d % 32] and V at [b][h][d][t].
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2609_07883_amd import runtime  # noqa: E402


def _bf16(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)


def _bits(t: torch.Tensor) -> np.ndarray:
    return t.view(torch.int16).numpy().view(np.uint16)


def _indexed_write(kp, vp, blk, tok, k, v):
    n, hkv, hd = k.shape
    b, t = torch.from_numpy(blk), torch.from_numpy(tok)
    kp.permute(0, 3, 1, 2, 4)[b, t] = _bf16(k).view(n, hkv, hd // 32, 32)
    vp.permute(0, 3, 1, 2)[b, t] = _bf16(v)


def _indexed_read(kp, vp, blk, tok):
    b, t = torch.from_numpy(blk), torch.from_numpy(tok)
    k = kp.permute(0, 3, 1, 2, 4)[b, t]
    return _bits(k.reshape(len(blk), k.shape[1], -1).contiguous()), _bits(vp.permute(0, 3, 1, 2)[b, t].contiguous())


@pytest.mark.parametrize("hkv,hd", [(1, 64), (8, 128)])
def test_page_copies_match_the_indexed_layout(hkv, hd):
    rng = np.random.default_rng(hkv * 1000 + hd)
    blocks = 12
    k0 = rng.integers(0, 1 << 16, size=(blocks, hkv, hd // 32, 16, 32), dtype=np.uint16)
    v0 = rng.integers(0, 1 << 16, size=(blocks, hkv, hd, 16), dtype=np.uint16)
    pools = [(_bf16(k0).clone(), _bf16(v0).clone()) for _ in range(2)]
    bt = np.array([7, 2, 9, 4, 11], dtype=np.int64)  # scattered blocks of one sequence
    # positions 5..70: a partly covered first page, three whole pages, a partly covered last page
    pos = np.arange(5, 71)
    blk, tok = bt[pos // 16], pos % 16
    k = rng.integers(0, 1 << 16, size=(len(pos), hkv, hd), dtype=np.uint16)
    v = rng.integers(0, 1 << 16, size=(len(pos), hkv, hd), dtype=np.uint16)
    runtime.write_pages(*pools[0], blk, tok, k, v)
    _indexed_write(*pools[1], blk, tok, k, v)
    assert np.array_equal(_bits(pools[0][0]), _bits(pools[1][0]))
    assert np.array_equal(_bits(pools[0][1]), _bits(pools[1][1]))
    # untouched blocks and the uncovered tokens of the first and last pages kept their bits
    untouched = [b for b in range(blocks) if b not in bt]
    assert np.array_equal(_bits(pools[0][0])[untouched], k0[untouched])
    assert np.array_equal(_bits(pools[0][0])[7][:, :, :5], k0[7][:, :, :5])
    assert np.array_equal(_bits(pools[0][1])[11][:, :, 7:], v0[11][:, :, 7:])
    # reads: the written rows come back, and any positions read as the indexed gather does
    kr, vr = runtime.read_pages(*pools[0], blk, tok)
    assert np.array_equal(kr, k) and np.array_equal(vr, v)
    probe = rng.integers(0, 80, size=40)
    pb, pt = bt[probe // 16], probe % 16
    kr, vr = runtime.read_pages(*pools[0], pb, pt)
    ki, vi = _indexed_read(*pools[0], pb, pt)
    assert np.array_equal(kr, ki) and np.array_equal(vr, vi)
