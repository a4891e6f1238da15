"""CPU model of the global addresses of the many-row LM-head kernel
(paper_2608_12913_amd/csrc/lmhead_wide.hip: workgroup -> tile mapping, Stream::init,
Stream::dma, Stream::prefetch), checked for every lane, load and K-chunk of the ragged
workgroups:
every address stays inside its operand and every 32-bit lane offset is non-negative
and below 2^32.  The kernel's ragged path once formed a negative offset from a slab
that starts past the last row (a GPU memory fault); this guards the fix."""
import numpy as np
import pytest

TT, TR, CB = 256, 256, 128          # tile tokens, tile rows, K-chunk bytes
LPR = CB // 16                      # lanes per row in one load
RPI = 64 // LPR                     # rows per load instruction
SLAB = TT // 4                      # rows of an operand one wave loads per chunk
LOADS = SLAB // RPI


def _ragged_groups(R, V):
    ntiles, nrt = (V + TT - 1) // TT, (R + TR - 1) // TR
    for gid in range((ntiles + 7) // 8 * 8 * nrt):
        xcd, local = gid % 8, gid // 8
        tile = (local // nrt) * 8 + xcd
        if tile >= ntiles:
            continue
        row0 = (local % nrt) * TR
        if (tile + 1) * TT > V or row0 + TR > R:
            yield tile * TT, row0


def _check(R, V, d):
    rowbytes = d * 2
    nch = (rowbytes + CB - 1) // CB
    lane = np.arange(64)
    r = lane // LPR
    col16 = (lane % LPR) ^ (r % LPR)  # the swizzled slot each lane fills
    q = np.arange(LOADS)[:, None]
    checked = 0
    for tile0, row0 in _ragged_groups(R, V):
        for wave in range(4):
            for first, count in ((tile0 + SLAB * wave, V), (row0 + SLAB * wave, R)):
                base = min(first, count - 1)          # the slab's base row, clamped
                skip, last = first - base, count - 1 - base
                assert skip >= 0 and last >= 0
                for c in range(nch + 2):  # the L2 prefetch runs two chunks ahead
                    if c < nch:
                        col = c * CB + col16 * 16
                        col = np.where(col < rowbytes, col, rowbytes - 16)  # weights; hidden: 0
                        rel = np.minimum(skip + RPI * q + r, last)
                        off = rel * rowbytes + col
                        assert np.all(off >= 0) and np.all(off < 2 ** 32)
                        byte = base * rowbytes + off
                        assert np.all(byte >= 0) and np.all(byte + 16 <= count * rowbytes)
                        checked += off.size
                    # the prefetch: 4 bytes of slab row `lane` at the chunk's start
                    # (clamped to the row's last 16 bytes)
                    poff = np.minimum(skip + lane, last) * rowbytes + min(c * CB, rowbytes - 16)
                    assert np.all(poff >= 0) and np.all(poff < 2 ** 32)
                    assert np.all(base * rowbytes + poff + 4 <= count * rowbytes)
    return checked


@pytest.mark.parametrize("R,V,d", [(576, 4099, 512), (576, 4099, 200), (640, 4099, 200),
                                   (512, 300, 64), (513, 257, 8), (576, 257, 24), (2049, 128256, 256)])
def test_ragged_load_addresses_stay_in_bounds(R, V, d):
    assert _check(R, V, d) > 0


def _check_dense_rows(R, V):
    """The untruncated epilogue's float4 accesses to the dense rows [R][tiles*256]:
    row = row0 + 128 wr + 16 rb + lane%16 (clamped to R-1 for loads, skipped past R for
    stores), column = tile*256 + 128 wt + 4 (lane/16) + 16 vb .. +3, for every workgroup
    the kernel launches."""
    ntiles, nrt = (V + TT - 1) // TT, (R + 256 - 1) // 256
    zstride = ntiles * TT
    lane = np.arange(64)
    rb, vb, ln = np.meshgrid(np.arange(8), np.arange(8), lane, indexing="ij")
    n, g = ln % 16, ln // 16
    checked = 0
    for gid in range((ntiles + 7) // 8 * 8 * nrt):
        xcd, local = gid % 8, gid // 8
        tile = (local // nrt) * 8 + xcd
        if tile >= ntiles:
            continue
        row0 = (local % nrt) * 256
        for wave in range(4):
            wt, wr = wave & 1, wave >> 1
            row = row0 + 128 * wr + 16 * rb + n
            col = tile * TT + 128 * wt + 4 * g + 16 * vb
            assert np.all(col % 4 == 0) and np.all(col + 4 <= zstride)
            load = np.minimum(row, R - 1) * zstride + col
            assert np.all(load >= 0) and np.all(load + 4 <= R * zstride)
            store = (row * zstride + col)[row < R]
            assert np.all(store + 4 <= R * zstride)
            checked += row.size
    return checked


@pytest.mark.parametrize("R,V", [(512, 300), (520, 3001), (576, 257), (2048, 128256)])
def test_untruncated_dense_row_accesses_stay_in_bounds(R, V):
    assert _check_dense_rows(R, V) > 0
