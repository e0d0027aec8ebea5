"""Host checks of the swizzled LDS tile layout the kernels use (no GPU).

The formulas mirror paper_2607_01701_amd/csrc/t2v_device.hpp: swz<D>, swz_off<D>, the
per-lane offsets of the 16-byte and transposing operand reads, and the two XOR identities
that let each read be one base register plus one XOR. The DMA writer's lane -> (row, slot)
mapping must place every logical chunk exactly once.
"""
import pytest


def swz(D, r):
    return (((r & 3) << 2) | ((r >> 2) & 3)) if D == 128 else ((r >> 1) & 7)


def off(D, r, col):
    """Byte offset of element (r, col) in a swizzled tile with row stride D (bf16)."""
    return 2 * (r * D + (((col >> 3) ^ swz(D, r)) << 3) + (col & 7))


@pytest.mark.parametrize("D", [128, 64])
def test_swizzle_is_a_permutation_of_each_row(D):
    for r in range(128):
        assert sorted(c ^ swz(D, r) for c in range(D // 8)) == list(range(D // 8))


@pytest.mark.parametrize("D", [128, 64])
def test_dma_fills_every_chunk_once(D):
    cpr, rows = D // 8, 64
    seen = set()
    for i in range(rows * cpr // 64):          # wave instructions
        for lane in range(64):
            r = i * (64 // cpr) + lane // cpr
            c = (lane % cpr) ^ swz(D, r)        # logical chunk this lane loads
            dst = i * 1024 + lane * 16          # where global_load_lds puts it
            assert dst == 2 * (r * D) + 16 * (c ^ swz(D, r))
            seen.add((r, c))
    assert len(seen) == rows * cpr


@pytest.mark.parametrize("D", [128, 64])
def test_xor_addressing_identities(D):
    for lane in range(64):
        G, l32, s, dh = lane >> 5, lane & 31, lane & 15, (lane >> 4) & 1
        ko = off(D, l32, 8 * G)
        for r0 in (0, 32):
            for kk in range(D // 16):
                assert off(D, r0 + l32, 16 * kk + 8 * G) == 2 * r0 * D + (ko ^ (kk << 5))
        for h in (0, 1):
            to = off(D, 4 * G + (s >> 2) + 8 * h, 16 * dh + 4 * (s & 3))
            for r0 in (0, 16, 32, 48):
                for db in range(D // 32):
                    a = off(D, r0 + 4 * G + (s >> 2) + 8 * h, 32 * db + 16 * dh + 4 * (s & 3))
                    assert a == 2 * r0 * D + (to ^ (db << 6))


def banks_conflict_free(addrs, width):
    """True if the byte ranges [a, a + width) of one 256-byte LDS cycle hit distinct banks."""
    used = set()
    for a in addrs:
        for w in range(0, width, 4):
            bank = ((a + w) // 4) % 64
            if bank in used:
                return False
            used.add(bank)
    return True


def test_d128_reads_are_bank_conflict_free():
    """16 lanes of a 16-byte operand read and 32 lanes of a transposing read per cycle."""
    D = 128
    for half in range(2):            # lanes 0-15 / 16-31 (rows differ), same chunk
        for kk in range(8):
            addrs = [off(D, l, 16 * kk) for l in range(16 * half, 16 * half + 16)]
            assert banks_conflict_free(addrs, 16)
    for G in range(2):
        for h in range(2):
            for db in range(4):
                addrs = []
                for lane in range(32 * G, 32 * G + 32):
                    s, dh = lane & 15, (lane >> 4) & 1
                    addrs.append(off(D, 4 * G + (s >> 2) + 8 * h, 32 * db + 16 * dh + 4 * (s & 3)))
                assert banks_conflict_free(addrs, 8)


def tile_dma_sources(D, R, nthreads, rs, row0, L):
    """Byte offsets (from token 0 of the clip) that the TileDma model reads, per (wave, lane, j),
    with the destination (row, logical chunk) each lands in. Mirrors TileDma::copy."""
    cpr, rpi = D // 8, 64 // (D // 8)
    nw = nthreads // 64
    nj = (R // rpi) // nw
    out = []
    for wave in range(nw):
        for lane in range(64):
            r0 = rpi * wave + lane // cpr
            col = ((lane % cpr) ^ swz(D, r0)) * 16
            off0 = r0 * rs * 2 + col
            for j in range(nj):
                rj = r0 + rpi * nw * j
                if row0 + R <= L:
                    src = row0 * rs * 2 + j * rpi * nw * rs * 2 + off0
                else:
                    src = row0 * rs * 2 + min(rj, L - 1 - row0) * rs * 2 + col
                dst_slot = lane % cpr
                out.append((src, rj, dst_slot ^ swz(D, rj), wave + nw * j, lane))
    return out


@pytest.mark.parametrize("D", [128, 64])
@pytest.mark.parametrize("L", [1, 2, 31, 32, 33, 63, 64, 65, 100, 127, 128, 129, 200])
def test_tile_dma_reads_stay_inside_the_clip(D, L):
    """Every DMA source row lies in [0, L); a full tile reads exactly its rows; each source is
    the logical chunk of the row its destination slot holds, as the old per-lane formula did."""
    H = 24
    rs = H * D
    for row0 in range(0, L, 64):
        seen = set()
        for src, rj, chunk, instr, lane in tile_dma_sources(D, 64, 256, rs, row0, L):
            row, rem = divmod(src, rs * 2)
            assert 0 <= row < L, (row0, rj, row)
            assert row == min(row0 + rj, L - 1)        # clamped to the clip's last row
            assert rem == chunk * 16                    # logical chunk of the destination row
            assert src < 2 ** 32 + row0 * rs * 2       # per-lane part fits 32 bits
            seen.add((rj, chunk))
        assert len(seen) == 64 * (D // 8)               # every (row, chunk) of the tile once


@pytest.mark.parametrize("L", [1, 2, 17, 31, 32, 33, 40, 63, 64, 65, 96, 97, 130])
def test_row_statistics_dma_stays_inside_the_clip(L):
    """rows64_dma: base = row i0 of the tile, lane offset min(off + lane, L - 1 - i0): the row
    read is in [i0, L - 1] for every piece (off = 0 or 32) and lane, including pieces that
    start past the clip's end in a short last tile."""
    for i0 in range(0, L, 64):
        for off in (0, 32):
            for lane in range(32):
                r = min(off + lane, L - 1 - i0)
                assert r >= 0
                assert i0 <= i0 + r <= L - 1
                if i0 + off + lane < L:
                    assert i0 + r == i0 + off + lane
