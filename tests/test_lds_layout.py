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
