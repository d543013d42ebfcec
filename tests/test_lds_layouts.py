"""CPU model of the LDS layout of the dS blocks in the dQ-from-dS kernel (attn_bwd_dqds.hip).

The test restates the kernel's address formulas: the 16-byte-unit permutation applied while
copying a stored 8 KB dS block into LDS, and the per-lane addresses of the transposing reads
(ds_read_b64_tr_b16) that form the dS^T operand.  It checks that the copy is a permutation
inside each 1 KB copy instruction, that every swizzled read fetches the chunk the unswizzled
layout held at the address the kernel read before the permutation (whose operand mapping the GPU
parity tests cover), and that the 32 lanes of each read pass hit 32 distinct bank pairs (LDS:
64 banks of 4 bytes; a b64 read is served 32 lanes per pass)."""
from collections import Counter


def dsw(u: int) -> int:
    """XOR applied to bits 1-3 of 16-byte unit u = 128 sub-block + 32 row + v."""
    row = (u >> 5) & 3
    return ((row & 1) << 1) | ((row >> 1) << 2) | (((u >> 4) & 1) << 3)


def place(u: int) -> int:
    return u ^ dsw(u)


def lane_offset(w: int, lane: int, swizzled: bool) -> int:
    gq, sq, qq = lane >> 4, (lane & 15) >> 2, lane & 3
    off = ((2 * (gq & 1) + (qq >> 1)) * 64 + 32 * (qq & 1) + 4 * (gq >> 1) + sq) * 8
    if swizzled:
        off ^= (((qq >> 1) << 1) | ((gq & 1) << 2) | ((qq & 1) << 3)) * 16
    return (w & 1) * 4096 + off


def read_address(w: int, lane: int, c: int, swizzled: bool) -> int:
    """Byte address in the block of chunk step c (0..7) of this lane's dS^T operand."""
    if swizzled:
        return (c >> 2) * 2048 + (lane_offset(w, lane, True) ^ (64 * (c & 3)))
    return (c >> 2) * 2048 + lane_offset(w, lane, False) + 64 * (c & 3)


def test_copy_is_a_permutation_inside_each_part():
    units = [place(u) for u in range(512)]
    assert sorted(units) == list(range(512))
    assert all(place(place(u)) == u for u in range(512))
    # LDS unit part * 64 + lane is filled by copy instruction `part` from global unit place(...)
    assert all(place(p * 64 + l) >> 6 == p for p in range(8) for l in range(64))


def test_swizzled_reads_fetch_the_same_chunks():
    for w in range(4):
        for c in range(8):
            for lane in range(64):
                a = read_address(w, lane, c, False)
                b = read_address(w, lane, c, True)
                assert 0 <= b < 8192 and b % 8 == 0
                # LDS unit b >> 4 holds global unit place(b >> 4)
                assert place(b >> 4) == a >> 4 and b % 16 == a % 16, (w, c, lane)


def worst_pass(swizzled: bool) -> int:
    worst = 0
    for w in range(4):
        for c in range(8):
            for p in range(2):
                pairs = Counter((read_address(w, lane, c, swizzled) // 8) % 32 for lane in range(32 * p, 32 * p + 32))
                worst = max(worst, max(pairs.values()))
    return worst


def test_reads_are_conflict_free_after_the_swizzle():
    assert worst_pass(False) == 8      # the stored order: 4 bank pairs per pass
    assert worst_pass(True) == 1
