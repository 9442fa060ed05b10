"""Host check of the LDS fragment-offset identities the dQ kernel's S+1 variant
relies on: with the bf16 tile swizzle (16-byte chunk index XORed with a 3-bit
function of the row; the same formula as Swz<bf16> in the kernels' header),
every lane's offsets of key blocks 1-3 and of the transposed reads' other halves
and rows follow from two base offsets by fixed XOR patterns."""

K_D, K_VEC = 64, 8           # row length and bf16 elements per 16-byte chunk
TILE_BYTES = 64 * 64 * 2


def _sw(r):
    return ((r ^ (r >> 3)) & 1) | ((r >> 1) & 2) | ((r << 1) & 4)


def _off(r, col):
    return r * K_D + (((col // K_VEC) ^ _sw(r)) * K_VEC) + (col % K_VEC)


def test_swizzle_is_a_permutation_of_each_row():
    for r in range(64):
        assert sorted(_off(r, c) - r * K_D for c in range(K_D)) == list(range(K_D))


def test_fragment_offsets_follow_from_two_bases():
    for pair in range(2):
        pb = pair * 4 * TILE_BYTES
        for lane in range(64):
            hh, s16, cb = lane >> 5, lane & 15, 16 * ((lane >> 4) & 1)
            kofs = [pb + _off(lane & 31, 16 * kb + 8 * hh) * 2 for kb in range(4)]
            for kb in range(4):
                assert kofs[kb] == kofs[0] ^ (kb << 5), (pair, lane, kb)
            for dh in range(2):
                for r8 in range(2):
                    t = pb + _off(8 * r8 + 4 * hh + (s16 >> 2), 32 * dh + cb + 4 * (s16 & 3)) * 2
                    t00 = pb + _off(4 * hh + (s16 >> 2), cb + 4 * (s16 & 3)) * 2
                    assert t == t00 ^ ((dh << 6) | (1040 if r8 else 0)), (pair, lane, dh, r8)
            # a ring slot's offset (a multiple of 16 KiB) adds without touching those bits
            for slot in range(2):
                co = slot * 2 * TILE_BYTES
                assert (kofs[0] + co) ^ (3 << 5) == (kofs[0] ^ (3 << 5)) + co
