"""Invariants of the LDS layouts the backward GEMM reads with gfx950's
transposing loads (ds_read_b64_tr_b16), checked on the CPU by enumeration.

The read's lane mapping, as measured on the GPU: within each group of 16
lanes, lane i receives element i mod 4 of the 8-byte pieces addressed by
lanes i/4, i/4 + 4, i/4 + 8 and i/4 + 12 of its group.

Layouts (16-byte slots; a K-slice holds 64 stored rows of 256 columns):
  K-row:        slot(row r, chunk c) = 32 r + (c ^ krow_xor(r))
  chunk-major:  slot(row r, chunk c) = 64 c + (r ^ cm_xor(c))
For each, a lane reading block columns m0 .. m0+31 at sub-step kk addresses
row 16 kk + 8 half + 4 j + a/4 and column m0 + 16 g + 4 (a mod 4) (a = lane
mod 16, g = (lane / 16) mod 2, half = lane / 32, j = which 4 of its 8 K
values).  Checked: the result is the MFMA operand (column m0 + lane mod 32,
K values 8 half .. 8 half + 7 of the sub-step, in order), and the 16- and
32-lane subsets a transposing read serves together land in distinct bank
ranges whether the LDS serves 128 or 256 bytes per clock.
"""


def krow_xor(r):
    j0, j1 = r & 1, (r >> 1) & 1
    return 2 * j1 + 4 * j0 + 8 * (j0 ^ j1)


def cm_xor(c):
    return 4 * (c & 3)


def slot_krow(r, c):
    return 32 * r + (c ^ krow_xor(r))


def slot_cm(r, c):
    return 64 * c + (r ^ cm_xor(c))


def lane_address(slot_fn, lane, kk, j, m0):
    a, g, half = lane & 15, (lane >> 4) & 1, lane >> 5
    r = 16 * kk + 8 * half + 4 * j + a // 4
    m = m0 + 16 * g + 4 * (a % 4)
    return slot_fn(r, m // 8) * 16 + (m % 8) * 2, (r, m)


def transposed_read(slot_fn, kk, j, m0):
    """Emulate one ds_read_b64_tr_b16: per lane, the 4 (row, column) elements received."""
    addr = [lane_address(slot_fn, l, kk, j, m0) for l in range(64)]
    out = []
    for l in range(64):
        g0, i = (l // 16) * 16, l % 16
        elems = []
        for q in range(4):
            _, (r, m) = addr[g0 + i // 4 + 4 * q]
            elems.append((r, m + i % 4))          # element i mod 4 of that lane's 8-byte piece
        out.append(elems)
    return out


def test_xor_patterns_are_bijections():
    for r in range(64):
        assert sorted(c ^ krow_xor(r) for c in range(32)) == list(range(32))
    for c in range(32):
        assert sorted(r ^ cm_xor(c) for r in range(64)) == list(range(64))


def test_transposed_reads_deliver_mfma_fragments():
    for slot_fn in (slot_krow, slot_cm):
        for kk in range(4):
            for m0 in range(0, 256, 32):
                got = [transposed_read(slot_fn, kk, j, m0) for j in range(2)]
                for l in range(64):
                    frag = got[0][l] + got[1][l]
                    want = [(16 * kk + 8 * (l >> 5) + t, m0 + (l & 31)) for t in range(8)]
                    assert frag == want, (slot_fn.__name__, kk, m0, l)


def test_transposed_reads_are_bank_conflict_free():
    # 64 banks x 4 bytes; a request set is conflict-free when no two lanes
    # touch different addresses in the same bank within one served group
    for slot_fn in (slot_krow, slot_cm):
        for kk in range(4):
            for m0 in range(0, 256, 32):
                for j in range(2):
                    addrs = [lane_address(slot_fn, l, kk, j, m0)[0] for l in range(64)]
                    for width, group in ((128, 16), (256, 32)):   # bytes per clock, lanes served together
                        for g0 in range(0, 64, group):
                            seen = {}
                            for a in addrs[g0:g0 + group]:
                                for b in range(a, a + 8, 4):
                                    bank = (b % width) // 4
                                    assert seen.setdefault(bank, b) == b, (slot_fn.__name__, width, kk, m0, j)


# ---- the fused lm-head kernel's 16 x 16 x 32 fragment reads ---------------
# A K-slice tile holds 256 rows of 8 sixteen-byte chunks (128 bytes), chunk
# c of row r at slot 8 r + (c ^ row_xor(r)).  Fragment lane l reads row
# R + (l mod 16) (R a multiple of 16) and chunk 4 ks + sigma(l div 16).  The
# counters show a ds_read_b128 serving lanes i..i+7 together with lanes
# i+32..i+39 (i = 0, 8, 16, 24) from 64 four-byte banks; under that model
# sigma = (0, 2, 1, 3) is conflict-free and the identity is not (it collides
# two-way in every pass, as the 4-per-read SQ_LDS_BANK_CONFLICT count of the
# identity layout said).  The same model leaves the round-1 32 x 32 reads
# (lane l: row l mod 32, chunk 2 kk + l div 32) conflict-free, as measured.


def row_xor(r):
    return (r & 7) ^ ((r >> 3) & 1)


def frag_slot(R, ks, lane, sigma):
    r = R + (lane & 15)
    c = 4 * ks + sigma[lane >> 4]
    return 8 * r + (c ^ row_xor(r))


def frag32_slot(R, kk, lane):
    r = R + (lane & 31)
    c = 2 * kk + (lane >> 5)
    return 8 * r + (c ^ row_xor(r))


def pass_conflicts(slots):
    """Two-way-or-worse bank collisions in the passes of one ds_read_b128."""
    worst = 1
    for i in range(0, 32, 8):
        lanes = list(range(i, i + 8)) + list(range(i + 32, i + 40))
        banks = {}
        for l in lanes:
            base = (slots[l] * 16 % 256) // 4
            for b in range(base, base + 4):
                banks[b] = banks.get(b, 0) + 1
        worst = max(worst, max(banks.values()))
    return worst


def test_fused_fragment_reads_cover_the_fragment():
    # every lane group reads a different chunk of the same 16 rows: together
    # the 64 lanes read 16 rows x 4 chunks of the K-step exactly once
    sigma = (0, 2, 1, 3)
    for R in range(0, 256, 16):
        for ks in range(2):
            got = sorted(frag_slot(R, ks, l, sigma) for l in range(64))
            want = sorted(8 * (R + a) + ((4 * ks + c) ^ row_xor(R + a)) for a in range(16) for c in range(4))
            assert got == want


def test_fused_fragment_reads_are_bank_conflict_free():
    for R in range(0, 256, 16):
        for ks in range(2):
            assert pass_conflicts([frag_slot(R, ks, l, (0, 2, 1, 3)) for l in range(64)]) == 1
            assert pass_conflicts([frag_slot(R, ks, l, (0, 1, 2, 3)) for l in range(64)]) == 2
    for R in range(0, 256, 32):
        for kk in range(4):
            assert pass_conflicts([frag32_slot(R, kk, l) for l in range(64)]) == 1
