"""Invariants of the LDS layouts of the MFMA tile kernels, checked on the CPU
by enumeration.

Backward GEMM (lmhead_backward.hip).  Operands whose stored rows run along
the contracted index K are read with gfx950's transposing load
ds_read_b64_tr_b16, whose lane mapping, as measured on the GPU, is: within
each group of 16 lanes, lane i receives element i mod 4 of the 8-byte pieces
addressed by lanes i/4, i/4 + 4, i/4 + 8 and i/4 + 12 of its group.

Layouts (16-byte slots; a K-slice holds 64 stored K rows of 256 columns):
  K-row:        slot(row r, chunk c) = 32 r + (c ^ krow_xor(r))
  chunk-major:  slot(row r, chunk c) = 64 c + (r ^ cm_xor(c, r))
For the 16-column fragment m0 .. m0+15 at K-step ks, lane a of lane group g
addresses K row 32 ks + 8 sigma(g) + 4 j + a/4 and column m0 + 4 (a mod 4)
(read j = 0, 1; sigma = (0, 2, 1, 3), the K chunk each lane group takes in
every tile kernel).  Checked: the result is the MFMA operand (column
m0 + lane mod 16, K values 8 sigma(g) .. 8 sigma(g) + 7 of the K-step, in
order), and the lanes a read serves together touch distinct banks whether
the LDS serves 16 lanes (128 bytes) or 32 lanes (256 bytes) per clock, and
for either pairing of 16-lane groups.
"""

SIGMA = (0, 2, 1, 3)


def krow_xor(r):
    return 2 * ((r & 3) | ((((r >> 3) ^ (r >> 4)) & 1) << 2))


def cm_xor(c, r):
    return (4 * (c & 1)) ^ (8 * ((r >> 4) & 1))


def slot_krow(r, c):
    return 32 * r + (c ^ krow_xor(r))


def slot_cm(r, c):
    return 64 * c + (r ^ cm_xor(c, r))


def lane_address(slot_fn, lane, ks, j, m0):
    a, g = lane & 15, lane >> 4
    r = 32 * ks + 8 * SIGMA[g] + 4 * j + a // 4
    m = m0 + 4 * (a % 4)
    return slot_fn(r, m // 8) * 16 + (m % 8) * 2, (r, m)


def transposed_read(slot_fn, ks, j, m0):
    """Emulate one ds_read_b64_tr_b16: per lane, the 4 (row, column) elements received."""
    addr = [lane_address(slot_fn, l, ks, j, m0) for l in range(64)]
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
        assert sorted(r ^ cm_xor(c, r) for r in range(64)) == list(range(64))
        # the DMA side inverts the chunk-major pattern by applying it again
        assert all((r ^ cm_xor(c, r)) ^ cm_xor(c, r ^ cm_xor(c, r)) == r for r in range(64))


def test_transposed_reads_deliver_mfma_fragments():
    for slot_fn in (slot_krow, slot_cm):
        for ks in range(2):
            for m0 in range(0, 256, 16):
                got = [transposed_read(slot_fn, ks, j, m0) for j in range(2)]
                for l in range(64):
                    frag = got[0][l] + got[1][l]
                    want = [(32 * ks + 8 * SIGMA[l >> 4] + t, m0 + (l & 15)) for t in range(8)]
                    assert frag == want, (slot_fn.__name__, ks, m0, l)


def _collisions(addrs, lanes, nbytes, width):
    banks = {}
    for l in lanes:
        for b in range(addrs[l], addrs[l] + nbytes, 4):
            banks.setdefault((b % width) // 4, set()).add(b)
    return max(len(v) for v in banks.values())


def test_transposed_reads_are_bank_conflict_free():
    groups = [(128, [list(range(i, i + 16)) for i in range(0, 64, 16)]),      # 16 lanes per clock
              (256, [list(range(0, 32)), list(range(32, 64))]),               # 32 consecutive lanes
              (256, [list(range(0, 16)) + list(range(32, 48)),                # or groups g and g + 2
                     list(range(16, 32)) + list(range(48, 64))])]
    for slot_fn in (slot_krow, slot_cm):
        for ks in range(2):
            for m0 in range(0, 256, 16):
                for j in range(2):
                    addrs = [lane_address(slot_fn, l, ks, j, m0)[0] for l in range(64)]
                    for width, sets in groups:
                        for lanes in sets:
                            assert _collisions(addrs, lanes, 8, width) == 1, (slot_fn.__name__, width, ks, m0, j)


def test_chunk_major_plain_reads_pair_like_the_measured_layout():
    # The plain (ds_read_b128) reads of the GEMM's chunk-major operands:
    # slot c * 256 + i, lane l reads row m0 + l mod 16 of chunk
    # 4 ks + sigma(l div 16).  Lanes i..i+7 and i+32..i+39 then read the
    # same 8 rows of chunks 2 m and 2 m + 1, the pairing the 32-row
    # fragments of this layout used (lane l: row l mod 32, chunk
    # 2 kk + l div 32), for which the counters showed no bank conflict; and
    # every 16 consecutive lanes read 256 contiguous bytes.
    for m0 in range(0, 256, 16):
        for ks in range(2):
            slot = [(4 * ks + SIGMA[l >> 4]) * 256 + m0 + (l & 15) for l in range(64)]
            for i in range(0, 32, 8):
                lo = [slot[l] for l in range(i, i + 8)]
                hi = [slot[l] for l in range(i + 32, i + 40)]
                assert [h - x for x, h in zip(lo, hi)] == [256] * 8
                assert (lo[0] // 256) % 2 == 0
            for g in range(4):
                s16 = slot[16 * g:16 * g + 16]
                assert s16 == list(range(s16[0], s16[0] + 16))
            # every lane group's 8 K values: chunk 4 ks + sigma(g)
            assert sorted({s // 256 for s in slot}) == [4 * ks + c for c in range(4)]


# ---- the fused lm-head kernel's 16 x 16 x 32 fragment reads ---------------
# A K-slice tile holds 256 rows of 8 sixteen-byte chunks (128 bytes), chunk
# c of row r at slot 8 r + (c ^ row_xor(r)).  Fragment lane l reads row
# R + (l mod 16) (R a multiple of 16) and chunk 4 ks + sigma(l div 16).  The
# counters show a ds_read_b128 serving lanes i..i+7 together with lanes
# i+32..i+39 (i = 0, 8, 16, 24) from 64 four-byte banks; under that model
# sigma = (0, 2, 1, 3) is conflict-free and the identity is not (it collides
# two-way in every pass, as the 4-per-read SQ_LDS_BANK_CONFLICT count of the
# identity layout said).  The same model leaves the earlier 32 x 32 reads
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


# Gradient-mode G stores (lmhead_logprob.hip, gradient epilogue).  In a
# 16 x 16 result block lane l holds token column l mod 16 and the 4
# consecutive vocabulary rows 4 (l div 16) .. + 3 of the block.  Blocks are
# paired (bm, bm + 1) and v_permlane16_swap_b32 is applied to each packed
# word (first block's word as the first operand, second block's as the
# second).  Its lane mapping, as measured on the GPU: within each pair of
# 16-lane rows (0, 1) and (2, 3), lane i of the even row returns (its own
# first operand, the first operand of lane i + 16), and lane i + 16 of the
# odd row returns (the second operand of lane i, its own second operand).


def permlane16_swap(first, second):
    """Per-lane results (new first, new second) of v_permlane16_swap_b32."""
    out = []
    for l in range(64):
        if (l >> 4) % 2 == 0:
            out.append((first[l], first[l + 16]))
        else:
            out.append((second[l - 16], second[l]))
    return out


def test_grad_store_pairs_deliver_whole_chunks():
    # word r (0, 1) of a lane's block holds the vocabulary rows 2 r, 2 r + 1
    # of its four; after the swaps lane group g must hold, in order, the 8
    # rows of chunk SIGMA[g] of the pair's four (chunks of 8 rows, counted
    # from the pair's first row) for its own token column.
    def word(l, h, r):
        v0 = 16 * h + 4 * (l >> 4)   # first row of lane l in block h of the pair
        return ((l & 15), (v0 + 2 * r, v0 + 2 * r + 1))

    s = [permlane16_swap([word(l, 0, r) for l in range(64)], [word(l, 1, r) for l in range(64)]) for r in range(2)]
    for l in range(64):
        stored = [s[0][l][0], s[1][l][0], s[0][l][1], s[1][l][1]]
        assert all(col == (l & 15) for col, _ in stored)
        rows = [v for _, pair in stored for v in pair]
        chunk = SIGMA[l >> 4]
        assert rows == list(range(8 * chunk, 8 * chunk + 8)), (l, rows)
