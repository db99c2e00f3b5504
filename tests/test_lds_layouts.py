"""CPU model of the raw-tile LDS layout of the bfloat16 tile pass (d = 32, 64, 128).

The tile pass copies a raw 32-row K (or V) tile into LDS with direct-to-LDS
loads of 16 bytes per lane, each 1 KB load covering whole rows; lane p of load
i writes LDS byte i*1024 + 16p and fetches the block that an XOR swizzle of
the 16-byte blocks within each row puts there. The matrix-core operands are
then read with ds_read_b128 (K, row layout) and ds_read_b64_tr_b16 (V^T,
transposed layout). This model restates the swizzles of csrc/tile.hip
(raw_swz_k, raw_swz_v) and checks, per lane and value, that the reads deliver
the operands of v_mfma_f32_32x32x16_bf16 as the tile pass uses them, and that
no LDS pass has a bank conflict (64 banks of 4 bytes; 16 lanes per
ds_read_b128 pass, 32 lanes per ds_read_b64 pass). The GPU parity tests check
the kernels themselves (the raw path is bit-identical to the packed one).
"""
import pytest


def swz_k(d, r):
    return {128: r & 15, 64: (r >> 1) & 7, 32: (r >> 2) & 3}[d]


def swz_v(d, r):
    return {128: 4 * (r & 3), 64: ((r >> 1) & 1) << 2, 32: 0}[d]


def offset(d, r, c, swz):
    """LDS byte of element (r, c) of a tile (bf16, d columns)."""
    rb = 2 * d
    return r * rb + (((2 * c) // 16 ^ swz(d, r)) * 16) + (2 * c) % 16


def conflict_ways(addrs, width):
    """Largest number of distinct addresses sharing a bank in one pass."""
    banks = {}
    for a in addrs:
        for b in range(width // 4):
            banks.setdefault((a // 4 + b) % 64, set()).add(a)
    return max(len(v) for v in banks.values())


@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("which", ["k", "v"])
def test_copies_cover_whole_rows_once(d, which):
    swz = swz_k if which == "k" else swz_v
    rb = 2 * d
    sources = set()
    for i in range(32 * rb // 1024):
        rows = set()
        for p in range(64):
            q = i * 1024 + 16 * p
            r, slot = q // rb, (q % rb) // 16
            blk = slot ^ swz(d, r)
            assert 0 <= blk < rb // 16
            rows.add(r)
            sources.add(r * rb + 16 * blk)
            assert offset(d, r, 8 * blk, swz) == q           # the block lands where reads expect it
        assert len(rows) * rb == 1024                         # one load = whole rows
    assert len(sources) == 32 * rb // 16                      # every block copied once


@pytest.mark.parametrize("d", [32, 64, 128])
def test_k_row_operand_reads(d):
    """Chunk s of lane (h, j) = K[j][(d/2)h + 8s .. +7] (16 contiguous bytes);
    no bank conflict in any 16-lane pass."""
    for s in range(d // 16):
        addrs = []
        for lane in range(64):
            h, j = lane // 32, lane % 32
            a = offset(d, j, (d // 2) * h + 8 * s, swz_k)
            for e in range(8):
                assert offset(d, j, (d // 2) * h + 8 * s + e, swz_k) == a + 2 * e
            addrs.append(a)
        for p0 in range(0, 64, 16):
            assert conflict_ways(addrs[p0:p0 + 16], 16) == 1


@pytest.mark.parametrize("d", [32, 64, 128])
def test_v_transposed_operand_reads(d):
    """ds_read_b64_tr_b16: within a group of 16 lanes, lane i receives as value
    k the element i%4 of the 8 bytes addressed by lane 4k + i/4. Each lane
    supplies 4 columns of one row; two reads (rows 8 apart) must give lane
    l = 32h + j the 8 values V[16u + 8(e/4) + 4h + e%4][32t + j], e = 0..7 --
    the key order of the weights in the second product. No bank conflict in
    any 32-lane pass."""
    for u in range(2):
        for t in range(d // 32):
            for half in range(2):
                sup = []
                for lane in range(64):
                    i = lane % 16
                    row = 16 * u + 8 * half + 4 * (lane // 32) + i // 4
                    col = 32 * t + 16 * ((lane // 16) & 1) + 4 * (i % 4)
                    sup.append((row, col, offset(d, row, col, swz_v)))
                for lane in range(64):
                    g0, i = lane - lane % 16, lane % 16
                    for k in range(4):
                        row, col, a = sup[g0 + 4 * k + i // 4]
                        want = (16 * u + 8 * half + 4 * (lane // 32) + k, 32 * t + lane % 32)
                        assert (row, col + i % 4) == want
                        assert offset(d, row, col + i % 4, swz_v) == a + 2 * (i % 4)
                for p0 in range(0, 64, 32):
                    assert conflict_ways([a for _, _, a in sup[p0:p0 + 32]], 8) == 1
                # the address of the second read is the first one's plus 8 rows
                if half == 1:
                    for lane in range(64):
                        i = lane % 16
                        r0 = 16 * u + 4 * (lane // 32) + i // 4
                        c0 = 32 * t + 16 * ((lane // 16) & 1) + 4 * (i % 4)
                        assert offset(d, r0 + 8, c0, swz_v) - offset(d, r0, c0, swz_v) == 8 * 2 * d


def test_d128_copy_offsets_repeat():
    """d = 128: the source offset of copy i less i KB repeats with period 4 in i
    for K (its swizzle depends on the row mod 16, four rows per copy) and is
    the same for every copy for V (row mod 4), so four lane offsets (K) and
    one (V) serve all eight copies of a tile."""
    d, rb = 128, 256

    def src(i, p, swz):
        q = i * 1024 + 16 * p
        r, slot = q // rb, (q % rb) // 16
        return r * rb + 16 * (slot ^ swz(d, r))
    for p in range(64):
        for i in range(8):
            assert src(i, p, swz_k) - 1024 * i == src(i % 4, p, swz_k) - 1024 * (i % 4)
            assert src(i, p, swz_v) - 1024 * i == src(0, p, swz_v)
            assert 0 <= src(i % 4, p, swz_k) - 1024 * (i % 4) < 1024


def test_unswizzled_rows_would_conflict():
    """Without the swizzle the K reads of d = 64 are 8-way conflicted (rows are
    128 bytes apart): the swizzle is what makes them conflict-free."""
    none = lambda d, r: 0
    addrs = [offset(64, lane % 32, 32 * (lane // 32), none) for lane in range(16)]
    assert conflict_ways(addrs, 16) == 8


# ---------------------------------------------------------------------------
# The gradient passes read each raw tile twice: in the row layout
# (ds_read_b128, as K above) and transposed (ds_read_b64_tr_b16, as V above).
# One swizzle serves both (csrc/bwd.hip, raw_swz_b): for d = 128 block b of
# row r sits at b ^ (4 (r & 3) + ((r >> 2) & 3)), for d = 64 at
# b ^ (4 ((r >> 1) & 1) + ((r >> 2) & 3)), for d = 32 at b ^ ((r >> 2) & 3).

def swz_b(d, r):
    if d == 128:
        return 4 * (r & 3) + ((r >> 2) & 3)
    return 4 * ((r >> 1) & 1) + ((r >> 2) & 3) if d == 64 else (r >> 2) & 3


@pytest.mark.parametrize("d", [32, 64, 128])
def test_b_copies_cover_whole_rows_once(d):
    rb = 2 * d
    sources = set()
    for i in range(32 * rb // 1024):
        rows = set()
        for p in range(64):
            q = i * 1024 + 16 * p
            r, slot = q // rb, (q % rb) // 16
            blk = slot ^ swz_b(d, r)
            assert 0 <= blk < rb // 16
            rows.add(r)
            sources.add(r * rb + 16 * blk)
            assert offset(d, r, 8 * blk, swz_b) == q
        assert len(rows) * rb == 1024
    assert len(sources) == 32 * rb // 16
    # the per-lane source offsets repeat with period 4 (d = 128), 2 (d = 64) or
    # 1 (d = 32) in the copy index, up to the 1 KB step of the copy
    period = {128: 4, 64: 2, 32: 1}[d]
    for i in range(period, 32 * rb // 1024):
        for p in range(64):
            def src(ii):
                q = ii * 1024 + 16 * p
                r, slot = q // rb, (q % rb) // 16
                return r * rb + 16 * (slot ^ swz_b(d, r))
            assert src(i) - src(i - period) == period * 1024


@pytest.mark.parametrize("d", [32, 64, 128])
def test_b_row_reads(d):
    """Chunk s of lane (h, j) = X[j][(d/2)h + 8s .. +7], conflict-free."""
    for s in range(d // 16):
        addrs = []
        for lane in range(64):
            h, j = lane // 32, lane % 32
            a = offset(d, j, (d // 2) * h + 8 * s, swz_b)
            for e in range(8):
                assert offset(d, j, (d // 2) * h + 8 * s + e, swz_b) == a + 2 * e
            addrs.append(a)
        for p0 in range(0, 64, 16):
            assert conflict_ways(addrs[p0:p0 + 16], 16) == 1


@pytest.mark.parametrize("d", [32, 64, 128])
def test_b_transposed_reads(d):
    """Transposed chunk (u, t) of lane l = 32h + j: X[16u + 8(s/4) + 4h + s%4]
    [32t + j], s = 0..7, from two transposing reads (half e = s/4). Each lane
    supplies row 4h + (l%16)/4 + 8e (+16u), columns 32t + 16((l/16)&1) +
    4(l%4) .. +3; the address for +16 rows is the one for +0 plus 16 rows'
    bytes (an immediate offset), the two halves need one address each.
    Conflict-free in every 32-lane pass."""
    rb = 2 * d
    for u in range(2):
        for t in range(d // 32):
            for e in range(2):
                sup = []
                for lane in range(64):
                    i = lane % 16
                    row = 16 * u + 8 * e + 4 * (lane // 32) + i // 4
                    col = 32 * t + 16 * ((lane // 16) & 1) + 4 * (i % 4)
                    a = offset(d, row, col, swz_b)
                    assert a == offset(d, row - 16 * u, col, swz_b) + 16 * u * rb
                    for c in range(4):
                        assert offset(d, row, col + c, swz_b) == a + 2 * c
                    sup.append((row, col, a))
                for lane in range(64):
                    g0, i = lane - lane % 16, lane % 16
                    for k in range(4):
                        row, col, _ = sup[g0 + 4 * k + i // 4]
                        assert (row, col + i % 4) == (16 * u + 8 * e + 4 * (lane // 32) + k, 32 * t + lane % 32)
                for p0 in range(0, 64, 32):
                    assert conflict_ways([a for _, _, a in sup[p0:p0 + 32]], 8) == 1


def test_forward_swizzles_do_not_serve_both_reads():
    """Why the gradient passes need their own swizzle: with the forward's K
    swizzle the transposed reads of d = 64 are 2-way conflicted, with its V
    swizzle the row reads are."""
    d = 64
    sup = [offset(d, 4 * (l // 32) + (l % 16) // 4, 16 * ((l // 16) & 1) + 4 * (l % 4), swz_k) for l in range(32)]
    assert conflict_ways(sup, 8) == 2
    addrs = [offset(d, l % 32, 8 * 0, swz_v) for l in range(16)]
    assert conflict_ways(addrs, 16) > 1


# ---------------------------------------------------------------- raw float32 tiles (d <= 64)
def f32v_slot(d, r):
    return 8 * (r >> 3) + 2 * (r & 3) + ((r >> 2) & 1) if d == 32 else r


def f32v_offset(d, r, c):
    """LDS byte of element (r, c) of a raw float32 V tile."""
    return f32v_slot(d, r) * (4 * d) + 16 * ((c >> 2) ^ (8 * ((r >> 2) & 1) if d == 64 else 0)) + 4 * (c & 3)


def f32v_copy_offset(d, i, lane):
    rb = 4 * d
    q = i * 1024 + 16 * lane
    sl, b = q // rb, (q % rb) // 16
    if d == 32:
        return (8 * (sl >> 3) + 4 * (sl & 1) + ((sl >> 1) & 3)) * rb + 16 * b
    return sl * rb + 16 * (b ^ (8 * ((sl >> 2) & 1)))


@pytest.mark.parametrize("d", [32, 64])
def test_f32_k_tile_is_the_bf16_geometry_of_twice_the_width(d):
    """A float32 K tile of d columns has the bytes of a bfloat16 tile of 2d
    columns; element (r, c) sits at the bfloat16 offset of (r, 2c), and the
    row-layout chunk s of lane (h, j), float32 columns (d/2) h + 4s .. + 3,
    is the bfloat16 chunk of the same lane."""
    d2 = 2 * d
    for lane in range(64):
        h, j = lane // 32, lane % 32
        for s_ in range(d // 8):
            a = offset(d2, j, (d2 // 2) * h + 8 * s_, swz_k)
            for e in range(4):
                assert offset(d2, j, 2 * ((d // 2) * h + 4 * s_ + e), swz_k) == a + 4 * e


@pytest.mark.parametrize("d", [32, 64])
def test_f32_v_copies_and_transposed_reads(d):
    """Copies place every 16-byte block of the row-major V tile once where
    f32v_offset expects it (with lane offsets of period 1 or 2 in the copy
    index); chunk (t, a) of lane (h, i) holds V[8a + 4h + e][32t + i], e < 4,
    read with two ds_read2st64_b32 from one address per column tile at
    offsets of 256 bytes, each dword pass over 64 lanes hitting 64 banks."""
    rb = 4 * d
    seen = set()
    for i in range(32 * rb // 1024):
        for lane in range(64):
            src = f32v_copy_offset(d, i, lane)
            r, c = src // rb, (src % rb) // 4
            assert 0 <= src and src + 16 <= 32 * rb             # inside the block's V tile
            assert f32v_offset(d, r, c) == i * 1024 + 16 * lane
            per = 1 if d == 32 else 2
            assert src - i * 1024 == f32v_copy_offset(d, i % per, lane) - (i % per) * 1024
            seen.add(src)
    assert len(seen) == 32 * rb // 16
    k64 = 4 if d == 32 else 8
    for t in range(d // 32):
        for a in range(4):
            for e0 in (0, 2):
                for e in (e0, e0 + 1):
                    addrs = []
                    for lane in range(64):
                        h, i = lane // 32, lane % 32
                        base = f32v_offset(d, 4 * h, 32 * t + i)
                        got = base + 256 * (k64 * a + e)
                        assert got == f32v_offset(d, 8 * a + 4 * h + e, 32 * t + i)
                        addrs.append(got)
                    assert conflict_ways(addrs, 4) == 1
