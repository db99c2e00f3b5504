"""CPU models of the kernels' index and bounds arithmetic (no GPU).

Each test restates the index math of one kernel from the HIP sources and
checks, exhaustively over the lanes, copies and sizes it uses, that every
global and LDS access stays inside its buffer or LDS region and that work is
covered exactly once:
* xcd_remap (common.h): a permutation of the workgroups, each XCD receiving a
  contiguous range;
* pool_kernel (pool.hip): two threads per 16-byte column chunk of a 32-row
  block, the second half's partner lane inside the same wave, reads and
  writes inside the tensors;
* the raw-tile copies and operand reads of tile_stream_kernel (tile.hip,
  tile_ops.h): buffer-load offsets inside the copied block (the scalar offset
  is outside the hardware range check, so this is the bound that matters),
  the period of the lanes' copy offsets the kernel relies on, LDS writes and
  reads inside the wave's slot, and the workgroup's LDS within the budget of
  its occupancy;
* rows_kernel (select.hip): the score/weight rows, the partial sums of the
  coarse term and the float64 query rows inside the dynamic LDS it requests,
  for every register tier, head dim and mode, within 160 KB; the coarse
  term's V~ buffer loads (vector plus immediate offsets; reads past the head's
  rows come back as zero, so an offset at or past the buffer's size must
  belong to a block past nb);
* the backward's coarse passes (bwd.hip): the column pass's dim groups (every
  output dim once, 16-byte aligned loads and stores) and its buffer-load
  offsets, the row pass's K~/V~ buffer-load offsets;
* the backward's column lists: the batched bitmap-word reads stay in the
  head's bitmap;
* the head-wide selection's register tier (select_global.hip): its three
  radix passes of 12, 10 and 10 bits with the block-wide digit pick find the
  budget-th largest key and the number of ties to take (against sorting).
"""
import pytest

LDS_PER_CU = 160 * 1024


# ------------------------------------------------------------------ common.h
def xcd_remap(p, total, xcds=8):
    xcd, slot = p % xcds, p // xcds
    q, r = total // xcds, total % xcds
    return xcd * (q + 1) + slot if xcd < r else r * (q + 1) + (xcd - r) * q + slot


@pytest.mark.parametrize("total", [1, 7, 8, 9, 64, 100, 1023, 1024, 1536, 3072, 4099])
def test_xcd_remap_is_a_permutation_with_contiguous_ranges(total):
    logical = [xcd_remap(p, total) for p in range(total)]
    assert sorted(logical) == list(range(total))
    for x in range(8):
        mine = sorted(logical[p] for p in range(x, total, 8))
        if mine:
            assert mine == list(range(mine[0], mine[0] + len(mine)))


# ------------------------------------------------------------------ pool.hip
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [32, 64, 128])
def test_pool_thread_map(dtype, d):
    per = 8 if dtype == "bf16" else 4
    bh, n = 3, 160
    cpr = d // per
    chunks = bh * (n // 32) * cpr
    threads = 256
    blocks = (2 * chunks + threads - 1) // threads
    covered = {}
    rows_total = bh * n
    for t in range(blocks * threads):
        blk = t // (2 * cpr)
        i = t - blk * 2 * cpr
        half, c = i // cpr, i % cpr
        if t >= 2 * chunks:
            continue
        row0 = blk * 32 + 16 * half
        for r in range(16):
            u = (row0 + r) * cpr + c                    # 16-byte unit read
            assert 0 <= u < rows_total * cpr
        if half == 0:
            partner = t + cpr
            assert partner // 64 == t // 64             # the shuffle stays in the wave
            pb = partner // (2 * cpr)
            assert pb == blk and (partner - pb * 2 * cpr) // cpr == 1 and (partner - pb * 2 * cpr) % cpr == c
            lo, hi = blk * d + c * per, blk * d + c * per + per
            assert 0 <= lo and hi <= bh * (n // 32) * d
            for e in range(lo, hi):
                assert e not in covered
                covered[e] = t
    assert len(covered) == bh * (n // 32) * d


# ------------------------------------------------------------------ tile.hip (raw bf16 tiles)
def swz_k(d, r):
    return {128: r & 15, 64: (r >> 1) & 7, 32: (r >> 2) & 3}[d]


def swz_v(d, r):
    return {128: 4 * (r & 3), 64: ((r >> 1) & 1) << 2, 32: 0}[d]


def raw_offset(d, swz, r, c):
    return r * (2 * d) + ((((2 * c) >> 4) ^ swz(d, r)) << 4) + ((2 * c) & 15)


def raw_copy_offset(d, swz, i, lane):
    q = i * 1024 + 16 * lane
    r, blk = q // (2 * d), (q % (2 * d)) // 16
    return r * (2 * d) + ((blk ^ swz(d, r)) << 4)


def tile_cfg(d):
    kc = d // 16                    # 16-byte row-layout chunks (= 1 KB copies of a K tile)
    nt = d // 32
    vc = 2 * nt
    return kc, vc, kc + vc, nt


@pytest.mark.parametrize("d", [32, 64, 128])
def test_raw_tile_copies_stay_in_the_block(d):
    """Copy i of block y: scalar offset y*KC*1K + i*1K, vector offset the
    lane's swizzled source offset of copy i mod period, minus its own copy's
    1 KB step. The sum must be the lane's source inside block y for every
    copy (this is what keeps the loads in bounds: the scalar offset is not
    range-checked), and the LDS destination inside the slot."""
    kc, vc, ch, nt = tile_cfg(d)
    kpb = {128: 4, 64: 2, 32: 1}[d]
    tile = kc * 1024
    for nb in (1, 3, 128):
        for y in (0, nb - 1):
            for i in range(kc):
                for lane in range(64):
                    koff = raw_copy_offset(d, swz_k, i % kpb, lane) - (i % kpb) * 1024
                    src = y * tile + i * 1024 + koff
                    assert src == y * tile + raw_copy_offset(d, swz_k, i, lane)
                    assert y * tile <= src and src + 16 <= (y + 1) * tile <= nb * tile
                    voff = raw_copy_offset(d, swz_v, 0, lane)
                    vsrc = y * tile + i * 1024 + voff
                    assert vsrc == y * tile + raw_copy_offset(d, swz_v, i, lane)
                    assert y * tile <= vsrc and vsrc + 16 <= (y + 1) * tile
                    assert i * 1024 + 16 * lane + 16 <= kc * 1024        # K part of the slot
                    assert kc * 1024 + i * 1024 + 16 * lane + 16 <= ch * 1024


@pytest.mark.parametrize("d", [32, 64, 128])
def test_raw_tile_operand_reads_stay_in_the_slot(d):
    kc, vc, ch, nt = tile_cfg(d)
    rb = 2 * d
    for lane in range(64):
        h, j, i16 = lane >> 5, lane & 31, lane & 15
        for c in range(kc):
            a = raw_offset(d, swz_k, j, (d // 2) * h + 8 * c)
            assert 0 <= a and a + 16 <= kc * 1024
        for t in range(nt):
            vr = kc * 1024 + raw_offset(d, swz_v, 4 * h + i16 // 4, 32 * t + 16 * ((lane >> 4) & 1) + 4 * (i16 & 3))
            for cc in range(vc):
                u = cc // nt
                for imm in (16 * u * rb, (16 * u + 8) * rb):   # the two transposing reads of a chunk
                    assert kc * 1024 <= vr + imm and vr + imm + 8 <= ch * 1024


@pytest.mark.parametrize("d,waves_per_cu,m", [(32, 16, 8), (64, 16, 16), (64, 16, 64), (128, 8, 32), (128, 8, 128)])
def test_tile_stream_lds_fits_its_occupancy(d, waves_per_cu, m):
    """tile_stream_kernel: 4 waves per workgroup, one slot of CH KB per wave
    plus the waves' selection lists (m ints each); the workgroups a CU holds
    at the kernel's occupancy (16 waves for d <= 64, 8 for d = 128, set by
    registers) must fit its LDS."""
    kc, vc, ch, nt = tile_cfg(d)
    waves, slots = 4, 1
    per_wg = waves * slots * ch * 1024 + waves * m * 4
    assert (waves_per_cu // waves) * per_wg <= LDS_PER_CU


# ------------------------------------------------------------------ select.hip (rows_kernel)
K_ROWS, K_CHUNK, K_U = 16, 64, 8


def rows_smem(jmax, nw, mode, d):
    if mode == 0:
        return 0, 0
    ldc = 64 * jmax
    part_off = (K_ROWS * ldc * 4 + 15) & ~15
    part = nw * 16 * 16 * 4 if mode in (1, 2) else 0
    qd = K_ROWS * d * 8 if mode in (2, 3) else 0
    return part_off, part_off + max(part, qd)


def rows_col(r, c):
    return c ^ ((r & 15) << 2)


def rows_qcol(r, c):
    return c ^ ((r & 15) << 1)


def rows_rpw(jmax):
    return 2 if jmax <= 16 else 1


@pytest.mark.parametrize("jmax", [2, 8, 16, 32])
@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("mode", [1, 2, 3])
def test_rows_kernel_lds_regions(jmax, d, mode):
    rpw = rows_rpw(jmax)
    nw = K_ROWS // rpw
    ntd = d // 16
    kq = nw // ntd
    assert kq >= 1 and nw % ntd == 0
    bpw = 2 * jmax // kq
    assert bpw * kq == 2 * jmax
    ldc = 64 * jmax
    part_off, total = rows_smem(jmax, nw, mode, d)
    assert total <= LDS_PER_CU
    if jmax <= 16:
        assert 2 * total <= LDS_PER_CU                   # two workgroups per CU
    # score / weight rows: row r < 16, column c < 64 JMAX, stored at c ^ 4r,
    # a permutation of the row's columns inside each group of 64
    for r in range(K_ROWS):
        cols = [rows_col(r, c) for c in range(64 * jmax)]
        assert sorted(cols) == list(range(64 * jmax))
        assert all(cc // 64 == c // 64 for c, cc in enumerate(cols))
    assert (K_ROWS - 1) * ldc + 64 * jmax - 1 < part_off // 4
    if mode in (1, 2):
        # partial sums part[(kq' * 16 + 4 ak + e) * D + 16 nt + ar]
        top = ((kq - 1) * K_ROWS + 4 * 3 + 3) * d + 16 * (ntd - 1) + 15
        assert part_off + 4 * (top + 1) <= total
        # phase 4's weight reads: two 16-byte reads per batch u < BPW
        for kqi in range(kq):
            for u in range(bpw):
                for ak in range(4):
                    col = K_U * ak + 4 * K_U * (kqi + kq * u)
                    assert col + 8 <= 64 * jmax          # inside the row (zero past nb)
                    for ar in range(K_ROWS):
                        c0 = rows_col(ar, col)         # the two 16-byte reads: c0, c0 ^ 4
                        assert c0 % 4 == 0
                        assert [c0 + i for i in range(4)] == [rows_col(ar, col + i) for i in range(4)]
                        assert [(c0 ^ 4) + i for i in range(4)] == [rows_col(ar, col + 4 + i) for i in range(4)]
    if mode in (2, 3):
        assert part_off + K_ROWS * d * 8 <= total
        # the float64 query rows: column c of row r at c ^ 2r (a permutation of
        # the row); a lane reads pairs (c0 + 16 s) ^ x and that ^ 2 for
        # c0 = 4g, g < 4
        for r in range(K_ROWS):
            assert sorted(rows_qcol(r, c) for c in range(d)) == list(range(d))
            x = rows_qcol(r, 0)
            for g in range(4):
                for s16 in range(d // 16):
                    c = (4 * g + 16 * s16) ^ x
                    assert c % 2 == 0 and c + 1 < d
                    assert [c, c + 1] == [rows_qcol(r, 4 * g + 16 * s16), rows_qcol(r, 4 * g + 16 * s16 + 1)]
                    assert [c ^ 2, (c ^ 2) + 1] == [rows_qcol(r, 4 * g + 16 * s16 + 2), rows_qcol(r, 4 * g + 16 * s16 + 3)]


# ------------------------------------------------------------------ select.hip: the coarse term's V~ loads
@pytest.mark.parametrize("jmax", [2, 8, 16, 32])
@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("nb", [1, 33, 100, 128])
def test_coarse_term_v_loads(jmax, d, nb):
    """vo = ((4 kU kq + kU ak) d + 16 nt + ar) 4 + u 4 kU KQ d 4 + e d 4: the
    immediate part (e d 4) fits the 12-bit field, every (block, dim) of the 64
    JMAX columns is read once per dim tile, and an offset at or past nb d 4
    (zero from the hardware) is a block past nb."""
    nb = min(nb, 64 * jmax)
    rpw = rows_rpw(jmax)
    nw = K_ROWS // rpw
    ntd = d // 16
    kq_n = nw // ntd
    bpw = 2 * jmax // kq_n
    ku = 8
    assert 7 * d * 4 < 4096                       # immediate offset field
    seen = set()
    for w in range(nw):
        nt, kq = w % ntd, w // ntd
        for lane in range(64):
            ar, ak = lane & 15, lane >> 4
            vlane = ((4 * ku * kq + ku * ak) * d + 16 * nt + ar) * 4
            for u in range(bpw):
                vo = vlane + u * (4 * ku * kq_n * d * 4)
                for e in range(ku):
                    off = vo + e * d * 4
                    block, dim = divmod(off // 4, d)
                    assert off % 4 == 0 and dim == 16 * nt + ar
                    assert block == 4 * ku * (kq + kq_n * u) + ku * ak + e
                    if off >= nb * d * 4:
                        assert block >= nb
                    seen.add((block, dim))
    assert seen == {(y, c) for y in range(64 * jmax) for c in range(d)}


# ------------------------------------------------------------------ bwd.hip: the coarse passes
def cols_cfg(d):
    tw = min(4, d // 16)
    groups = d // (16 * tw)
    return tw, groups, 2 * groups


@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("nb", [1, 5, 66, 128])
def test_column_pass_dim_groups_and_loads(d, nb):
    """Wave (kind, group dg), lane (lr, lg): dims d0 + t, d0 = 16 TW dg + TW lr;
    every output (row yy of the 16, dim) of each quantity once; the 16-byte
    loads and stores aligned; reads at or past the head's buffer (zero from the
    hardware) are exactly those of block-rows past nb."""
    tw, groups, waves = cols_cfg(d)
    assert 16 * tw * groups == d
    batch = 8
    for y0 in range(0, nb, 16):
        outs = set()
        for w in range(waves):
            kind, dg = w // groups, w % groups
            for lane in range(64):
                lr, lg = lane & 15, lane >> 4
                y = y0 + lr
                d0 = 16 * tw * dg + tw * lr
                assert (d0 * 4) % (4 * tw) == 0
                ao, bo = (lg * nb + y) * 4, (lg * d + d0) * 4
                for xs in range(0, nb, 4 * batch):
                    for u in range(batch):
                        x = xs + 4 * u + lg
                        a_off = ao + u * 4 * nb * 4
                        b_off = bo + u * 4 * d * 4
                        assert a_off == (x * nb + y) * 4 and b_off == (x * d + d0) * 4
                        # a lane of a column y < nb (its products reach stored
                        # rows) reads the real value for x < nb and zero past
                        # the head's rows; columns y >= nb feed rows not stored
                        if y < nb:
                            assert (a_off < nb * nb * 4) == (x < nb)
                        assert (b_off < nb * d * 4) == (x < nb)
                    ao += 4 * batch * nb * 4
                    bo += 4 * batch * d * 4
                for r in range(4):
                    yy = y0 + 4 * lg + r
                    if yy < nb:
                        for t in range(tw):
                            outs.add((kind, yy, d0 + t))
        assert outs == {(k, yy, c) for k in (0, 1) for yy in range(y0, min(y0 + 16, nb)) for c in range(d)}


@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("nb", [1, 66, 128, 300])
def test_row_pass_coarse_loads(d, nb):
    """Step 1 reads K~/V~ rows y0 + 16 t + lr, dims 16 u + 4 lg (16 bytes);
    step 3 reads K~[y0 + kq YK + 4 s + lg][16 nt + lr]; offsets at or past
    nb d 4 (zero from the hardware) are rows past nb; immediates fit."""
    yc, rows_wg = 128, 16
    ntd = d // 16
    kq_n = rows_wg // ntd
    yk = yc // kq_n
    assert 16 * (d // 16 - 1) * 4 < 4096
    for w in range(rows_wg):
        t = w & 7
        nt, kq = w % ntd, w // ntd
        for lane in range(64):
            lr, lg = lane & 15, lane >> 4
            b1 = ((16 * t + lr) * d + 4 * lg) * 4
            b3 = ((kq * yk + lg) * d + 16 * nt + lr) * 4
            for y0 in range(0, nb, yc):
                ystep = y0 * d * 4
                for u in range(d // 16):
                    off = b1 + ystep + 16 * u * 4
                    row = off // 4 // d
                    assert row == y0 + 16 * t + lr and off % 16 == 0
                    if off >= nb * d * 4:
                        assert row >= nb
                for s_ in range(yk // 4):
                    off = b3 + ystep + 4 * s_ * d * 4
                    row, dim = divmod(off // 4, d)
                    assert row == y0 + kq * yk + 4 * s_ + lg and dim == 16 * nt + lr
                    if off >= nb * d * 4:
                        assert row >= nb


@pytest.mark.parametrize("nb", [1, 63, 64, 66, 511, 512, 513, 1024, 2048])
def test_column_list_bitmap_reads(nb):
    """Batches of 8 x 64 rows; row x = min(x0 + 64 u + lane, nb - 1) reads word
    x nbw + y / 32 of the head's bitmap; rows past nb are dropped."""
    nbw = (nb + 31) // 32
    listed = []
    for y in {0, nb // 2, nb - 1}:
        listed = []
        for x0 in range(0, nb, 8 * 64):
            for u in range(8):
                for lane in range(64):
                    xr = x0 + 64 * u + lane
                    x = min(xr, nb - 1)
                    word = x * nbw + y // 32
                    assert 0 <= word < nb * nbw
                    if xr < nb:
                        listed.append(xr)
        assert listed == list(range(nb))


# ------------------------------------------------------------------ select_global.hip: register-tier radix passes
def pick_digit_block(hist, bins, remaining, threads=1024):
    """Thread t sums bins bins-1-t*per .. bins-(t+1)*per (descending); the thread
    whose exclusive..inclusive prefix holds `remaining` picks the digit."""
    per = bins // threads
    found = []
    incl = 0
    for t in range(threads):
        top = bins - 1 - t * per
        c = [hist[top - e] for e in range(per)]
        excl, incl = incl, incl + sum(c)
        if excl < remaining <= incl:
            acc = excl
            for e in range(per):
                if acc + c[e] >= remaining:
                    found.append((top - e, acc))
                    break
                acc += c[e]
    assert len(found) == 1                        # exactly one thread
    return found[0]


def radix_threshold(keys, budget):
    """The kernel's three passes of 12, 10 and 10 bits over the non-zero keys:
    the budget-th largest key T and how many keys equal to T to take."""
    prefix, remaining = 0, budget
    for shift, bits in ((20, 12), (10, 10), (0, 10)):
        bins = 1 << bits
        hi_mask = 0 if shift == 20 else (~((1 << (shift + bits)) - 1)) & 0xFFFFFFFF
        hist = [0] * bins
        for k in keys:
            if k != 0 and (k & hi_mask) == (prefix & hi_mask):
                hist[(k >> shift) & (bins - 1)] += 1
        digit, before = pick_digit_block(hist, bins, remaining)
        prefix |= digit << shift
        remaining -= before
    return prefix, remaining


@pytest.mark.parametrize("case", range(8))
def test_head_wide_radix_passes(case):
    import random
    rng = random.Random(case)
    n = rng.choice([16, 100, 1000, 4096])
    if case % 4 == 0:       # heavy ties
        keys = [rng.choice([0x80000000, 0xC0000000, 0xBF800000, 0x3F7FFFFF]) for _ in range(n)]
    elif case % 4 == 1:     # one exponent range (most keys share the top 12 bits)
        keys = [0xC0000000 | rng.getrandbits(20) for _ in range(n)]
    else:                   # anything non-zero
        keys = [rng.getrandbits(32) | 1 for _ in range(n)]
    keys += [0] * rng.randint(0, 5)            # blocks that do not take part
    nz = sorted((k for k in keys if k), reverse=True)
    for budget in sorted({1, len(nz) // 3 or 1, len(nz) - 1 or 1}):
        if budget >= len(nz):
            continue
        T, need = radix_threshold(keys, budget)
        assert T == nz[budget - 1]
        assert need == budget - sum(1 for k in nz if k > T) and need >= 1
