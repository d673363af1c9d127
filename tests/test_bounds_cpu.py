"""Every address the kernels form stays inside its buffer, whatever the hardware's range checks do.

For each launch of the plan (the five heads and small edge shapes, at several valid-token counts
Nv), this test recomputes, from the layout lce_plan_info reports, the largest byte offset that
each kernel's loads, stores and read-modify-writes can form and checks it against the size of
the region (workspace) or of the caller's tensor it addresses. The arithmetic follows the
kernels' index expressions:

* tiles are 384 x 256 (D % 64 == 0: 12 waves) or 256 x 256 (other widths: 8 waves); the rows of
  the last vocabulary tile past V are loaded through the out-of-range offset (zeros, no address),
  so the W rows addressed are those below V;
* K-major operands send the lanes whose columns lie past D (the hidden width) to the same offset;
* dH runs K over the slab's vs ids (a ragged last slice masks the rest), split into 1 to 8 parts;
* G and the dH accumulators hold rows_g rows, the 384-row tiles of the last token rows included;
* the dW / AdamW epilogues touch only the rows of the slab that exist.

Accesses sent to the out-of-range offset form no address and are not counted. No GPU is needed.
"""
import pytest

from paper_2605_21442_amd import binding as B

HEADS = [(256, 512, 4096), (8192, 2048, 128256), (16384, 4096, 128256), (32768, 3584, 152064),
         (16384, 8192, 128256)]
EDGES = [(1, 8, 5), (300, 264, 1000), (257, 64, 9000), (513, 520, 300), (300, 64, 12300), (200, 128, 12289),
         (768, 128, 1536), (520, 64, 40000), (33, 72, 1), (16385, 64, 383), (1000, 136, 385)]


def cdiv(a, b):
    return -(-a // b)


def rup(a, b):
    return cdiv(a, b) * b


class Extents:
    """Largest byte (exclusive end) formed in each buffer, against the buffer's size."""

    def __init__(self):
        self.ends = {}

    def touch(self, buf, end):
        self.ends[buf] = max(self.ends.get(buf, 0), end)

    def check(self, sizes, where):
        for buf, end in self.ends.items():
            assert end <= sizes[buf], f"{where}: {buf} reaches byte {end} of {sizes[buf]}"


def dh_tail_parts(nv, d, acc_rows):
    """The K parts z >= 1 of the tail tiles of a dH launch the host did not split, as the kernel
    assigns them: (xcd, first row of the tile, z, parts of the tile, slot)."""
    tm_live, dtc = cdiv(nv, 384), cdiv(d, 256)
    t = tm_live * dtc

    def c0(x):
        return (x * t) >> 3

    def parts(nt):
        return min(8, 32 // nt) if 0 < nt <= 16 else 1

    tails = [(c0(x + 1) - c0(x)) & 31 for x in range(8)]
    if sum((parts(nt) - 1) * nt for nt in tails) * 384 * 256 > (acc_rows - tm_live * 384) * d:
        return []
    out, slot0 = [], 0
    for x in range(8):
        n = c0(x + 1) - c0(x)
        nmain, nt = n & ~31, n & 31
        kz = parts(nt)
        for z in range(1, kz):
            for ti in range(nt):
                l = c0(x) + nmain + ti
                band, = divmod(l, 4 * dtc)[:1]
                r0 = band * 4
                rows = min(4, tm_live - r0)
                tm = r0 + (l - band * 4 * dtc) % rows
                out.append((x, tm * 384, z, kz, slot0 + (z - 1) * nt + ti))
        slot0 += (kz - 1) * nt
    return out


def walk(n, d, v, nv, ld_h=None, ld_w=None):
    """Extents of one lce_forward + lce_backward of an [n, d] x [v, d] problem with nv valid rows."""
    ld_h = ld_h or d
    ld_w = ld_w or d
    info = B.lce_plan_info(B.problem(n, d, v, ld_h=ld_h, ld_w=ld_w))
    npad, rows_g, vc, nslab = info["npad"], info["rows_g"], info["vc"], info["nslab"]
    e = Extents()
    # caller tensors: the last row holds only d elements of its stride
    sizes = {"H": 2 * ((n - 1) * ld_h + d) if n else 0, "W": 2 * ((v - 1) * ld_w + d),
             "dH": 2 * n * d, "dW": 2 * v * d, "lse": 4 * n, "targets": 4 * n,
             "idx": 4 * npad, "pos": 4 * npad, "hv": 2 * npad * d,
             "pm": 4 * info["part_rows"] * npad, "ps": 4 * info["part_rows"] * npad, "terms": 4 * npad,
             "G": 2 * rows_g * vc, "dh32": 4 * rows_g * d * info["dh_kz"]}
    twelve = d % 64 == 0
    tm_rows = 384 if twelve else 256          # vocabulary (A) rows of a forward / G tile

    # compaction: idx[0..nv), pos[0..n), the targets
    if nv:
        e.touch("idx", 4 * nv)
    e.touch("pos", 4 * n)
    e.touch("targets", 4 * n)

    def w_rows(v0, rows):
        # rows [v0, v0 + rows) of W, full K (the rows past V of a last tile are masked)
        last = min(v0 + rows, v) - 1
        e.touch("W", 2 * (last * ld_w + d))

    # forward statistics
    if nv:
        if twelve and info["fwd_gathers"]:
            e.touch("hv", 2 * rup(nv, 64) * d)                      # gather, zero rows to a multiple of 64
            for n0 in range(0, nv, 256):
                e.touch("hv", 2 * (n0 + 256) * d)                   # B: 256 dense rows of Hv
            for v0 in range(0, v, 384):
                w_rows(v0, 384)
            vt3 = cdiv(v, 384)
            if info["fwd_one_launch"]:
                e.touch("pm", 4 * ((vt3 - 1) * npad + nv))
            else:
                gw = vc // 384
                e.touch("pm", 4 * (2 * gw * npad + nv))             # running pair after the two row sets
        else:
            e.touch("H", 2 * ((n - 1) * ld_h + d))                  # rows gathered through idx (< n)
            for v0 in range(0, v, 256):
                w_rows(v0, 256)
            e.touch("pm", 4 * ((2 * min(cdiv(v, 256), 32) - 1) * npad + nv))
        e.touch("ps", e.ends["pm"])
        e.touch("terms", 4 * nv)
        e.touch("lse", 4 * n)

    # backward
    if nv:
        e.touch("hv", 2 * rup(nv, 64) * d)
    dh_kz = info["dh_kz"]
    for s in range(nslab):
        v0 = s * vc
        vs = min(vc, v - v0)
        if not nv:
            continue
        # G tiles: W rows v0 + [vt0, vt0 + tm_rows) (masked past V), Hv / gathered H rows, G written whole
        for vt0 in range(0, vs, tm_rows):
            w_rows(v0 + vt0, tm_rows)
            for n0 in range(0, nv, 256):
                if twelve:
                    e.touch("hv", 2 * (n0 + 256) * d)
                e.touch("G", 2 * ((n0 + 255) * vc + vt0 + tm_rows))
        # dH: 384-row tiles of G rows, K over [k0, k0 + kzn), W slab rows v0 + k (< v0 + vs), columns < d
        kt = rup(vs, 64)

        def dh_part(m0, z, kz, acc_end):
            kh = rup(cdiv(kt, kz), 64)
            k0 = z * kh
            kzn = min(vs - k0, kh)
            e.touch("dh32", acc_end)            # read-modify-write of the part's accumulator block
            if kzn > 0:
                e.touch("G", 2 * ((m0 + 383) * vc + k0 + kzn))
                w_rows(v0 + k0, kzn)

        if dh_kz > 1:
            for z in range(dh_kz):
                for m0 in range(0, nv, 384):
                    # the tile's rows in accumulator z (the parts follow each other)
                    dh_part(m0, z, dh_kz, 4 * (z * rows_g + m0 + 384) * d)
        else:
            # device-side split of each XCD's last partial round (dh_tile): part 0 in the tile's rows,
            # parts z >= 1 in 384 x 256 slots after row tm_live * 384
            tm_live, dtc = cdiv(nv, 384), cdiv(d, 256)
            for m0 in range(0, nv, 384):
                dh_part(m0, 0, 1, 4 * (m0 + 384) * d)
            for x, m0, z, kz, slot in dh_tail_parts(nv, d, rows_g):
                dh_part(m0, z, kz, 4 * (tm_live * 384 * d + (slot + 1) * 384 * 256))
        # dW: G and Hv read K-major over round_up(Nv, 64) token rows; dW rows of the slab only
        kpad = rup(nv, 64)
        for m0 in range(0, vs, 384):
            e.touch("G", 2 * ((kpad - 1) * vc + m0 + 384))
            e.touch("dW", 2 * (v0 + min(vs, m0 + 384)) * d)
        e.touch("hv", 2 * ((kpad - 1) * d + d))
    e.touch("dH", 2 * n * d)
    return e, sizes, info


CASES = [(n, d, v, nv) for (n, d, v) in HEADS + EDGES
         for nv in sorted({0, 1, max(n // 2, 1), max(n - 1, 0), n}) if nv <= n]


@pytest.mark.parametrize("n,d,v,nv", CASES)
def test_no_access_leaves_its_buffer(n, d, v, nv):
    e, sizes, _ = walk(n, d, v, nv)
    e.check(sizes, f"n={n} d={d} v={v} nv={nv}")


@pytest.mark.parametrize("n,d,v", [(300, 64, 1000), (1000, 136, 385), (16384, 4096, 128256)])
def test_no_access_leaves_its_buffer_with_row_strides(n, d, v):
    for nv in (1, n):
        e, sizes, _ = walk(n, d, v, nv, ld_h=d + 64, ld_w=d + 8)
        e.check(sizes, f"strided n={n} d={d} v={v} nv={nv}")


@pytest.mark.parametrize("n,d,v", HEADS + EDGES)
def test_workspace_regions_are_disjoint_and_inside_the_workspace(n, d, v):
    info = B.lce_plan_info(B.problem(n, d, v))
    npad, rows_g, vc = info["npad"], info["rows_g"], info["vc"]
    prefix = [("idx", info["o_idx"], 4 * npad), ("pos", info["o_pos"], 4 * npad), ("nv", info["o_nv"], 4),
              ("hv", info["o_hv"], 2 * npad * d)]
    fwd = prefix + [("pm", info["o_pm"], 4 * info["part_rows"] * npad), ("ps", info["o_ps"], 4 * info["part_rows"] * npad),
                    ("terms", info["o_terms"], 4 * npad)]
    bwd = prefix + [("G", info["o_g"], 2 * rows_g * vc), ("dh32", info["o_dh32"], 4 * rows_g * d * info["dh_kz"])]
    assert 1 <= info["dh_kz"] <= 8
    assert info["o_dh32b"] == (info["o_dh32"] + 4 * rows_g * d if info["dh_kz"] > 1 else 0)
    assert rows_g % 384 == 0 and rows_g >= npad and npad % 256 == 0 and npad >= n
    assert vc % 768 == 0
    for regions, total in ((fwd, info["fwd_bytes"]), (bwd, info["bwd_bytes"])):
        regions = sorted(regions, key=lambda r: r[1])
        for (a, oa, sa), (b, ob, sb) in zip(regions, regions[1:]):
            assert oa + sa <= ob, f"{a} overlaps {b}"
        for name, o, size in regions:
            assert o % 256 == 0, name
        assert regions[-1][1] + regions[-1][2] <= total


@pytest.mark.parametrize("n,d,v", HEADS + EDGES)
def test_in_tile_offsets_fit_a_buffer_resource(n, d, v):
    # buffer resources hold at most 2^31 - 1 bytes; every tile's offsets from its resource base
    # (a W tile, a G tile row block, a dH accumulator tile, a 64-row K slice) stay below that
    info = B.lce_plan_info(B.problem(n, d, v))
    vc = info["vc"]
    lim = 2 ** 31 - 1
    assert 384 * d * 2 <= lim                      # W / Hv tile
    assert 256 * vc * 2 <= lim                     # G rows of one token tile
    assert 384 * d * 4 <= lim                      # dH accumulator tile
    assert 64 * max(d, vc) * 2 <= lim              # one K-major slice


def test_the_walk_flags_regions_sized_to_npad_rows():
    # with G and the dH accumulators sized to Npad rows (not the 384-row tile grid), the dH tiles of
    # the last token rows of the 8B head with every token valid reach past them
    e, sizes, info = walk(16384, 4096, 128256, 16384)
    assert info["rows_g"] > info["npad"]
    for buf, row_bytes in (("G", 2 * info["vc"]), ("dh32", 4 * 4096 * info["dh_kz"])):
        short = dict(sizes)
        short[buf] = info["npad"] * row_bytes
        with pytest.raises(AssertionError, match=buf):
            e.check(short, "npad rows")


@pytest.mark.parametrize("n,d,v,nv", [(12288, 2048, 1000, 300), (12288, 2048, 1000, 1400), (12288, 2048, 1000, 3686),
                                      (12288, 2048, 1000, 4423), (8192, 4096, 1000, 6209),
                                      (32768, 3584, 152064, 22936), (16384, 8192, 128256, 13107)])
def test_split_dh_tails_stay_inside_the_accumulator(n, d, v, nv):
    # the shapes whose dH tails the kernel splits on the device (and one whose tails do not fit)
    e, sizes, info = walk(n, d, v, nv)
    e.check(sizes, f"n={n} d={d} v={v} nv={nv}")
    parts = dh_tail_parts(nv, d, info["rows_g"])
    slots = sorted(p[4] for p in parts)
    assert slots == list(range(len(slots)))            # numbered densely, each once
    tm_live = cdiv(nv, 384)
    assert len(slots) * 384 * 256 <= (info["rows_g"] - tm_live * 384) * d


@pytest.mark.parametrize("nv,d", [(300, 2048), (3686, 2048), (22936, 3584), (13107, 8192), (12288, 4096), (1, 64)])
def test_split_dh_blocks_cover_every_tile_and_k_part_once(nv, d):
    # the blocks of a launch the host did not split, as dh_tile maps them: every live tile once,
    # with parts 0 .. kz - 1 of one kz
    tm_live, dtc = cdiv(nv, 384), cdiv(d, 256)
    t = tm_live * dtc
    rows_g = rup(rup(max(nv, 1), 256), 384) + 384 * 64
    tails = {(p[1] // 384, p[2]): p[3] for p in dh_tail_parts(nv, d, rows_g)}
    seen = {}
    for x in range(8):
        c0, c1 = (x * t) >> 3, ((x + 1) * t) >> 3
        for l in range(c0, c1):
            band = l // (4 * dtc)
            rows = min(4, tm_live - band * 4)
            k = l - band * 4 * dtc
            seen.setdefault((band * 4 + k % rows, k // rows), set()).add(0)
    assert sorted(seen) == sorted((tm, tn) for tm in range(tm_live) for tn in range(dtc))
    for (tm, z), kz in tails.items():
        assert 1 <= z < kz <= 8


def dw_block_tile(blk, tm_count, d):
    """The dW tile of block blk as dw_tile maps it (None: the block has no tile): the slab's
    tm_count x ceil(D / 256) tiles cut evenly over the 8 XCDs, bands of 4 row tiles walked column
    by column."""
    dtc = cdiv(d, 256)
    t = tm_count * dtc
    x, k = blk & 7, blk >> 3
    c0, c1 = (x * t) >> 3, ((x + 1) * t) >> 3
    if k >= c1 - c0:
        return None
    l = c0 + k
    band = l // (4 * dtc)
    rows = min(4, tm_count - band * 4)
    kk = l - band * 4 * dtc
    return band * 4 + kk % rows, kk // rows


@pytest.mark.parametrize("tm_count,d", [(48, 4096), (54, 3584), (18, 3584), (64, 2048), (14, 2048), (96, 8192),
                                        (12, 512), (1, 8), (3, 264), (5, 72)])
def test_dw_blocks_cover_every_tile_once_in_balanced_xcd_shares(tm_count, d):
    dtc = cdiv(d, 256)
    t = tm_count * dtc
    grid = 8 * cdiv(t, 8)                      # the host's dW grid
    tiles = [dw_block_tile(b, tm_count, d) for b in range(grid)]
    live = [tt for tt in tiles if tt is not None]
    assert sorted(live) == sorted((tm, tn) for tm in range(tm_count) for tn in range(dtc))
    per_xcd = [sum(tiles[b] is not None for b in range(x, grid, 8)) for x in range(8)]
    assert max(per_xcd) - min(per_xcd) <= 1


def dw_rounds(v, d, r):
    # workgroup rounds of the dW launches with slabs of r row tiles (8 XCDs x 32 CUs)
    dtc, vt = cdiv(d, 256), cdiv(v, 384)
    return sum(cdiv(cdiv(min(r, vt - t0) * dtc, 8), 32) for t0 in range(0, vt, r))


@pytest.mark.parametrize("d,v", [(512, 4096), (2048, 128256), (4096, 128256), (3584, 152064), (8192, 128256),
                                 (2560, 151936), (1536, 151936), (5120, 152064), (3584, 1000)])
def test_the_slab_width_gives_the_dw_launches_the_fewest_rounds_in_its_range(d, v):
    info = B.lce_plan_info(B.problem(4096, d, v))
    vc = info["vc"]
    assert vc % 768 == 0 and info["nslab"] == cdiv(v, vc)
    lo = max(8192, 4 * d)
    hi = min(rup(v, 768), max(vc, min(24576, (160 << 20) // (2 * d))))
    if vc >= rup(v, 768):
        return                                  # one slab holds the whole vocabulary
    best = min(dw_rounds(v, d, r) for r in range(cdiv(lo, 768) * 2, hi // 384 + 1, 2))
    assert dw_rounds(v, d, vc // 384) <= best
    assert lo <= vc <= hi
    if (d, v) == (3584, 152064):                # the 3584-wide head: whole rounds, as few as the tiles allow
        assert dw_rounds(v, d, vc // 384) == cdiv(cdiv(v, 384) * cdiv(d, 256), 256) == 22


def xcd_tile(b, tiles, gw, nt):
    """The (vocabulary tile, token tile) of block b of a forward or G launch, as xcd_tile maps it."""
    a = tiles & ~7
    ba = a * nt
    if b < ba:
        full, g = a // gw, b // (gw * nt)
        wl = gw if g < full else a - full * gw
        r = b - g * gw * nt
        return g * gw + r % wl, r // wl
    rem, r = tiles - a, b - ba
    if rem == 0:
        return None
    k = r >> 3
    tn = (r & 7) + 8 * (k // rem)
    return (a + k % rem, tn) if tn < nt else None


def tile_order(tiles, nt, width):
    a = tiles & ~7
    rem = tiles - a
    return a * nt + (8 * rem * cdiv(nt, 8) if rem else 0), max(8, min(width, a) & ~7)


@pytest.mark.parametrize("tiles,nt,width", [(334, 48, 48), (54, 90, 54), (46, 48, 46), (96, 52, 24), (64, 24, 64),
                                            (12, 1, 12), (11, 2, 11), (3, 5, 3), (72, 64, 72), (17, 9, 17), (1, 1, 1),
                                            (8, 7, 8), (40, 33, 16)])
def test_forward_and_g_blocks_cover_every_tile_once_and_keep_w_tiles_on_one_xcd(tiles, nt, width):
    grid, gw = tile_order(tiles, nt, width)
    assert gw % 8 == 0
    got = [xcd_tile(b, tiles, gw, nt) for b in range(grid)]
    live = [t for t in got if t is not None]
    assert sorted(live) == [(tm, tn) for tm in range(tiles) for tn in range(nt)]
    a = tiles & ~7
    for b, t in enumerate(got):
        if t is None:
            continue
        tm, tn = t
        if tm < a:
            assert tm % 8 == b % 8          # each XCD keeps its own W tiles of the aligned part
        else:
            assert tn % 8 == b % 8          # and its own token tiles of the last few vocabulary tiles
