"""CPU replay of the index arithmetic of the matrix-core kernels' staging.

The GEMM stages ROWS x BK tiles in 16-byte chunks; every K segment is tiled
on its own and chunks at or past the segment end are never read.  The
post-attention layer kernel moves weight and activation chunks of FC units
to LDS by direct loads into XOR-swizzled tiles.  These tests replay both (the
same constants as the kernels) for every call each workload issues and check
that every read lands inside its matrix and that every element is covered
exactly once."""
import pytest

from paper_1910_01578_amd import workloads as W

BK = {"bf16": 64, "f32": 32}


def _gemm_calls(cfg):
    """(label, a-elem-bytes, k1, k2) of every GEMM / LN-GEMM of one forward."""
    b = 2 if cfg.dtype == "bf16" else 4
    calls = []
    for l in range(cfg.gnn_layers):
        hin = cfg.feat_dim if l == 0 else cfg.hidden
        calls.append(("pool", b, hin, 0))
        calls.append(("update", b, hin, cfg.hidden))
    calls.append(("qkv", 4, cfg.d_model, 0))           # layer 0; A = fp32 residual stream
    return calls


def _replay(a_bytes, k1, k2, bk):
    epa = 16 // a_bytes
    cpr = bk // epa
    seen = {1: [], 2: []}
    kt1 = -(-k1 // bk)
    kt = kt1 + -(-k2 // bk)
    for t in range(kt):
        seg, k0, kmax = (1, t * bk, k1) if t < kt1 else (2, (t - kt1) * bk, k2)
        for c in range(cpr):
            col = c * epa
            if k0 + col < kmax:
                assert k0 + col + epa <= kmax, "a chunk would straddle the segment end"
                seen[seg].extend(range(k0 + col, k0 + col + epa))
    assert sorted(seen[1]) == list(range(k1))
    assert sorted(seen[2]) == list(range(k2))


@pytest.mark.parametrize("name", W.CONFIG_ORDER)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_tile_loader_stays_in_rows(name, dtype):
    cfg = W.get_config(name).replace(dtype=dtype)
    for label, ab, k1, k2 in _gemm_calls(cfg):
        # the weights are staged in the MFMA type
        _replay(ab, k1, k2, BK[dtype])
        _replay(2 if dtype == "bf16" else 4, k1, k2, BK[dtype])


@pytest.mark.parametrize("k1,k2", [(32, 128), (32, 0), (96, 64), (64, 256), (160, 32)])
def test_partial_tiles(k1, k2):
    for dtype in ("f32", "bf16"):
        for ab in (2, 4):
            _replay(ab, k1, k2, BK[dtype])


def _xcd_remap(p, total, nx=8):
    per, rem = divmod(total, nx)
    x, idx = p % nx, p // nx
    return x * per + min(x, rem) + idx


@pytest.mark.parametrize("total", [1, 2, 7, 8, 9, 10, 63, 64, 65, 813, 2442, 3264, 5000])
def test_xcd_remap_is_a_bijection_with_contiguous_runs(total):
    """Work-group ids are dealt to 8 XCDs round-robin; the kernels map them to
    logical tiles so that every XCD owns one contiguous run of tiles."""
    logical = [_xcd_remap(p, total) for p in range(total)]
    assert sorted(logical) == list(range(total))
    for x in range(8):
        mine = sorted(logical[p] for p in range(x, total, 8))
        assert mine == list(range(mine[0], mine[0] + len(mine))) if mine else True


# ---- post-attention layer kernel ------------------------------------------------
# Operands reach LDS by direct global -> LDS loads: load i of wave w writes
# the 64 lanes' 16-byte granules to tile granules (w * PER + i) * 64 + lane,
# and granule g of tile row r sits at granule g ^ key(r) of that row.
LAYER_FC = {"bf16": 64, "f32": 32}      # units per chunk (FFN, W_o and QKV)
LAYER_RB1 = {"bf16": 2, "f32": 1}       # unit-tiling row blocks per wave
LAYER_MFMA_K = {"bf16": 32, "f32": 4}
LAYER_ROWS = 128
LAYER_THREADS = 512
LAYER_WAVES = 8
EB = {"bf16": 2, "f32": 4}


def _key(gpr, r):
    if gpr >= 16:
        return r & 15
    if gpr == 8:
        return r & 7
    assert gpr == 4
    return ((r >> 2) ^ (r >> 1)) & 3


def _swz(cols, epv, r, c):
    return r * cols + ((c // epv) ^ _key(cols // epv, r)) * epv + c % epv


def _dma_tile(rows, cols, eb, ld, row_max, nw=LAYER_WAVES):
    """(tile element offset, source element offset, row, column) of every
    element moved by dma_tile<T, rows, cols>(tile, src, ld, row_max), from the
    kernel's split of each address into a wave-uniform row base and a per-lane
    offset."""
    epv = 16 // eb
    gpr = cols // epv
    granules = rows * gpr
    assert granules % (64 * nw) == 0 and 4 <= gpr <= 64
    per = granules // (64 * nw)
    clamp = row_max < rows - 1
    out = []
    for wave in range(nw):
        for i in range(per):
            q = (wave * per + i) * 64
            rb = q // gpr
            for lane in range(64):
                lr = lane // gpr
                g = (lane % gpr) ^ _key(gpr, lr) ^ _key(gpr, rb)
                # the split equals the plain per-granule formula
                p = q + lane
                assert p // gpr == rb + lr and g == (p % gpr) ^ _key(gpr, p // gpr)
                r0, rel = rb, lr
                if clamp:
                    r0 = min(rb, row_max)
                    rel = min(rb + lr, row_max) - r0
                assert rel >= 0
                off_bytes = (rel * ld + g * epv) * eb
                assert 0 <= off_bytes < 2 ** 32
                src_row = r0 + rel
                assert src_row == min(rb + lr, row_max)
                for e in range(epv):
                    out.append((p * epv + e, src_row * ld + g * epv + e, rb + lr, g * epv + e))
    return out


def _geo(dtype, d):
    fc, rb1, k = LAYER_FC[dtype], LAYER_RB1[dtype], LAYER_MFMA_K[dtype]
    p1m = LAYER_ROWS // (16 * rb1)
    p1n = LAYER_WAVES // p1m
    nz = LAYER_ROWS // fc
    qh = 2 if (LAYER_WAVES // p1m) == 2 and (3 * d) % (2 * fc) == 0 else 1
    return dict(qh=qh, fcq=qh * fc, hpwq=qh * fc // p1n, fc=fc, rb1=rb1, k=k, p1m=p1m, p1n=p1n, hpw=fc // p1n, buf=fc * max(d, LAYER_ROWS), nz=nz, zc=d // nz,
                epv=16 // EB[dtype], mb2=LAYER_ROWS // 2 // 16, nb2=d // 4 // 16)


def _check_tile(rows, cols, dtype, d, ld, src_rows, row_max=None, nw=LAYER_WAVES):
    """The DMA of a rows x cols tile writes every tile element exactly once,
    inside the staging buffer, with the source element that swz() reads there."""
    g = _geo(dtype, d)
    eb, epv = EB[dtype], g["epv"]
    row_max = rows - 1 if row_max is None else row_max
    moved = _dma_tile(rows, cols, eb, ld, row_max, nw)
    dst = [m[0] for m in moved]
    assert sorted(dst) == list(range(rows * cols))
    assert rows * cols <= g["buf"]
    for t, srcoff, r, c in moved:
        assert _swz(cols, epv, r, c) == t
        assert 0 <= srcoff < src_rows * ld
        assert srcoff == min(r, row_max) * ld + c
    return moved


@pytest.mark.parametrize("d", [64, 128, 256])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_layer_kernel_dma_tiles(d, dtype):
    g = _geo(dtype, d)
    fc = g["fc"]
    dff = 4 * d
    # W_1 / W_qkv chunk: fc rows x d (ld d); W_2 / W_o chunk: d rows x fc (ld d_ff / d);
    # loaded by all 8 waves or (spread over a product) by waves 0 .. 3
    for nw in (8, 4):
        _check_tile(fc, d, dtype, d, d, fc, nw=nw)
        for ld in (dff, d):
            _check_tile(d, fc, dtype, d, ld, d, nw=nw)
    # O chunk: 128 rows x fc of an [M, d] matrix; a ragged last block clamps rows
    for rows_valid in (128, 100, 1):
        moved = _check_tile(LAYER_ROWS, fc, dtype, d, d, rows_valid, row_max=rows_valid - 1)
        assert {r for _, _, r, _ in moved if r < rows_valid} == set(range(rows_valid))
    # QKV chunks: FCQ = QH * FC units as QH tiles of FC rows; together they cover W_qkv once
    cover = []
    for q in range(3 * d // g["fcq"]):
        for h in range(g["qh"]):
            r0 = q * g["fcq"] + h * fc
            cover += [r0 * d + s for _, s, _, _ in _dma_tile(fc, d, EB[dtype], d, fc - 1)]
    assert sorted(cover) == list(range(3 * d * d))
    assert d % g["fcq"] == 0            # a QKV chunk lies within q, k or v
    # every chunk of W_1, W_2, W_qkv, W_o covers its matrix exactly once
    for total_rows in (dff, 3 * d):
        cover = []
        for c in range(total_rows // fc):
            cover += [c * fc * d + s for _, s, _, _ in _dma_tile(fc, d, EB[dtype], d, fc - 1)]
        assert sorted(cover) == list(range(total_rows * d))
    for kt in (dff, d):
        cover = []
        for c in range(kt // fc):
            cover += [c * fc + s for _, s, _, _ in _dma_tile(d, fc, EB[dtype], kt, d - 1)]
        assert sorted(cover) == list(range(d * kt))


@pytest.mark.parametrize("gpr", [4, 8, 16, 32, 64])
def test_layer_swizzle_is_bank_conflict_free(gpr):
    """A fragment load reads one granule from each of 16 consecutive rows; any
    8 aligned of them land in distinct 16-byte bank groups (the keys' measured
    conflict-freedom on the device is recorded with the kernels), and each
    row's key is a permutation of its granules."""
    for r0 in range(0, 64, 16):
        for gl in range(gpr):
            pos = [(r * gpr + (gl ^ _key(gpr, r))) for r in range(r0, r0 + 16)]
            for h in (0, 8):
                assert len({p % 8 for p in pos[h:h + 8]}) == 8
                assert len({p % 16 for p in pos[h:h + 8]}) == 8
            if gpr >= 16:
                assert len({p % 16 for p in pos}) == 16
    for r in range(64):
        assert sorted(gl ^ _key(gpr, r) for gl in range(gpr)) == list(range(gpr))


@pytest.mark.parametrize("d", [64, 128, 256])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_layer_kernel_lds_reads_in_range(d, dtype):
    g = _geo(dtype, d)
    fc, k, epv, zc = g["fc"], g["k"], g["epv"], g["zc"]
    kv = k // 4
    ks1, ks2 = d // k, fc // k
    assert ks1 >= 1 and ks2 >= 1 and d % fc == 0 and zc % k == 0 and zc % (d // 4) == 0
    jb1 = g["hpw"] // 16
    for wave in range(LAYER_WAVES):
        p1m, p1n = wave // g["p1n"], wave % g["p1n"]
        w2m, w2n = wave // 4, wave % 4
        zpart = w2n * g["nb2"] * 16 // zc
        assert zpart < g["nz"]
        for lane in range(64):
            col, g4 = lane & 15, lane >> 4
            # unit tiling: weight rows (units) x k in an fc x d tile; bias units
            for j in range(jb1):
                u = p1n * g["hpw"] + j * 16 + col
                assert u < fc
                for s in range(ks1):
                    assert 0 <= _swz(d, epv, u, s * k + kv * g4) < fc * d
                hc = p1n * g["hpw"] + j * 16 + 4 * g4
                assert hc + 4 <= fc and hc % epv + 4 <= epv       # H store within a granule
                for i in range(g["rb1"]):
                    assert 0 <= _swz(fc, epv, (p1m * g["rb1"] + i) * 16 + col, hc) < LAYER_ROWS * fc
            # QKV: the wave's units lie in one FC-row tile (its half of the chunk)
            for j in range(g["hpwq"] // 16):
                u0 = 0 if g["qh"] == 2 else p1n * g["hpwq"]
                assert u0 + j * 16 + col < fc
                hcq = p1n * g["hpwq"] + j * 16 + 4 * g4
                assert hcq + 4 <= g["fcq"]
                if g["qh"] == 2:
                    assert hcq // fc == p1n           # bias entry of the wave's own half
            # activation parts (128 x zc, one staging buffer each): writes and reads
            assert LAYER_ROWS * zc <= g["buf"]
            for i in range(g["mb2"]):
                for j in range(g["nb2"]):
                    c = w2n * g["nb2"] * 16 + 4 * g4 + j * 16 - zpart * zc
                    assert 0 <= c and c + 4 <= zc and c % epv + 4 <= epv
                    assert _swz(zc, epv, w2m * g["mb2"] * 16 + col + i * 16, c) < LAYER_ROWS * zc
            for i in range(g["rb1"]):
                for s in range(ks1):
                    z = s * k // zc
                    cc = s * k - z * zc + kv * g4
                    assert z < g["nz"] and 0 <= cc < zc
                    assert _swz(zc, epv, (p1m * g["rb1"] + i) * 16 + col, cc) < LAYER_ROWS * zc
            # row tiling: A (128 x fc) and W (d x fc) fragments
            for s in range(ks2):
                for i in range(g["mb2"]):
                    assert _swz(fc, epv, w2m * g["mb2"] * 16 + i * 16 + col, s * k + kv * g4) < LAYER_ROWS * fc
                for j in range(g["nb2"]):
                    assert _swz(fc, epv, w2n * g["nb2"] * 16 + j * 16 + col, s * k + kv * g4) < d * fc
    # LDS budget: 4 staging buffers + H + 2 bias chunks + LayerNorm sums
    total = (4 * g["buf"] + LAYER_ROWS * fc + 2 * g["fcq"]) * EB[dtype] + LAYER_ROWS * 4 * 4
    assert total <= 160 * 1024


@pytest.mark.parametrize("name", W.CONFIG_ORDER)
def test_layer_kernel_accepts_workload_shapes(name):
    cfg = W.get_config(name)
    for dtype in ("f32", "bf16"):
        fc = LAYER_FC[dtype]
        assert cfg.d_ff % (2 * fc) == 0 and cfg.d_model % fc == 0
        assert cfg.d_model in (64, 128, 256)


@pytest.mark.parametrize("d", [128, 256])
def test_layer_qkv_store_transpose(d):
    """bf16 QKV outputs pass through each wave's 2 KB of H: the 16 x 64 block a
    wave writes (4 units a lane) is read back as 16-byte pieces of whole rows,
    every (row, unit) exactly once and to its own global position."""
    g = _geo("bf16", d)
    assert g["qh"] == 2
    wu, epv = g["hpwq"], 8
    assert wu * 2 == 128 and LAYER_WAVES * 16 * wu <= LAYER_ROWS * g["fc"]
    for wave in range(LAYER_WAVES):
        p1n = wave % g["p1n"]
        base = wave * 16 * wu
        written = {}
        for lane in range(64):
            col, g4 = lane & 15, lane >> 4
            for j in range(wu // 16):
                u = j * 16 + 4 * g4
                t = _swz(wu, epv, col, u)
                assert u % epv + 4 <= epv
                for e in range(4):
                    written[base + t + e] = (col, u + e)
        assert len(written) == 16 * wu
        read = []
        for hf in range(2):
            for lane in range(64):
                rr, gg = (lane >> 3) + 8 * hf, lane & 7
                t = base + _swz(wu, epv, rr, gg * 8)
                for e in range(8):
                    row, unit = written[t + e]
                    assert row == rr and unit == gg * 8 + e      # stored at column p1n*64 + gg*8 + e
                    read.append((row, unit))
        assert sorted(read) == sorted(written.values())
        assert 0 <= base and base + 16 * wu <= LAYER_ROWS * g["fc"]


@pytest.mark.parametrize("d", [128, 256])
def test_layer_wide_qkv_tiling(d):
    """The bf16 QKV phase with 64-row waves (2 row groups x 4 unit groups of 32
    units): over the 8 waves every (row, unit) of a 128-unit chunk is formed
    exactly once, each wave's weight fragments lie in one 64-unit half (the u
    or r buffer), the activation reads stay inside the two ZC-column parts,
    and the 16 x 32 staging block in the wave's own 1 KB of H is read back as
    16-byte pieces of whole 64-byte rows, every (row, unit) exactly once."""
    g = _geo("bf16", d)
    assert g["qh"] == 2
    fc, fcq, epv = g["fc"], 2 * g["fc"], 8
    rb, pm, pn = 4, LAYER_ROWS // 64, LAYER_WAVES // (LAYER_ROWS // 64)
    wu = fcq // pn
    assert (pm, pn, wu) == (2, 4, 32)
    nz = LAYER_ROWS // fc
    zc = d // nz
    formed = []
    for wave in range(LAYER_WAVES):
        wm, wn = wave // pn, wave % pn
        half, u0 = (wn * wu) // fc, (wn * wu) % fc
        assert u0 + wu <= fc                                  # one buffer of the pair
        for i in range(rb):
            for j in range(wu // 16):
                for col in range(16):
                    for g4 in range(4):
                        for r in range(4):
                            formed.append(((wm * rb + i) * 16 + col, half * fc + u0 + j * 16 + 4 * g4 + r))
        for s in range(d // 32):                              # activation fragment reads
            z = s * 32 // zc
            for i in range(rb):
                for col in range(16):
                    for g4 in range(4):
                        c = s * 32 - z * zc + 8 * g4
                        assert 0 <= c and c + 8 <= zc and z < nz
                        t = _swz(zc, epv, (wm * rb + i) * 16 + col, c)
                        assert 0 <= t and t + 8 <= LAYER_ROWS * zc
        base = wave * 16 * wu                                 # staging
        assert base + 16 * wu <= LAYER_ROWS * fc
        written = {}
        for lane in range(64):
            col, g4 = lane & 15, lane >> 4
            for j in range(wu // 16):
                u = j * 16 + 4 * g4
                t = _swz(wu, epv, col, u)
                for e in range(4):
                    written[base + t + e] = (col, u + e)
        assert len(written) == 16 * wu
        read = []
        for lane in range(64):
            rr, gg = lane >> 2, lane & 3
            t = base + _swz(wu, epv, rr, gg * 8)
            assert t % epv == 0
            for e in range(8):
                row, unit = written[t + e]
                assert row == rr and unit == gg * 8 + e       # stored at column wn*32 + gg*8 + e
                read.append((row, unit))
        assert sorted(read) == sorted(written.values())
    assert sorted(formed) == [(r, u) for r in range(LAYER_ROWS) for u in range(fcq)]


@pytest.mark.parametrize("d", [128, 256])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_layer_residual_store_transpose(d, dtype):
    """Y' (fp32) leaves the row tiling through each wave's 2 KB of H in
    16-row x 32-column pieces: every (row, column) of the wave's 64 x d/4
    block is stored exactly once, from the lane that holds it."""
    g = _geo(dtype, d)
    nb2, mb2 = g["nb2"], g["mb2"]
    assert nb2 % 2 == 0 and LAYER_WAVES * 16 * 32 * 4 <= LAYER_ROWS * g["fc"] * EB[dtype]
    for wave in range(LAYER_WAVES):
        w2m, w2n = wave // 4, wave % 4
        base = wave * 16 * 32
        stored = []
        for i in range(mb2):
            for jh in range(nb2 // 2):
                lds = {}
                for lane in range(64):
                    col, g4 = lane & 15, lane >> 4
                    for jj in range(2):
                        c = w2n * nb2 * 16 + 4 * g4 + (2 * jh + jj) * 16      # the lane's columns
                        t = base + _swz(32, 4, col, jj * 16 + 4 * g4)
                        for e in range(4):
                            lds[t + e] = (w2m * mb2 * 16 + i * 16 + col, c + e)
                assert len(lds) == 16 * 32
                c0 = w2n * nb2 * 16 + jh * 32
                for hf in range(2):
                    for lane in range(64):
                        rr, gg = (lane >> 3) + 8 * hf, lane & 7
                        t = base + _swz(32, 4, rr, gg * 4)
                        for e in range(4):
                            assert lds[t + e] == (w2m * mb2 * 16 + i * 16 + rr, c0 + gg * 4 + e)
                            stored.append(lds[t + e])
        expect = [(w2m * 64 + r, w2n * nb2 * 16 + c) for r in range(64) for c in range(nb2 * 16)]
        assert sorted(stored) == sorted(expect)


@pytest.mark.parametrize("d", [128, 256])
def test_row_gemm_store_transpose(d):
    """The GNN dense-layer kernel's bf16 output leaves the row tiling through
    each wave's slice of H: the wave's 16-row x WC block (WC = d/4 columns, 4 a
    lane) is read back as 16-byte parts of whole rows; every element is stored
    once, at its own position, and the slice stays inside H."""
    g = _geo("bf16", d)
    wc = g["nb2"] * 16
    lpr = wc * 2 // 16
    rpi = 64 // lpr
    assert LAYER_WAVES * 16 * wc <= LAYER_ROWS * g["fc"]
    for wave in range(LAYER_WAVES):
        base = wave * 16 * wc
        lds = {}
        for lane in range(64):
            col, g4 = lane & 15, lane >> 4
            for j in range(g["nb2"]):
                c = j * 16 + 4 * g4
                t = base + _swz(wc, 8, col, c)
                assert c % 8 + 4 <= 8
                for e in range(4):
                    lds[t + e] = (col, c + e)
        assert len(lds) == 16 * wc
        out = []
        for hf in range(16 // rpi):
            for lane in range(64):
                rr, gg = lane // lpr + rpi * hf, lane % lpr
                t = base + _swz(wc, 8, rr, gg * 8)
                for e in range(8):
                    assert lds[t + e] == (rr, gg * 8 + e)
                    out.append(lds[t + e])
        assert sorted(out) == sorted(lds.values())


@pytest.mark.parametrize("R", [2, 4])
@pytest.mark.parametrize("nk", [1, 2, 3, 4, 5, 8])
def test_row_gemm_chunk_schedule(R, nk):
    """Replay of the GNN dense-layer kernel's load schedule: the prologue loads
    A(0 .. R-2) and W(0); the top of chunk c loads W(c+1) then A(c+R-1).
    Every chunk's A and W are loaded exactly once, before the chunk that
    reads them, into a slot / buffer not read since the previous barrier, and
    the loads that may still be in flight at chunk c's wait are exactly the
    ones issued after W(c) (A(c+R-2) when it exists)."""
    issued = []                       # (kind, chunk, slot) in issue order
    for c in range(min(R - 1, nk)):
        issued.append(("A", c, c % R))
    issued.append(("W", 0, 0))
    last_read = {}                    # ("A", slot) / ("W", buf) -> chunk that last read it
    for c in range(nk):
        # the kernel's wait leaves the newest group in flight (the A(c+R-2) loads)
        # when R > 2, c >= 1 and c + R - 2 < nk, and nothing otherwise
        partial = R > 2 and c >= 1 and c + R - 2 < nk
        in_flight = issued[-1:] if partial else []
        if partial:
            assert in_flight == [("A", c + R - 2, (c + R - 2) % R)], (c, issued[-3:])
        done = issued[:len(issued) - len(in_flight)]
        assert ("A", c, c % R) in done and ("W", c, c % 2) in done, c
        # issues at the top of chunk c write buffers last read in chunk c - 1 (or never)
        if c + 1 < nk:
            assert last_read.get(("W", (c + 1) % 2), -1) <= c - 1
            issued.append(("W", c + 1, (c + 1) % 2))
        if c + R - 1 < nk:
            assert last_read.get(("A", (c + R - 1) % R), -1) <= c - 1
            issued.append(("A", c + R - 1, (c + R - 1) % R))
        last_read[("A", c % R)] = c
        last_read[("W", c % 2)] = c
    assert sorted(x[1] for x in issued if x[0] == "A") == list(range(nk))
    assert sorted(x[1] for x in issued if x[0] == "W") == list(range(nk))


# ---- segment attention: V tiles read back transposed ---------------------------
# ds_read_b64_tr_b16: within each group of 16 lanes, destination lane 4q + p
# receives in slot e element p of the 8-byte word addressed by source lane 4e + q.
ATTN_BKV = 64


def _tr16(word_elem):
    """Element offset that (lane, slot) receives, given each lane's word address."""
    out = {}
    for lane in range(64):
        grp, i = lane // 16, lane % 16
        q, p = i // 4, i % 4
        for e in range(4):
            out[(lane, e)] = word_elem[16 * grp + 4 * e + q] + p
    return out


@pytest.mark.parametrize("dh", [32, 64])
@pytest.mark.parametrize("row_max", [63, 40, 0])
def test_attention_v_fragments(dh, row_max):
    """Direct loads put the V tile in LDS row-major and swizzled; the transposing
    reads give lane (g4, d) dim 16b + d of the keys its MFMA k slots stand for
    (slot 8*g4 + i: key 32c + 4*g4 + i, or 32c + 16 + 4*g4 + i - 4), and each
    read's 32-lane halves touch distinct banks."""
    epv = 8
    ld = 3 * 8 * dh
    moved = _dma_tile(ATTN_BKV, dh, 2, ld, row_max, nw=4)
    tile = {t: (min(r, row_max), c) for t, _, r, c in moved}
    assert sorted(tile) == list(range(ATTN_BKV * dh))
    for c2 in range(2):
        for b in range(dh // 16):
            frag = {}
            for h in range(2):
                words = []
                for lane in range(64):
                    col, g4 = lane % 16, lane // 16
                    key, dim = 32 * c2 + 16 * h + 4 * g4 + (col >> 2), 16 * b + 4 * (col & 3)
                    w = _swz(dh, epv, key, dim)
                    assert w % 4 == 0 and w // epv == (w + 3) // epv   # 8 aligned bytes in one granule
                    words.append(w)
                for half in range(2):
                    banks = set()
                    for w in words[32 * half:32 * half + 32]:
                        banks |= {(2 * w // 4 + k) % 64 for k in range(2)}
                    assert len(banks) == 64
                for (lane, e), t in _tr16(words).items():
                    frag[(lane, 4 * h + e)] = tile[t]
            for lane in range(64):
                col, g4 = lane % 16, lane // 16
                for i in range(8):
                    key = 32 * c2 + 4 * g4 + (i if i < 4 else 16 + i - 4)
                    assert frag[(lane, i)] == (min(key, row_max), 16 * b + col)


# ---- segment attention: the K/V tile ring ---------------------------------------
def _attention_ring_program(ntiles, kp, ns=3):
    """One wave's program order over a segment's key tiles, as the kernel issues
    it (direct loads, ring of ns buffers, loads ns - 1 tiles ahead): ("load", t,
    buf), ("wait", t, tiles allowed to stay in flight), ("barrier",),
    ("read", t, buf)."""
    prog = [("load", 0, 0)]
    if ntiles > 1:
        prog.append(("load", 1, 1))
    prog += [("wait", min(ntiles, 2) - 1, 0), ("barrier",)]        # every load so far
    if kp:
        prog.append(("read", 0, 0))                       # K fragments of tile 0
    for t in range(ntiles):
        cur = t % ns
        if not kp:
            prog.append(("read", t, cur))                 # K fragments
        prog.append(("read", t, cur))                     # V fragments
        if t + ns - 1 < ntiles:
            prog.append(("load", t + ns - 1, (t + ns - 1) % ns))
        if kp and t + 1 < ntiles:
            prog += [("wait", t + 1, 1 if t + 2 < ntiles else 0), ("barrier",), ("read", t + 1, (t + 1) % ns)]
        if not kp:                                        # after the last tile: a full wait
            prog += [("wait", min(t + 1, ntiles - 1), 1 if t + 2 < ntiles else 0), ("barrier",)]
    return prog


@pytest.mark.parametrize("kp", [True, False], ids=["k_prefetch", "end_barrier"])
@pytest.mark.parametrize("ntiles", list(range(1, 10)))
def test_attention_ring_schedule(ntiles, kp):
    """Replay of the tile ring: every wave runs the same program and passes each
    barrier only when all have reached it, so (1) a tile is read only after a
    barrier that follows the wait covering its loads, (2) a buffer is loaded
    again only after a barrier that follows every read of its previous tile,
    and (3) each wait's count leaves in flight exactly the loads issued after
    the tile it waits for (vector memory operations complete in issue order)."""
    prog = _attention_ring_program(ntiles, kp)
    barriers = [i for i, x in enumerate(prog) if x[0] == "barrier"]

    def barrier_before(i):
        b = [j for j in barriers if j < i]
        return b[-1] if b else -1

    load_pos = {x[1]: i for i, x in enumerate(prog) if x[0] == "load"}
    assert sorted(load_pos) == list(range(ntiles))
    occupant = {}
    last_read = {}
    for i, x in enumerate(prog):
        if x[0] == "load":
            t, buf = x[1], x[2]
            if buf in occupant:                           # (2)
                assert last_read[occupant[buf]] < barrier_before(i), (t, buf)
            occupant[buf] = t
        elif x[0] == "read":
            t, buf = x[1], x[2]
            assert occupant.get(buf) == t
            waits = [j for j, y in enumerate(prog[:i]) if y[0] == "wait" and y[1] >= t]
            assert waits and waits[0] < barrier_before(i), t   # (1)
            last_read[t] = i
        elif x[0] == "wait":
            t, allowed = x[1], x[2]
            later = [u for u, p in load_pos.items() if u > t and p < i]
            # (3): vmcnt(N) covers all but the N most recent operations, so the
            # count may not exceed the loads issued after tile t (equal: no over-wait)
            assert allowed == len(later), (t, later)
            # the tiles it must cover were all issued before it
            assert all(load_pos[u] < i for u in range(t + 1))
    assert set(last_read) == set(range(ntiles))
