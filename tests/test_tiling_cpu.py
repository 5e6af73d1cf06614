"""CPU replay of the index arithmetic of the matrix-core kernels' staging.

The GEMM stages ROWS x BK tiles in 16-byte chunks; every K segment is tiled
on its own and chunks at or past the segment end are never read.  The
post-attention layer kernel stages weight and activation chunks of FC units
in 16-byte pieces spread over its 512 threads.  These tests replay both (the
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
LAYER_FC = {"bf16": 64, "f32": 32}      # FFN, W_o and QKV chunks
LAYER_FCQ = LAYER_FC
LAYER_RB1 = {"bf16": 2, "f32": 1}       # unit-tiling row blocks per wave
LAYER_ROWS = 128
LAYER_THREADS = 512
LAYER_WAVES = 8


def _stage_reads(rows, cols, elem_bytes, base, ld, rows_valid=None):
    """Element offsets read by Stage<T, rows, cols>.load(base, ld, rows_valid)."""
    epv = 16 // elem_bytes
    cpr = cols // epv
    chunks = rows * cpr
    per = -(-chunks // LAYER_THREADS)
    rv = rows if rows_valid is None else rows_valid
    out = []
    for t in range(LAYER_THREADS):
        for i in range(per):
            q = t + i * LAYER_THREADS
            if q < chunks and q // cpr < rv:
                out.append((base + (q // cpr) * ld + (q % cpr) * epv, epv))
    return out


def _check_cover(reads, size, expect):
    seen = []
    for off, n in reads:
        assert 0 <= off and off + n <= size, (off, n, size)
        seen.extend(range(off, off + n))
    assert sorted(seen) == sorted(expect)


def _lane_bias_units(dtype, fcx):
    """Units u0 + 16 j + [0, 4) each lane reads from a chunk's biases."""
    rb1 = LAYER_RB1[dtype]
    p1m = LAYER_ROWS // (16 * rb1)
    p1n = LAYER_WAVES // p1m
    hpw = fcx // p1n
    units = set()
    for wave in range(LAYER_WAVES):
        for lane in range(64):
            u0 = (wave % p1n) * hpw + 4 * (lane >> 4)
            for j in range(hpw // 16):
                units.update(range(u0 + 16 * j, u0 + 16 * j + 4))
    return units


@pytest.mark.parametrize("name", W.CONFIG_ORDER)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_layer_kernel_staging_stays_in_bounds(name, dtype):
    cfg = W.get_config(name).replace(dtype=dtype)
    d, dff, eb = cfg.d_model, cfg.d_ff, (2 if dtype == "bf16" else 4)
    fc, fcq = LAYER_FC[dtype], LAYER_FCQ[dtype]
    assert d % fc == 0 and dff % fc == 0 and (3 * d) % fcq == 0
    # W_1 [dff, d] in chunks of fc rows, W_qkv [3d, d] in chunks of fcq rows
    for rows_total, step in ((dff, fc), (3 * d, fcq)):
        reads = []
        for c in range(rows_total // step):
            reads += _stage_reads(step, d, eb, c * step * d, d)
        _check_cover(reads, rows_total * d, range(rows_total * d))
    # W_2 [d, dff] and W_o [d, d]: all d rows x columns [c fc, c fc + fc)
    for k_total in (dff, d):
        reads = []
        for c in range(k_total // fc):
            reads += _stage_reads(d, fc, eb, c * fc, k_total)
        _check_cover(reads, d * k_total, range(d * k_total))
    # O [M, d]: block m0 = rows [m0, m0 + 128) (rows >= M not read) x column chunks
    M = 300 if cfg.n_nodes > 300 else cfg.n_nodes
    reads = []
    for m0 in range(0, M, LAYER_ROWS):
        for c in range(d // fc):
            reads += _stage_reads(LAYER_ROWS, fc, eb, m0 * d + c * fc, d, rows_valid=M - m0)
    _check_cover(reads, M * d, range(M * d))
    # biases: every lane's 4-unit pieces cover each chunk exactly within its range
    assert _lane_bias_units(dtype, fc) == set(range(fc))
    assert _lane_bias_units(dtype, fcq) == set(range(fcq))
