"""CPU replay of the GEMM tile loader's index arithmetic.

The matrix-core GEMM stages ROWS x BK tiles in 16-byte chunks; every K
segment is tiled on its own and chunks at or past the segment end are never
read.  This test replays that arithmetic (the same constants as the kernel:
BK = 64 for bf16, 32 for fp32; 16-byte chunks of the staged type) for every
GEMM each workload issues and checks that every read lands inside its row
and that every K column is covered exactly once."""
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
    for _ in range(cfg.placer_layers):
        calls.append(("qkv", 4, cfg.d_model, 0))       # A = fp32 residual stream
        calls.append(("out_ln", b, cfg.d_model, 0))
        calls.append(("ffn1", 4, cfg.d_model, 0))
        calls.append(("ffn2_ln", b, cfg.d_ff, 0))
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
