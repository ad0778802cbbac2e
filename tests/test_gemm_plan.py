"""CPU checks of the projection tile planner through the C ABI: every
residual projection of every workload fits the split-K workspace the state
allocates, at every live row count.

The residual projections (O and the dense down projection) may split K on
the device: with S splits each writes its raw partial tile to
ws[S][row tiles * bm][N], and the next RMSNorm folds them.  S is chosen
from the live row count M (doubling while the output tiles times 2S stay
within the workgroup target, the split depth stays a multiple of 128 and at
least 256, and S stays within zmax), so the extent S * ceil(M / bm) * bm * N
is restated here independently of the library and maximised over M.
"""
import numpy as np
import pytest

from bd_synth import WORKLOADS


def _rows_caps(w):
    """Row capacities a state of this workload can hold: the step window
    (2 n_inflight B rows per sequence) and the prefill (P rows per sequence),
    each rounded up to 256, for the workload's own batch and smaller and
    larger ones."""
    caps = set()
    for b in sorted({1, 2, 7, 16, w.batch, 64, 256}):
        for nb in sorted({1, 2, 3, w.n_inflight, 8}):
            caps.add(-(-b * 2 * nb * w.block_size // 256) * 256)
        if w.prompt_len:
            caps.add(-(-b * w.prompt_len // 256) * 256)
    return sorted(caps)


def _splits(M, nx, bm, K, zmax):
    """Split count for M live rows (restated from the planner's rule)."""
    tiles = nx * (-(-M // bm))
    target = 256 if bm == 128 else 512
    S = 1
    while 2 * S <= zmax and tiles * 2 * S <= target and K % (2 * S * 128) == 0 and K // (2 * S) >= 256:
        S *= 2
    return S


def _extent_max(N, K, rows_cap, bm, bn, zmax):
    best = 0
    for M in range(1, rows_cap + 1):
        S = _splits(M, N // bn, bm, K, zmax)
        if S > 1:
            best = max(best, S * (-(-M // bm)) * bm * N)
    return best


def _resid_shapes(w):
    d, hdim = w.d_model, w.n_heads * w.head_dim
    shapes = [(d, hdim)]
    if w.n_experts == 0:
        shapes.append((d, w.ffn_dim))
    return shapes


@pytest.mark.parametrize("cfg", sorted(k for k in WORKLOADS if WORKLOADS[k].dtype == "bf16"))
def test_residual_workspace_covers_every_row_count(cfg):
    from paper_2609_33887_amd import bd
    w = WORKLOADS[cfg]
    for N, K in _resid_shapes(w):
        for rc in _rows_caps(w):
            bm, bn, zmax, wsf = bd.bd_plan_projection(N, K, rc, True)
            assert (bm, bn) in ((128, 256), (128, 128), (64, 64)) and 1 <= zmax <= 8
            need = _extent_max(N, K, rc, bm, bn, zmax)
            assert wsf == need, (N, K, rc, bm, wsf, need)


def test_plain_projections_do_not_split():
    from paper_2609_33887_amd import bd
    for w in WORKLOADS.values():
        if w.dtype != "bf16":
            continue
        for N, K in [(w.qkv_dim, w.d_model), (2 * max(w.ffn_dim, 64), w.d_model)]:
            for rc in _rows_caps(w):
                bm, bn, zmax, wsf = bd.bd_plan_projection(N, K, rc, False)
                assert zmax == 1 and wsf == 0 and N % bn == 0


def test_plain_projection_tiles():
    """Tile choice of plain (non-residual) bf16 projections: 128 x 256 on
    windows of at least 2,048 rows for products at least 8,192 wide, 128 x 128
    when that grid has at least 1,024 workgroups over the row capacity,
    64 x 128 on windows of at most 1,024 rows, else 64 x 64 (the query takes
    N and K multiples of 128 only)."""
    from paper_2609_33887_amd import bd
    # the dense-1024 step window (16 sequences x 64 rows): gate/up 8,192 wide
    assert bd.bd_plan_projection(8192, 1024, 1024, False)[:2] == (64, 128)
    # the same product on the MoE step window (4,096 rows): wide tiles; a
    # product half as wide there: a 128 x 128 grid of 32 x 32 = 1,024
    # workgroups
    assert bd.bd_plan_projection(8192, 1024, 4096, False)[:2] == (128, 256)
    assert bd.bd_plan_projection(4096, 1024, 4096, False)[:2] == (128, 128)
    # a narrow product on that window: 22 x 32 = 704 128 x 128 workgroups,
    # too few, and the window is over 1,024 rows
    assert bd.bd_plan_projection(2816, 2048, 4096, False)[:2] == (64, 64)
    # the multi-block window (6,144 rows): gate/up 16,384 wide
    assert bd.bd_plan_projection(16384, 2048, 6144, False)[:2] == (128, 256)
    for rc in (256, 512, 768, 1024):
        for N in (128, 256, 1024, 3072):
            bm, bn, zmax, _ = bd.bd_plan_projection(N, 1024, rc, False)
            assert (bm, bn) == (64, 128) and zmax == 1


def test_retired_192_row_tile_exceeds_the_old_fixed_workspace():
    """The removed 192 x 128 tile took the 512-workgroup target (every tile
    height but 128 did), so on the dense-1024 down projection (N 1024,
    K 4096) over a 1,024-row capacity it planned 6 row tiles x 8 column tiles
    with S = 8: 9.4 M floats of partials against the fixed 4.19 M-float
    workspace of 256 x 128 x 128 floats -- writes past the allocation, the
    illegal memory access that ended its decode.  The workspace is now sized
    per state from the plan, and a plan whose extent does not fit is refused."""
    old_fixed = 256 * 128 * 128
    assert _extent_max(1024, 4096, 1024, 192, 128, 8) == 8 * 6 * 192 * 1024 > old_fixed
    # the tiles in use stay within the same bound by construction
    for bm in (64, 128):
        assert _extent_max(1024, 4096, 1024, bm, bm, 8) <= old_fixed


def test_plan_query_errors():
    from paper_2609_33887_amd import bd
    with pytest.raises(bd.BDError) as e:
        bd.bd_plan_projection(0, 128, 256, True)
    assert e.value.status == bd.BD_EINVAL
    with pytest.raises(bd.BDError) as e:
        bd.bd_plan_projection(1000, 128, 256, True)
    assert e.value.status == bd.BD_EUNSUPPORTED
