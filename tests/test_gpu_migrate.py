"""dit_migration_execute on the GPU: device buffers stand in for the ranks'
slices; applying a plan rebuilds every destination slice bit for bit as
direct slicing of the global tensor does (SP row layouts of the 720p token
matrix, box layouts of a channel-major latent, odd sizes that force narrow
copy units, a replicated field)."""
import numpy as np
import pytest
import torch

from gpu_util import log, require_gpu
from oracle import migrate as M

pytestmark = pytest.mark.gpu


def _run(kind, global_t, src, dst):
    B = require_gpu()
    shape = tuple(global_t.shape)
    eb = global_t.element_size()
    f = B.MigField(kind, shape, eb, src, dst)
    entries, n = B.migration_plan(f)
    sb = [global_t[tuple(slice(a, b) for a, b in zip(s, e))].contiguous().clone() for _, s, e in src]
    db = [torch.full([b - a for a, b in zip(s, e)], 7, dtype=global_t.dtype, device="cuda") for _, s, e in dst]
    B.migration_execute(f, entries, n, sb, db)
    torch.cuda.synchronize()
    for (r, s, e), got in zip(dst, db):
        want = global_t[tuple(slice(a, b) for a, b in zip(s, e))]
        assert torch.equal(got, want), (r, s, e)
    return n


@pytest.mark.parametrize("d1,d2", [(1, 8), (8, 2), (4, 3), (2, 4), (8, 8), (5, 7)])
def test_sp_token_layouts(d1, d2):
    log(f"case migrate tokens 75600x64 bf16 SP{d1} -> SP{d2}")
    g = torch.randn(75600, 64, device="cuda").to(torch.bfloat16)
    n = _run(M.SHARDED, g, M.row_layout(75600, list(range(d1)), [64]), M.row_layout(75600, list(range(8, 8 + d2)), [64]))
    log(f"  {n} entries")


def test_latent_boxes_fp32():
    log("case migrate latent 16x21x90x160 fp32, (f, h) boxes -> h bands")
    g = torch.randn(16, 21, 90, 160, device="cuda")
    src = [(3 * i + j, [0, fa, ha, 0], [16, fb, hb, 160]) for i, (fa, fb) in enumerate([(0, 7), (7, 21)])
           for j, (ha, hb) in enumerate([(0, 30), (30, 61), (61, 90)])]
    dst = [(10 + k, [0, 0, a, 0], [16, 21, b, 160]) for k, (a, b) in enumerate([(0, 23), (23, 45), (45, 68), (68, 90)])]
    _run(M.SHARDED, g, src, dst)


def test_odd_sizes_narrow_units():
    log("case migrate 7x13x5 bf16 and 3x3 int8-sized")
    g = torch.randn(7, 13, 5, device="cuda").to(torch.bfloat16)
    src = M.row_layout(7, [0, 1, 2], [13, 5])
    dst = [(5, [0, 3, 1], [7, 11, 4]), (6, [2, 0, 0], [5, 13, 5])]
    _run(M.SHARDED, g, src, dst)
    g8 = torch.randint(0, 255, (9, 3), device="cuda", dtype=torch.uint8)
    _run(M.SHARDED, g8, M.row_layout(9, [0, 1], [3]), M.row_layout(9, [2, 3, 4, 5], [3]))


def test_replicated():
    log("case migrate replicated 33x65 fp32 to 4 ranks")
    g = torch.randn(33, 65, device="cuda")
    whole = ([0, 0], [33, 65])
    _run(M.REPLICATED, g, [(0,) + whole, (1,) + whole], [(r,) + whole for r in (1, 2, 3, 4)])
