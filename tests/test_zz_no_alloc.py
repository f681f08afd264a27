"""The allocation-free backward-weights entry point against the workspace one.

cf_conv3d_bwd_weight_noalloc runs the same kernels as cf_conv3d_bwd_weight
with the split reduction's partials in the library's per-GPU scratch region
instead of a caller workspace, so its dW must equal the workspace entry
point's bit for bit.  Two calls in a row on the same GPU, the second with a
smaller input: the region then still holds the first call's partials, which
the second call must overwrite wherever it reads.
"""
import numpy as np
import pytest
import torch

from paper_1808_04728_amd import binding as B
from tests._util import dev

pytestmark = pytest.mark.gpu

# (N, (D,H,W), CI, CO, k, stride): larger first, then smaller, per dtype; they
# cover the first-layer, 16 -> 32, deep-layer and generic weight-gradient kernels
SEQS = {
    "bf16": [(2, (32, 32, 32), 32, 64, 4, 2), (1, (16, 16, 16), 16, 32, 4, 1), (1, (32, 32, 32), 1, 16, 3, 1)],
    "f32": [(1, (32, 32, 32), 32, 64, 4, 2), (1, (16, 16, 16), 16, 32, 4, 1), (1, (8, 8, 8), 64, 64, 3, 1)],
}


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_noalloc_matches_workspace_entry_point(dt):
    rng = np.random.default_rng(77)
    sizes = []
    for N, dhw, ci, co, k, s in SEQS[dt]:
        desc = B.make_desc(N, dhw, ci, co, k, s, "same", dt)
        od = B.cf_conv3d_out_shape(desc)
        x = dev(rng.standard_normal((N, *dhw, ci)), dt)
        dz = dev(rng.standard_normal((N, *od, co)), dt)
        need = B.cf_conv3d_bwd_weight_workspace_size(desc)
        assert 0 < need <= 16 << 20
        sizes.append(need)
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        ref = torch.full((k, k, k, ci, co), float("nan"), device="cuda")
        got = torch.full_like(ref, float("nan"))
        B.cf_conv3d_bwd_weight(desc, x, dz, ref, ws)
        B.cf_conv3d_bwd_weight_noalloc(desc, x, dz, got)
        torch.cuda.synchronize()
        assert torch.isfinite(ref).all()
        assert torch.equal(got, ref), (N, dhw, ci, co, k, s)
    assert sizes[1] < sizes[0]  # the second call of each sequence is the smaller one
