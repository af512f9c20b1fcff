"""h3_statepass_conv_noalloc (state passing on the library's static scratch,
for callers that cannot allocate) against h3_statepass_conv on the same
inputs: two calls in a row, the second smaller and on the other state-passing
path (the first uses the fused initial-state term, the second the separate
correction term), so the second runs on scratch the first left behind."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from tests._util import check, cplx64, cplx_to_f32pairs, f32dev, to_dev

pytestmark = pytest.mark.gpu


def _inputs(w):
    A, B, C, dt = w.ssm.complex64()
    Ab, Bb = oracle.zoh(A, B, dt)
    return (f32dev(cplx_to_f32pairs(Ab)), f32dev(cplx_to_f32pairs(Bb)), f32dev(w.ssm.C), f32dev(w.D))


def test_noalloc_matches_workspace_entry_point():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2212_14052_amd as h3
    cases = [  # (B, H, L, chunk, dtype, seed): the second is smaller
        (2, 256, 65536, 8192, workloads.F16, 1),
        (1, 64, 16384, 2048, workloads.BF16, 2),
    ]
    need = [h3.workspace_size(h3.OP_STATEPASS, B, H, L, 64, ch, {workloads.F16: h3.F16, workloads.BF16: h3.BF16}[dt])
            for B, H, L, ch, dt, _ in cases]
    assert need[1] < need[0] <= (128 << 20)
    for B, H, L, chunk, dtype, seed in cases:
        print(f"noalloc case B={B} H={H} L={L} chunk={chunk} {dtype}", flush=True)
        w = workloads.statepass_workload("t", B, H, L, chunk, dtype, seed=seed, dt_lo=1e-4, dt_hi=1e-2,
                                         x0_scale=0.5)
        u = to_dev(w.u, dtype)
        args = _inputs(w)
        x0 = f32dev(w.x0)
        y_ref, x_ref = h3.statepass_conv(u, *args, chunk, x0=x0)
        y, xf = h3.statepass_conv_noalloc(u, *args, chunk, x0=x0)
        torch.cuda.synchronize()
        check(y, y_ref.float().cpu().numpy(), 2e-2, "y")
        check(cplx64(xf.cpu().numpy()), cplx64(x_ref.cpu().numpy()), 2e-2, "x_final")
        # same kernels on the same inputs: identical results
        assert torch.equal(y, y_ref)
        assert torch.equal(xf, x_ref)
