"""GPU parity of the path-weight-shared equivariant linear layer
(tdn_ps_linear: y^(l) = x^(l) W for every degree) against the oracle's
degree-by-degree layer.ps_linear, through the C ABI."""
import numpy as np
import pytest
import torch

import paper_2507_01131_amd as tdn
import workloads
from oracle import layer
from tests._gpu_helpers import TOL_BF16, TOL_F32, rel_err

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("N,L,C,bf16", [(37, 3, 16, False), (37, 3, 48, False), (50, 0, 128, False),
                                        (41, 4, 128, False), (29, 6, 256, False), (37, 2, 64, True),
                                        (3200, 4, 128, False), (0, 2, 32, False)])
def test_ps_linear_matches_the_per_degree_layer(N, L, C, bf16):
    rng = np.random.default_rng(N + L + C)
    d = (L + 1) ** 2
    x = rng.standard_normal((N, d, C)).astype(np.float32)
    W = (rng.standard_normal((C, C)) / np.sqrt(C)).astype(np.float32)
    if bf16:
        wb = workloads.bf16_round(W)
        Wt = torch.from_numpy(wb.view(np.int16)).cuda().view(torch.bfloat16)
        W = workloads.bf16_to_f32(wb)
    else:
        Wt = torch.from_numpy(W).cuda()
    y = tdn.ps_linear(torch.from_numpy(x).cuda(), Wt)
    torch.cuda.synchronize()
    if N == 0:
        assert y.shape == (0, d, C)
        return
    ref = layer.ps_linear(x, W, L)
    assert rel_err(y.cpu().numpy(), ref) < (TOL_BF16 if bf16 else TOL_F32)
