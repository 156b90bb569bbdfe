"""GPU parity of the dense Adam update (the servers' and workers' update of
Algorithm 1, trained with Adam in section 7.2) through the C ABI against the
float64 oracle.  Each step is checked on the GPU's own float32 state: the
oracle takes the GPU's parameters and moments before the step, and the move
of the parameters, m and v are compared after it.  Sizes: one element, a
ragged 257, the image model's 1,066,060 parameters (4096-256-64-12 weights
and biases), and 2^21 + 77 (past one pass of the grid-stride loop), plus arrays that start
off 16-byte boundaries (the element-wise kernel instead of the 16-byte one).  The
bf16 copy must be bit-exact: round-to-nearest-even of the float32 result."""
import numpy as np
import pytest
import torch

from oracle import oracle
from tests.parity import RTOL, assert_close

pytestmark = pytest.mark.gpu
F32 = RTOL["f32"]


@pytest.mark.parametrize("n,off", [(1, 0), (257, 0), (4096 * 256 + 256 + 256 * 64 + 64 + 64 * 12 + 12, 0),
                                   ((1 << 21) + 77, 0), (1003, 1), (4096, 3)])
def test_adam_update_matches_oracle(n, off):
    """off > 0: every array starts `off` elements into its allocation, so the
    16-byte path is not taken (the element-wise kernel runs)."""
    from paper_1711_06505_amd import ams
    print(f"adam n={n} off={off}", flush=True)
    rng = np.random.default_rng(n)
    p = torch.empty(n + off, device="cuda")[off:]
    p.copy_(torch.from_numpy((rng.standard_normal(n) * 0.05).astype(np.float32)))
    m = torch.zeros(n + off, device="cuda")[off:]
    v = torch.zeros(n + off, device="cuda")[off:]
    pb = torch.empty(n + off, dtype=torch.bfloat16, device="cuda")[off:]
    for t in (1, 2, 3, 24001):
        g = (rng.standard_normal(n) * 10.0 ** rng.uniform(-4, 0, n)).astype(np.float32)
        if n > 8:
            g[::7] = 0.0
        p0, m0, v0 = (x.cpu().numpy().astype(np.float64) for x in (p, m, v))
        lr = oracle.paper_lr(t)
        rp, rm, rv = oracle.adam(p0, g, m0, v0, lr=lr, t=t)
        gd = torch.empty(n + off, device="cuda")[off:]
        gd.copy_(torch.from_numpy(g))
        ams.ams_adam_update(p, gd, m, v, lr, t, param_bf16=pb.view(torch.int16))
        torch.cuda.synchronize()
        pg = p.cpu().numpy().astype(np.float64)
        assert_close(pg - p0, rp - p0, F32, f"param move (t={t})")
        assert_close(m, rm, F32, f"m (t={t})")
        assert_close(v, rv, F32, f"v (t={t})")
        assert torch.equal(pb.view(torch.int16), p.to(torch.bfloat16).view(torch.int16)), "bf16 copy"
