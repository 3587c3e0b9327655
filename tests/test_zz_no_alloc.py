"""The no-allocation projection (galore_project_noalloc) against the same
projection with a caller workspace (galore_project), through the C ABI, run
with -m gpu: two calls in a row, the second with a smaller input, in both
orientations; the results are bit-identical (same kernels, the scratch only
moves into the library's own device array), and sampled entries are checked
against host fp64 at the projection's tolerance (|x - ref| <= 1e-6 + 1e-5 |ref|)."""
import numpy as np
import pytest

import galore_inputs as gi
from metrics import max_rel_violation

pytestmark = pytest.mark.gpu


def _orthonormal(b, s, r, seed):
    import torch
    g = torch.Generator(device="cuda").manual_seed(seed)
    z = torch.randn((b, s, r), generator=g, device="cuda")
    return torch.linalg.qr(z)[0].contiguous()


@pytest.mark.parametrize("shapes", [((4096, 11008, 1024, 2), (1024, 2752, 256, 3)),
                                    ((11008, 4096, 1024, 2), (2736, 1024, 256, 1))])
def test_project_noalloc_equals_workspace_call(shapes):
    import torch
    import paper_2504_20437_amd as gl
    for call, (m, n, r, B) in enumerate(shapes):
        s, l = min(m, n), max(m, n)
        print("no-alloc projection call %d: %d x %dx%d r=%d" % (call, B, m, n, r), flush=True)
        G = gi.torch_planted_group(m, n, B, gi.spectrum_power(s, 0.7), 1e-4, seed=7000 + call, dtype="bf16")
        P = _orthonormal(B, s, r, 7100 + call)
        R_ws = gl.galore_project(P, G)                        # caller workspace (allocated by the binding)
        R_na = torch.full((B, r, l), float("nan"), device="cuda")
        gl.galore_project_noalloc(P, G, R_na)
        torch.cuda.synchronize()
        assert torch.equal(R_na, R_ws)
        rng = np.random.default_rng(call)
        ii, jj = rng.integers(0, r, 48), rng.integers(0, l, 48)
        for b in range(B):
            Pb = P[b].double().cpu().numpy()
            A = G[b].double().cpu().numpy()
            A = A if m <= n else A.T
            ref = np.array([Pb[:, i] @ A[:, j] for i, j in zip(ii, jj)])
            got = R_na[b].double().cpu().numpy()[ii, jj]
            assert max_rel_violation(got, ref, 1e-5, 1e-6) <= 1.0
