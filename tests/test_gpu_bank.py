"""GPU parity of the orthogonal random-feature bank sampler (App. B.1) with the
float64 oracle (oracle.features.orthogonal_bank_from) on the same draws,
through the C ABI (include/linsimp_bank.h), with and without the QR sign
correction, including a last block cut short (m not a multiple of D).

The device factorises in float64 and writes float32: the bar is relative L2
<= 1e-6 and max |diff| <= 1e-6 max |Omega| (float32 rounding of the output).
"""

import numpy as np
import pytest
import torch

from oracle import features
from paper_2608_09307_amd import linsimp as L
from paper_2608_09307_amd.workloads import make_bank_draws

from helpers import rel_l2

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.mark.parametrize("sign_correct", [True, False])
@pytest.mark.parametrize("H,m,D", [(1, 32, 32), (3, 91, 32), (2, 128, 64), (2, 250, 64),
                                   (1, 128, 128), (2, 300, 128)])
def test_feature_bank_parity(H, m, D, sign_correct):
    print(f"[bank] H={H} m={m} D={D} sign_correct={sign_correct}", flush=True)
    gauss, radii = make_bank_draws(H, m, D, seed=81, device=DEV)
    om = L.feature_bank(gauss, radii, m, sign_correct)
    torch.cuda.synchronize()
    got = om.double().cpu().numpy()
    G = gauss.double().cpu().numpy()
    R = radii.double().cpu().numpy()
    ref = np.stack([features.orthogonal_bank_from(G[h], R[h], m, sign_correct) for h in range(H)])
    e = rel_l2(got, ref)
    mx = float(np.max(np.abs(got - ref)) / np.max(np.abs(ref)))
    print(f"       rel_l2={e:.2e} max={mx:.2e}", flush=True)
    assert e <= 1e-6 and mx <= 1e-6, (e, mx)


def test_feature_bank_structure_at_layer_size():
    """m = 4096, D = 128, 16 heads: row norms equal the radii and each block's
    directions are orthonormal (float32 output)."""
    H, m, D = 16, 4096, 128
    gauss, radii = make_bank_draws(H, m, D, seed=82, device=DEV)
    om = L.feature_bank(gauss, radii, m)
    torch.cuda.synchronize()
    o = om.double()
    r = radii.double().reshape(H, m)
    assert torch.allclose(o.norm(dim=-1), r, rtol=2e-6)
    dirs = (o / r[..., None]).reshape(H, m // D, D, D)
    eye = torch.eye(D, dtype=torch.float64, device=DEV)
    gram = dirs @ dirs.transpose(-1, -2)
    assert float((gram - eye).abs().max()) < 2e-6
