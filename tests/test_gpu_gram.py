"""GPU parity of the Gram-forming kernels whose work is split differently from the oracle's
plain sums: the feature Gram of bf16 cells on the matrix cores (section 4: the feature-mode
spectrum stays exact) and the second CholeskyQR pass of the FlashJoLT range finder split over
row chunks (section 5).

The feature Gram of a bf16 cell is a sum of exact products (bf16 x bf16 fits fp32), so only
the fp32 accumulation and the fp32 eigensolver separate it from the fp64 oracle: the
feature spectrum is checked at 1e-5 of its largest eigenvalue, the energy (fp64 on both
sides) at 1e-10 relative.  Row counts are chosen so the 64-row stages end ragged and, at
T = 4096, the rows of a cell are spread over several workgroups.
"""
import numpy as np
import pytest

import kvsynth
import paper_2607_12550_amd as J
from gpu_util import ctx, device_cells, note, workspace
from oracle import tucker as otk

pytestmark = pytest.mark.gpu


def kv_cell(T, H, d=128, seed=0, alpha=1.5, tensor=0):
    return kvsynth.layer_kv(layer=0, tensor=tensor, n_heads=H, T=T, d=d, alpha=alpha,
                            data_seed=seed)[0].astype(np.float64)


@pytest.mark.parametrize("T,H", [(1000, 4), (4096, 8)])
def test_bf16_feature_spectrum_and_energy_tight(T, H):
    cells = [kv_cell(T, H, seed=11), kv_cell(T, H, seed=12, alpha=0.7, tensor=1)]
    xs, ex, desc = device_cells(cells, "bf16")
    o = J.SpectrumOpts(J.JOLT_FLASH, 16, 0.0, 4, 0)
    ws = workspace(desc, 2, o)
    note("jolt_spectrum (feature Gram on the matrix cores)", T, H)
    E, _, lamd = J.jolt_spectrum(ctx(), desc, xs, [1, 2], o, ws)
    for c in range(2):
        lam_d, _ = otk.feature_spectrum(ex[c])
        assert abs(E[c] / otk.energy(ex[c]) - 1) < 1e-10
        np.testing.assert_allclose(lamd[c], lam_d, rtol=0, atol=1e-5 * lam_d[0])


def test_flash_second_gram_split_over_rows_matches_oracle():
    """T = 4096 rows: the second CholeskyQR pass's Gram of the T x l basis runs as two row
    chunks summed in fp64; q = 40, p = 10, one power iteration, against the oracle run with
    the same sketch (bf16 tolerance, 1e-3)."""
    cells = [kv_cell(4096, 4, seed=21), kv_cell(4096, 4, seed=22, alpha=0.7, tensor=1)]
    xs, ex, desc = device_cells(cells, "bf16")
    o = J.SpectrumOpts(J.JOLT_FLASH, 40, 0.0, 10, 1)
    ws = workspace(desc, 2, o)
    seeds = [31, 32]
    note("jolt_spectrum flash, T = 4096")
    E, lamT, _ = J.jolt_spectrum(ctx(), desc, xs, seeds, o, ws)
    for c in range(2):
        lam, _, _ = otk.token_spectrum_flash(ex[c], q=40, p=10, power_iters=1, seed=seeds[c])
        Er = otk.energy(ex[c])
        np.testing.assert_allclose(lamT[c, :40], lam[:40], rtol=0, atol=1e-3 * lam[0])
        assert abs(lamT[c, 40] - lam[40]) <= 1e-3 * Er
        np.testing.assert_allclose(lamT[c].sum(), Er, rtol=1e-9)
