"""The HIP quantizer's variance against the oracle's exact form: over many Philox steps,
the mean of sum (g_hat - x)^2 of the PSQ (samples) and PCQ (channels) estimates,
dequantized from the codes and scales fqt_agp_scq_quantize returns, must match
quantizer_variance within five standard errors.  This checks the whole distribution of the
GPU quantizer (the AGP masks, the 1/p rescale, stochastic rounding), not one draw."""
import sys

import numpy as np
import pytest

from oracle import fqt as ofqt
from paper_2408_14267_amd.workloads import WORKLOADS, draw_layer

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def dequantized(fqt, q, N, D, P):
    """(PSQ estimate, PCQ estimate) as float64 [N][D][P] from the device buffers of q."""
    R = N * P
    Wd, Wr = (D + 63) // 64, (R + 63) // 64
    out = []
    for side in ("psq", "pcq"):
        count = int(getattr(q, side + "_count").item())
        kept = getattr(q, side + "_kept")[:count].long()
        S = getattr(q, side + "_scale").double()[kept]
        Z = getattr(q, side + "_offset").double()[kept]
        g = torch.zeros((N, D, P), dtype=torch.float64, device="cuda")
        if side == "psq":
            codes = q.psq_codes.view(2 * Wd, R, 32).permute(1, 0, 2).reshape(R, 64 * Wd)[:, :D]
            rows = codes[:count * P].double().view(count, P, D).permute(0, 2, 1)
            g[kept] = S[:, None, None] * rows + Z[:, None, None]
        else:
            codes = q.pcq_codes.view(2 * Wr, D, 32).permute(1, 0, 2).reshape(D, 64 * Wr)[:, :R]
            rows = codes[:count].double().view(count, N, P).permute(1, 0, 2)
            g[:, kept] = S[None, :, None] * rows + Z[None, :, None]
        out.append(g)
    return out


@pytest.mark.parametrize("bits,mode", [(1, 2), (2, 0), (4, 0), (8, 0)],
                         ids=["1bit_psq_no_agp", "b2_agp", "b4_agp", "b8_agp"])
def test_gpu_quantizer_variance_matches_exact(bits, mode):
    from paper_2408_14267_amd import fqt
    wl = WORKLOADS["resnet18_32px"]
    layer = wl.layers[5]                        # l2.0.c1: N = 128, D = 128, 4 x 4 maps
    print(f"[gpu variance] {layer.name} b={bits} mode={mode}", flush=True)
    sys.stdout.flush()
    _, _, dy = draw_layer(layer, wl.recipe, 5)
    N, D, P = layer.N, layer.D, layer.Ho * layer.Wo
    desc = fqt.layer_desc(layer)
    x = torch.from_numpy(dy).cuda().double().view(N, D, P)
    dY = torch.from_numpy(dy).cuda()
    S = 160
    tot = {"samples": [], "channels": []}
    for step in range(S):
        cfg = fqt.quant_cfg(bits, mode, 17, step, 4)
        q = fqt.QGrad(desc, cfg)
        fqt.fqt_agp_scq_quantize(desc, cfg, dY, q, fqt.workspace(desc, cfg, fqt.FQT_WS_QUANTIZE))
        gs, gc = dequantized(fqt, q, N, D, P)
        tot["samples"].append(float(((gs - x) ** 2).sum()))
        tot["channels"].append(float(((gc - x) ** 2).sum()))
    for side in ("samples", "channels"):
        exact = float(ofqt.quantizer_variance(dy, bits, mode, side).sum())
        t = np.array(tot[side])
        se = t.std(ddof=1) / np.sqrt(S)
        assert abs(t.mean() - exact) <= 5 * se + 1e-9 * exact, (side, t.mean(), exact, se)
