"""The allocation-free GRU entry point (isam_gru_forward_noalloc), called through the C ABI,
against the workspace entry point (isam_gru_forward) on the same inputs: two calls in a row
on the shared static scratch, the second smaller than the first, under both schedules."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests._util import TOL_BF16, TOL_F32, bits, to_gpu

pytestmark = pytest.mark.gpu

import paper_1810_09958_amd as isam


def _inputs(T, B, I, H, seed, dt):
    x = synth.normal(seed, 3, (T, B, I))
    W = synth.uniform(seed, 0, (3 * H, I), -1 / 8, 1 / 8)
    U = synth.uniform(seed, 1, (3 * H, H), -1 / 8, 1 / 8)
    b = synth.normal(seed, 2, (3 * H,), scale=0.1)
    bhn = synth.normal(seed, 5, (H,), scale=0.1)
    h0 = synth.normal(seed, 4, (B, H), scale=0.5)
    if dt == "bf16":
        x, W, U = bits(x), bits(W), bits(U)
    return x, W, U, b, bhn, h0


@pytest.mark.parametrize("mode", ["persistent", "steps"])
@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_noalloc_matches_workspace_entry_point(mode, dt, monkeypatch):
    monkeypatch.setenv("ISAM_GRU_MODE", mode)
    L = isam.lib()
    wt = isam.ISAM_BF16 if dt == "bf16" else isam.ISAM_F32
    for (T, B, I, H, seed) in [(12, 33, 96, 256, 1), (5, 4, 40, 64, 2)]:   # second call smaller
        x, W, U, b, bhn, h0 = _inputs(T, B, I, H, seed, dt)
        xg, Wg, Ug, bg, bhng, h0g = (to_gpu(a) for a in (x, W, U, b, bhn, h0))
        ref_hs, ref_hT = isam.gru_forward(xg, Wg, Ug, bias=bg, bias_hn=bhng, h0=h0g)
        hs = torch.full((T, B, H), float("nan"), device="cuda")
        hT = torch.full((B, H), float("nan"), device="cuda")
        rc = L.isam_gru_forward_noalloc(T, B, I, H, wt, xg.data_ptr(), h0g.data_ptr(), Wg.data_ptr(),
                                        Ug.data_ptr(), bg.data_ptr(), bhng.data_ptr(), hs.data_ptr(),
                                        hT.data_ptr(), torch.cuda.current_stream().cuda_stream)
        assert rc == 0, L.isam_last_error()
        torch.cuda.synchronize()
        # same kernels, same plan: the same bits as the workspace entry point
        assert torch.equal(hs, ref_hs) and torch.equal(hT, ref_hT), f"T={T} B={B} H={H}"
        err = float(np.max(np.abs(hs.cpu().numpy().astype(np.float64) - oracle.gru(x, W, U, b, bhn, h0))))
        assert err <= (TOL_BF16 if dt == "bf16" else TOL_F32), err
