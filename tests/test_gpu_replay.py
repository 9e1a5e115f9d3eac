"""Recorded launches (uniquan.record / Launches) replay the same work: two
layers built from the same seeded inputs, one stepped through the checked
wrappers, one through replays recorded on its first step, must agree bit for
bit after several steps (codes, What, loss, parameters)."""
import numpy as np
import pytest
import torch

import oracle.uniquan as O
from paper_2506_03781_amd import synth
from paper_2506_03781_amd import uniquan as uq
from paper_2506_03781_amd.layer import QuantLayer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    uq.lib()
    torch.cuda.set_device(0)


def _layer(m, p, k, g):
    lay = QuantLayer(m.W, m.X, m.s, k, g, delta=p["delta"], z_u=p["z_u"], s_r=p["s_r"], z_b=p["z_b"],
                     residual=True)
    lay.alpha.copy_(torch.from_numpy(np.asarray(p["alpha"], np.float32).reshape(-1)))
    lay.prepare()
    return lay


def _direct(lay, mode):
    lay.fq_fwd(mode)
    lay.recon(backward=False)
    uq.uniquan_layer_grad(lay.T, lay.R, lay.C, lay.Et, lay.Xt, lay.G)
    lay.fq_bwd_sgd()


@pytest.mark.parametrize("stream_kind", ["current", "side"])
def test_replay_matches_direct(stream_kind):
    k, g = 3, 128
    spec = synth.scaled(synth.WORKLOADS["attn4096"].matrices[0], R=384, C=512, T=256)
    m = synth.make_matrix(spec, 11)
    p = O.init_param_set_b(m.W, m.s, k, g)
    a, b = _layer(m, p, k, g), _layer(m, p, k, g)
    side = torch.cuda.Stream() if stream_kind == "side" else None
    rec = {}
    for step, mode in enumerate([uq.MAP_FULL, uq.MAP_LOCAL, uq.MAP_FROZEN, uq.MAP_LOCAL, uq.MAP_FROZEN]):
        _direct(a, mode)
        torch.cuda.synchronize()
        if mode not in rec:
            rec[mode] = uq.record(_direct, b, mode)
        else:
            rec[mode](side)
        torch.cuda.synchronize()
        for name in ("codes", "W_hat", "loss", "s", "alpha", "z_b", "Et"):
            x, y = getattr(a, name), getattr(b, name)
            assert torch.equal(x.view(torch.uint8) if x.dtype == torch.bfloat16 else x,
                               y.view(torch.uint8) if y.dtype == torch.bfloat16 else y), (step, name)
    assert len(rec[uq.MAP_LOCAL]) == 4
