"""uniquan_layer_recon_noalloc (loss partials in the library's fixed device
array, nothing allocated by the call) against uniquan_layer_recon with a
caller workspace: the same kernels in the same order, so loss, Et and
dL/dWhat must agree bit for bit.  Two calls in a row, the second smaller,
so the second reads only partials it wrote itself."""
import numpy as np
import pytest
import torch

from paper_2506_03781_amd import uniquan as uq

pytestmark = pytest.mark.gpu


def _case(T, R, C, seed, target):
    rs = np.random.default_rng(seed)
    X = torch.from_numpy(rs.standard_normal((T, C)).astype(np.float32)).cuda().to(torch.bfloat16)
    Wh = torch.from_numpy((0.02 * rs.standard_normal((R, C))).astype(np.float32)).cuda().to(torch.bfloat16)
    Yt = torch.from_numpy((0.2 * rs.standard_normal((R, T))).astype(np.float32)).cuda() if target else None
    Xt = torch.empty(C, T, dtype=torch.bfloat16, device="cuda")
    uq.uniquan_transpose_bf16(T, C, X, Xt)
    return X, Xt, Wh, Yt


def _with_ws(T, R, C, X, Xt, Wh, Yt):
    loss = torch.zeros(1, device="cuda")
    Et = torch.empty(R, T, dtype=torch.bfloat16, device="cuda")
    G = torch.empty(R, C, dtype=torch.bfloat16, device="cuda")
    part = torch.empty(uq.uniquan_recon_ws(T, R, C), device="cuda")
    uq.uniquan_layer_recon(T, R, C, X, Xt, Wh, Yt, loss, Et, part, G)
    return loss, Et, G


def _noalloc(T, R, C, X, Xt, Wh, Yt):
    loss = torch.full((1,), -1.0, device="cuda")
    Et = torch.empty(R, T, dtype=torch.bfloat16, device="cuda")
    G = torch.empty(R, C, dtype=torch.bfloat16, device="cuda")
    uq.uniquan_layer_recon_noalloc(T, R, C, X, Xt, Wh, Yt, loss, Et, G)
    return loss, Et, G


@pytest.mark.parametrize("target", [False, True])
def test_noalloc_matches_workspace_entry(target):
    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    # 1536 x 1024 loss tiles: 24 workgroups of 256 x 256; then 200 x 136 (ragged, 128 x 128 tiles)
    for (T, R, C, seed) in ((1024, 1536, 512, 1), (136, 200, 264, 2)):
        args = _case(T, R, C, seed, target)
        ref = _with_ws(T, R, C, *args)
        got = _noalloc(T, R, C, *args)
        torch.cuda.synchronize()
        assert float(got[0].item()) == float(ref[0].item()), (T, R, C)
        assert torch.equal(got[1], ref[1]) and torch.equal(got[2], ref[2]), (T, R, C)


def test_noalloc_rejects_oversize():
    T, R = 1 << 16, 1 << 20     # 2^36 outputs: far more partials than the fixed array holds
    assert uq.uniquan_recon_ws(T, R, 8) > uq.lib().uniquan_recon_noalloc_max_partials()
    fake = 1 << 20              # aligned, never dereferenced: the call fails before any HIP call
    st = uq.lib().uniquan_layer_recon_noalloc(T, R, 8, fake, None, fake, None, fake, fake, None, uq.UQ_BF16, None)
    assert st == uq.UQ_EUNSUPPORTED and b"scratch" in uq.lib().uniquan_last_error()
