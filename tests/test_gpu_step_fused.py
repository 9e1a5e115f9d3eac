"""GPU parity of uniquan_fq_step: the straight-through backward with the SGD
update of step t fused with the forward of step t + 1.

It must equal uniquan_fq_bwd_sgd followed by uniquan_fq_fwd (or
uniquan_fq_fwd_residual) bit for bit in every output (s, alpha, z_B, the
code bytes, What), both of which are checked against the oracle elsewhere;
and, against the oracle directly, the codes of the next step agree on
>= 99.9% of the weights (the device's group sums are fp32, the oracle's fp64,
so a weight on a level midpoint may round the other way) and the updated
parameters' steps within 1e-2.  Inputs: the seeded generator and the
oracle's parameter recipe; nothing the device produced feeds the oracle.
"""
import numpy as np
import pytest
import torch

import oracle.uniquan as O
from paper_2506_03781_amd import synth
from paper_2506_03781_amd import uniquan as uq

import test_gpu_parity as P

pytestmark = pytest.mark.gpu

F32 = np.float32
dev, host, close = P.dev, P.host, P.close
LR_F, LR_B = 0.005, 0.0005


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    uq.lib()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _state(m, p, codes, k):
    return dict(s=dev(m.s), alpha=dev(p["alpha"].reshape(-1)), z_b=dev(p["z_b"]),
                codes=dev(codes, torch.uint8).reshape(-1))


def _run_pair(m, p, k, g, codes, G, mode, resid, wdt, gdt, odt):
    """Fused call and the two-call sequence on identical copies; returns both states."""
    R, C = m.W.shape
    W = dev(m.W, wdt)
    Gd = dev(G, gdt)
    fixed = (dev(p["s_r"]), dev(p["delta"]), dev(p["z_u"]))
    a, b = _state(m, p, codes, k), _state(m, p, codes, k)
    Wa = torch.empty(R * C, dtype=odt, device="cuda")
    Wb = torch.empty_like(Wa)
    uq.uniquan_fq_step(R, C, k, g, W, a["s"], *fixed, a["alpha"], a["z_b"], a["codes"], Gd, LR_F, LR_B, mode, Wa,
                       residual=resid)
    uq.uniquan_fq_bwd_sgd(R, C, k, g, W, b["s"], fixed[0], fixed[1], fixed[2], b["alpha"], b["z_b"], b["codes"], Gd,
                          None, None, None, LR_F, LR_B)
    fwd = uq.uniquan_fq_fwd_residual if resid else uq.uniquan_fq_fwd
    fwd(R, C, k, g, W, b["s"], *fixed, b["alpha"], b["z_b"], mode, b["codes"], Wb)
    torch.cuda.synchronize()
    a["W_hat"], b["W_hat"] = Wa, Wb
    return a, b


def _assert_same(a, b, what):
    for n in ("s", "alpha", "z_b", "codes", "W_hat"):
        assert torch.equal(a[n], b[n]), f"{what}: {n} differs from the two-call sequence"


@pytest.mark.parametrize("mode", [uq.MAP_FULL, uq.MAP_LOCAL, uq.MAP_FROZEN])
@pytest.mark.parametrize("k", [1, 2, 3, 4, 7])
@pytest.mark.parametrize("resid", [False, True])
def test_step_equals_two_passes(mode, k, resid):
    g = 128
    m = P.small_matrix(37, 384, 100 + k)
    p = P.params(m.W, m.s, k, g, "B")
    p["s_r"] = synth.perturb(p["s_r"], 0.01, k, 23)
    f0 = O.fq_fwd(m.W, m.s, p["alpha"], p["z_b"], k, g, p["s_r"], p["delta"], p["z_u"])
    G = synth.round_to_bf16(np.random.default_rng(k).standard_normal(m.W.shape).astype(F32))
    a, b = _run_pair(m, p, k, g, f0["codes"], G, mode, resid, torch.bfloat16, torch.bfloat16, torch.bfloat16)
    _assert_same(a, b, f"k={k} mode={mode}")


@pytest.mark.parametrize("g,k,mode", [(8, 3, uq.MAP_LOCAL), (32, 4, uq.MAP_FULL), (512, 2, uq.MAP_LOCAL),
                                      (8, 7, uq.MAP_LOCAL), (8, 7, uq.MAP_FROZEN), (1024, 3, uq.MAP_LOCAL)])
def test_step_group_sizes_and_dtypes(g, k, mode):
    """Every group size path: the fused kernel (g <= 512), the two-pass
    sequence where the neighbour table does not fit (g = 8, k = 7, LOCAL) and
    for large groups; fp32 weights, fp32 dL/dWhat and fp32 What."""
    m = P.small_matrix(9, 2048, 110 + g + k, dtype="f32")
    p = P.params(m.W, m.s, k, g, "B")
    f0 = O.fq_fwd(m.W, m.s, p["alpha"], p["z_b"], k, g, p["s_r"], p["delta"], p["z_u"])
    G = np.random.default_rng(g).standard_normal(m.W.shape).astype(F32)
    for wdt, gdt, odt in ((torch.float32, torch.float32, torch.float32), (torch.bfloat16, torch.float32, torch.bfloat16)):
        a, b = _run_pair(m, p, k, g, f0["codes"], G, mode, False, wdt, gdt, odt)
        _assert_same(a, b, f"g={g} k={k} {wdt} {gdt} {odt}")


def test_step_against_oracle():
    """The fused step against the oracle's own chain (fp64 backward, fp32 SGD,
    fp32 forward on its own updated parameters)."""
    k, g = 3, 128
    m = P.small_matrix(64, 1024, 120)
    p = P.params(m.W, m.s, k, g, "B")
    R, C = m.W.shape
    Gn = R * C // g
    f0 = O.fq_fwd(m.W, m.s, p["alpha"], p["z_b"], k, g, p["s_r"], p["delta"], p["z_u"])
    G = synth.round_to_bf16(np.random.default_rng(5).standard_normal(m.W.shape).astype(F32))
    a, _ = _run_pair(m, p, k, g, f0["codes"], G, uq.MAP_LOCAL, True, torch.bfloat16, torch.bfloat16, torch.bfloat16)
    bw = O.fq_bwd(m.W, m.s, p["alpha"], p["z_b"], f0["codes"], G, k, g, p["s_r"], p["delta"], p["z_u"])
    sgd = lambda th, gr, lr: (np.asarray(th, F32) - (F32(lr) * np.asarray(gr, np.float64).astype(F32))).astype(F32)  # noqa: E731
    s1, a1, z1 = sgd(m.s, bw["grad_s"], LR_F), sgd(p["alpha"], bw["grad_alpha"], LR_B), sgd(p["z_b"], bw["grad_z_b"], LR_B)
    close(host(a["s"]).reshape(R, C) - m.s, s1 - m.s, what="s step")
    close(host(a["alpha"]).reshape(Gn, k) - p["alpha"], a1 - p["alpha"], tol=2e-2, what="alpha step")
    close(host(a["z_b"]) - p["z_b"], z1 - p["z_b"], tol=2e-2, what="z_b step")
    f1 = O.fq_fwd(m.W, s1, a1, z1, k, g, p["s_r"], p["delta"], p["z_u"], O.MAP_LOCAL, f0["codes"])
    agree = np.mean(host(a["codes"]).reshape(R, C) == f1["codes"])
    assert agree >= 0.999, agree


@pytest.mark.parametrize("mode", [uq.MAP_LOCAL, uq.MAP_FROZEN])
def test_step_full_size_7b_gate(mode):
    """The 7B gate projection (11008 x 4096, k = 3, g = 128) in the launch
    configuration the bench times: bit-identical to the two-call sequence
    over the whole matrix."""
    spec = synth.WORKLOADS["mlp7b"].matrices[0]
    m = synth.make_matrix(synth.scaled(spec, T=8), 1)
    k, g = 3, 128
    import test_gpu_fullsize as FS
    p = FS.step_params(m.W, k, g, 1)
    prev = synth.random_codes(m.R, m.C, k, 2)
    G = synth.round_to_bf16((0.01 * np.random.default_rng(6).standard_normal(m.W.shape)).astype(F32))
    a, b = _run_pair(m, p, k, g, prev, G, mode, True, torch.bfloat16, torch.bfloat16, torch.bfloat16)
    _assert_same(a, b, "7B gate")


@pytest.mark.parametrize("mode", [uq.MAP_FULL, uq.MAP_LOCAL, uq.MAP_FROZEN])
@pytest.mark.parametrize("k,R,C,g", [(2, 6, 11008, 11008), (3, 12, 8192, 4096), (4, 10, 2064, 1032),
                                     (7, 4, 4096, 4096), (3, 3, 16384, 16384)])
@pytest.mark.parametrize("resid", [False, True])
def test_step_equals_two_passes_row_groups(mode, k, R, C, g, resid):
    """Groups of whole rows (one workgroup per group, every lane holding up
    to 8 chunks between the backward and the forward): the fused pass equals
    the backward with the update followed by the forward, bit for bit, at
    the 7B row lengths, a ragged chunk count (1032 = 129 chunks) and the
    largest group the fused pass takes (16384); fp32 What once."""
    m = P.small_matrix(R, C, 300 + k + g)
    p = P.params(m.W, m.s, k, g, "B")
    p["s_r"] = synth.perturb(p["s_r"], 0.01, k, 29)
    f0 = O.fq_fwd(m.W, m.s, p["alpha"], p["z_b"], k, g, p["s_r"], p["delta"], p["z_u"])
    G = synth.round_to_bf16(np.random.default_rng(k + g).standard_normal(m.W.shape).astype(F32))
    odt = torch.float32 if (k == 3 and g == 4096) else torch.bfloat16
    a, b = _run_pair(m, p, k, g, f0["codes"], G, mode, resid, torch.bfloat16, torch.bfloat16, odt)
    _assert_same(a, b, f"k={k} g={g} mode={mode}")
