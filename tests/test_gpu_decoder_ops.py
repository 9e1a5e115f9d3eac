"""GPU parity of the decoder-block operations (csrc/block_attn.hip and the
strided-batch GEMM) against oracle/block_decoder.py and plain definitions,
on seeded inputs generated here (never from device output).  Bars: layout
moves and fp32 adds bit-exact; bf16 outputs within one rounding (2^-8
relative) of the fp64 value plus the fp32 arithmetic before it; fp32 outputs
within 1e-5 of the row's scale."""
import numpy as np
import pytest
import torch

import oracle.block_decoder as D
import oracle.uniquan as O
from paper_2506_03781_amd import uniquan as uq

pytestmark = pytest.mark.gpu
F32 = np.float32


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    uq.lib()
    torch.cuda.set_device(0)


def dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, F32))).to("cuda").to(dtype).contiguous()


def host(t):
    return (t.float() if t.dtype == torch.bfloat16 else t).cpu().numpy().astype(np.float64)


def bfr(a):
    return O.bf16_rne(np.asarray(a, F32)).astype(np.float64)


def within_bf16(x, ref, floor=0.0, what="", rel=1e-5):
    """One bf16 rounding (2^-8 relative) on top of fp32 arithmetic (rel)."""
    err = np.abs(x - ref)
    lim = (2.0 ** -8 + rel) * np.abs(ref) + floor + 1e-30
    assert np.all(err <= lim), (what, float(np.max(err / lim)))


@pytest.mark.parametrize("M,N,K,batch,sa,sb", [(64, 64, 32, 5, 1, 1), (200, 264, 128, 3, 1, 0),
                                              (2048 // 4, 512, 128, 8, 1, 1), (256, 256, 96, 4, 1, 1)])
def test_gemm_nt_batched(M, N, K, batch, sa, sb):
    rs = np.random.default_rng(M + N + K + batch)
    A = bfr(rs.standard_normal((batch, M, K)))
    B = bfr(rs.standard_normal((batch, N, K)))
    if sb == 0:
        B[1:] = B[0]
    dA, dB = dev(A, torch.bfloat16), dev(B if sb else B[:1], torch.bfloat16)
    out = torch.empty(batch, M, N, device="cuda")
    uq.uniquan_gemm_nt_batched(M, N, K, batch, dA, M * K, dB, N * K * sb, out, M * N, 0.5)
    single = torch.empty(M, N, device="cuda")
    torch.cuda.synchronize()
    got = host(out)
    for b in range(batch):
        ref = 0.5 * A[b] @ B[b].T
        mag = 0.5 * np.abs(A[b]) @ np.abs(B[b]).T
        assert np.all(np.abs(got[b] - ref) <= 1e-5 * mag), b
        uq.uniquan_gemm_nt(M, N, K, dA[b], dB[b if sb else 0], single, 0.5)
        torch.cuda.synchronize()
        assert np.array_equal(host(single), got[b]), b   # the batch is the same kernel on each slice


@pytest.mark.parametrize("M,N,K", [(264, 520, 96), (600, 1032, 160), (4104, 3848, 96)])
@pytest.mark.parametrize("a_kslow,b_kslow", [(1, 1), (0, 1), (1, 0), (0, 0)])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_gemm_kslow_operands(M, N, K, a_kslow, b_kslow, out_dtype):
    """uniquan_gemm with operands stored K-slow ([K, M] / [K, N]): ragged
    multi-tile shapes on 256 x 128 tiles (the first two) and 256 x 256 tiles
    (the third, 17 x 16 tiles), against an fp64 product, and bit for bit
    against uniquan_gemm_nt on the K-contiguous copies (the same accumulation
    order over k)."""
    rs = np.random.default_rng(M * 7 + N * 3 + K + 10 * a_kslow + b_kslow)
    A = bfr(rs.standard_normal((M, K)))
    B = bfr(rs.standard_normal((N, K)))
    dA, dB = dev(A, torch.bfloat16), dev(B, torch.bfloat16)
    sA = dev(A.T, torch.bfloat16) if a_kslow else dA
    sB = dev(B.T, torch.bfloat16) if b_kslow else dB
    out = torch.full((M, N), float("nan"), device="cuda", dtype=out_dtype)
    nt = torch.full((M, N), float("nan"), device="cuda", dtype=out_dtype)
    uq.uniquan_gemm(M, N, K, sA, a_kslow, sB, b_kslow, out, 0.5)
    uq.uniquan_gemm_nt(M, N, K, dA, dB, nt, 0.5)
    torch.cuda.synchronize()
    got = host(out)
    assert np.array_equal(got, host(nt))
    ref = 0.5 * A @ B.T
    mag = 0.5 * np.abs(A) @ np.abs(B).T
    if out_dtype == torch.float32:
        assert np.all(np.abs(got - ref) <= 1e-5 * mag)
    else:
        within_bf16(got, ref, floor=1e-5 * mag, what="bf16 out")


@pytest.mark.parametrize("T,H,K,L,group,rotate", [(520, 4, 96, 260, 1, True), (2048, 8, 64, 512, 4, True),
                                                  (2048, 8, 64, 1024, 1, False), (8192, 32, 128, 2048, 1, True)])
def test_gemm_heads_matches_product_then_split(T, H, K, L, group, rotate):
    """The projection with the head split (and rotation) in the product's
    store equals uniquan_gemm_nt (fp32) followed by uniquan_rope_split, bit for
    bit: ragged rows (520 = 2 x 256 + 8), grouped slot order, no rotation, and
    the 7B shape (32 heads, sequences of 2048)."""
    rs = np.random.default_rng(T + H + K + L + group)
    d = 128
    A = dev(bfr(rs.standard_normal((T, K))), torch.bfloat16)
    W = dev(bfr(rs.standard_normal((H * d, K)) * 0.1), torch.bfloat16)
    cs = torch.empty(L, d // 2, 2, device="cuda")
    uq.uniquan_rope_table(L, d, cs)
    fused = torch.full((H, T, d), float("nan"), device="cuda", dtype=torch.bfloat16)
    uq.uniquan_gemm_heads(T, H, K, A, W, L, fused, group=group, rotate=rotate, cs=cs)
    Y = torch.empty(T, H * d, device="cuda")
    uq.uniquan_gemm_nt(T, H * d, K, A, W, Y)
    ref = torch.empty(H, T, d, device="cuda", dtype=torch.bfloat16)
    uq.uniquan_rope_split(T, H, d, L, Y, ref, rotate=rotate, group=group)
    torch.cuda.synchronize()
    assert torch.equal(fused.view(torch.int16), ref.view(torch.int16))
    # the table against the angle's definition (fp64 cos / sin of the fp32 angle within fp32 rounding)
    c = cs.cpu().numpy().astype(np.float64)
    p = np.arange(L, dtype=np.float64)[:, None]
    i = np.arange(d // 2, dtype=np.float64)[None, :]
    ang = p * 10000.0 ** (-2 * i / d)
    assert np.all(np.abs(c[..., 0] - np.cos(ang)) <= 1e-6 * (1 + np.abs(ang)))
    assert np.all(np.abs(c[..., 1] - np.sin(ang)) <= 1e-6 * (1 + np.abs(ang)))


@pytest.mark.parametrize("T,Hk,K,L", [(520, 2, 96, 260), (8192, 8, 128, 2048)])
def test_gemm_heads_leading_rotated(T, Hk, K, L):
    """Keys and values in one stacked product ([W_k; W_v], 2 Hk heads, the
    first Hk rotated): the key heads equal the rotated split of the key
    product and the value heads the plain split of the value product, bit
    for bit (ragged rows; the 7B grouped-query shape, 8 key/value heads)."""
    rs = np.random.default_rng(T + Hk + K + L)
    d = 128
    A = dev(bfr(rs.standard_normal((T, K))), torch.bfloat16)
    Wk = dev(bfr(rs.standard_normal((Hk * d, K)) * 0.1), torch.bfloat16)
    Wv = dev(bfr(rs.standard_normal((Hk * d, K)) * 0.1), torch.bfloat16)
    cs = torch.empty(L, d // 2, 2, device="cuda")
    uq.uniquan_rope_table(L, d, cs)
    Wkv = torch.cat([Wk, Wv]).contiguous()
    fused = torch.full((2 * Hk, T, d), float("nan"), device="cuda", dtype=torch.bfloat16)
    uq.uniquan_gemm_heads(T, 2 * Hk, K, A, Wkv, L, fused, cs=cs, n_rot=Hk)
    refs = []
    for W, rot in ((Wk, True), (Wv, False)):
        Y = torch.empty(T, Hk * d, device="cuda")
        uq.uniquan_gemm_nt(T, Hk * d, K, A, W, Y)
        r = torch.empty(Hk, T, d, device="cuda", dtype=torch.bfloat16)
        uq.uniquan_rope_split(T, Hk, d, L, Y, r, rotate=rot)
        refs.append(r)
    torch.cuda.synchronize()
    bits = lambda t: t.contiguous().view(torch.int16)
    assert torch.equal(bits(fused[:Hk]), bits(refs[0])) and torch.equal(bits(fused[Hk:]), bits(refs[1]))


@pytest.mark.parametrize("T,I,K", [(264, 352, 96), (600, 1056, 64), (8192, 11008, 128)])
def test_gemm_swiglu_matches_products_then_silu(T, I, K):
    """The gate and up products with the SiLU product in one (interleaved
    32-row blocks of W_g and W_u) equal two uniquan_gemm_nt products (bf16)
    followed by uniquan_silu_mul_fwd, bit for bit: ragged rows and columns
    (I = 352 is 2 tiles of 128 + 96), and the 7B width."""
    rs = np.random.default_rng(T + I + K)
    X = dev(bfr(rs.standard_normal((T, K))), torch.bfloat16)
    Wg = dev(bfr(rs.standard_normal((I, K)) * 0.2), torch.bfloat16)
    Wu = dev(bfr(rs.standard_normal((I, K)) * 0.2), torch.bfloat16)
    e = lambda: torch.full((T, I), float("nan"), device="cuda", dtype=torch.bfloat16)
    G, U, H = e(), e(), e()
    uq.uniquan_gemm_swiglu(T, I, K, X, Wg, Wu, G, U, H)
    G0, U0, H0 = e(), e(), e()
    uq.uniquan_gemm_nt(T, I, K, X, Wg, G0)
    uq.uniquan_gemm_nt(T, I, K, X, Wu, U0)
    uq.uniquan_silu_mul_fwd(G0, U0, H0)
    torch.cuda.synchronize()
    bits = lambda t: t.view(torch.int16)
    assert torch.equal(bits(G), bits(G0)) and torch.equal(bits(U), bits(U0)) and torch.equal(bits(H), bits(H0))


@pytest.mark.parametrize("M,N,K", [(264, 360, 96), (600, 1056, 72), (1000, 4096, 512), (8192, 4096, 4096)])
def test_gemm_nt_residual(M, N, K):
    """out = R + A B^T (the output projection with the first residual in its
    store) equals uniquan_gemm_nt (fp32 out) followed by the fp32 sum, bit for
    bit, on every kernel shape (128-, 256 x 128- and 256 x 256-row tiles, K a
    multiple of 32 or not); also in place (out = R)."""
    rs = np.random.default_rng(M + N + K)
    A = dev(bfr(rs.standard_normal((M, K))), torch.bfloat16)
    B = dev(bfr(rs.standard_normal((N, K)) * 0.1), torch.bfloat16)
    R = dev(rs.standard_normal((M, N)) * 3.0, torch.float32)
    P = torch.full((M, N), float("nan"), device="cuda")
    uq.uniquan_gemm_nt(M, N, K, A, B, P)
    out = torch.full((M, N), float("nan"), device="cuda")
    uq.uniquan_gemm_nt_residual(M, N, K, A, B, R, out)
    R2 = R.clone()
    uq.uniquan_gemm_nt_residual(M, N, K, A, B, R2, R2)
    ref = R + P
    torch.cuda.synchronize()
    bits = lambda t: t.view(torch.int32)
    assert torch.equal(bits(out), bits(ref)) and torch.equal(bits(R2), bits(ref))


@pytest.mark.parametrize("stacked", [False, True])
@pytest.mark.parametrize("T,I,K", [(264, 360, 96), (600, 1056, 64), (8192, 11008, 128)])
def test_gemm_silu_bwd_matches_product_then_silu_bwd(T, I, K, stacked):
    """dH = 2 E W_d (W_d stored [K, I]) with the SiLU product's backward in the
    product's store equals uniquan_gemm (bf16 dH) followed by
    uniquan_silu_mul_bwd, bit for bit (ragged shapes, the 7B width); stacked:
    dG and dU side by side in one [T, 2I] array (rows 2I apart)."""
    rs = np.random.default_rng(T * 3 + I + K)
    E = dev(bfr(rs.standard_normal((T, K))), torch.bfloat16)
    Wd = dev(bfr(rs.standard_normal((K, I)) * 0.2), torch.bfloat16)
    G = dev(bfr(rs.standard_normal((T, I)) * 2.0), torch.bfloat16)
    U = dev(bfr(rs.standard_normal((T, I))), torch.bfloat16)
    e = lambda: torch.full((T, I), float("nan"), device="cuda", dtype=torch.bfloat16)
    if stacked:
        dGU = torch.full((T, 2 * I), float("nan"), device="cuda", dtype=torch.bfloat16)
        dG, dU = dGU[:, :I], dGU[:, I:]
        uq.uniquan_gemm_silu_bwd(T, I, K, E, Wd, 2.0, G, U, dG, dU, ld_d=2 * I)
    else:
        dG, dU = e(), e()
        uq.uniquan_gemm_silu_bwd(T, I, K, E, Wd, 2.0, G, U, dG, dU)
    dH0, dG0, dU0 = e(), e(), e()
    uq.uniquan_gemm(T, I, K, E, 0, Wd, 1, dH0, 2.0)
    uq.uniquan_silu_mul_bwd(dH0, G, U, dG0, dU0)
    torch.cuda.synchronize()
    bits = lambda t: t.view(torch.int16)
    assert torch.equal(bits(dG), bits(dG0)) and torch.equal(bits(dU), bits(dU0))


@pytest.mark.parametrize("T,C", [(5, 8), (37, 264), (33, 1024), (9, 2048), (64, 4096)])
def test_add_rmsnorm(T, C):
    rs = np.random.default_rng(T * C)
    X = rs.standard_normal((T, C)).astype(F32)
    A = (0.5 * rs.standard_normal((T, C))).astype(F32)
    g = (1.0 + 0.2 * rs.standard_normal(C)).astype(F32)
    R, Z, r = torch.empty(T, C, device="cuda"), torch.empty(T, C, dtype=torch.bfloat16, device="cuda"), \
        torch.empty(T, device="cuda")
    uq.uniquan_add_rmsnorm(T, C, dev(X, torch.float32), dev(A, torch.float32), dev(g, torch.float32), R, Z, r)
    torch.cuda.synchronize()
    v = (X + A).astype(F32)
    assert np.array_equal(host(R), v.astype(np.float64))
    zref, rref = D.rmsnorm(v.astype(np.float64), g.astype(np.float64))
    assert np.allclose(host(r), rref[:, 0], rtol=1e-5)
    within_bf16(host(Z), zref, 1e-6 * np.abs(zref).max(), "Z")
    Z2, r2 = torch.empty_like(Z), torch.empty_like(r)
    uq.uniquan_add_rmsnorm(T, C, dev(X, torch.float32), None, dev(g, torch.float32), None, Z2, r2)
    torch.cuda.synchronize()
    zref2, _ = D.rmsnorm(X.astype(np.float64), g.astype(np.float64))
    within_bf16(host(Z2), zref2, 1e-6 * np.abs(zref2).max(), "Z without A")


@pytest.mark.parametrize("two", [True, False])
@pytest.mark.parametrize("T,C", [(7, 16), (33, 512), (33, 1024), (9, 2048), (64, 4096)])
def test_rmsnorm_bwd(T, C, two):
    """two: the gradient of Z given as two summed parts (dZa + dZb); else one (dZb NULL)."""
    rs = np.random.default_rng(T + C)
    X = rs.standard_normal((T, C))
    g = 1.0 + 0.2 * rs.standard_normal(C)
    dZa, dZb = rs.standard_normal((T, C)), rs.standard_normal((T, C))
    if not two:
        dZb = np.zeros((T, C))
    E = bfr(rs.standard_normal((T, C)))
    _, rref = D.rmsnorm(X, g)
    r32 = rref[:, 0].astype(F32)
    dR = torch.empty(T, C, dtype=torch.bfloat16, device="cuda")
    dRf = torch.empty(T, C, device="cuda")
    uq.uniquan_rmsnorm_bwd(T, C, dev(dZa, torch.float32), dev(dZb, torch.float32) if two else None,
                           dev(X, torch.float32), dev(g, torch.float32), dev(r32, torch.float32),
                           dev(E, torch.bfloat16), 2.0, dR, dRf)
    torch.cuda.synchronize()
    ref = 2.0 * E + D.rmsnorm_bwd(dZa.astype(F32).astype(np.float64) + dZb.astype(F32).astype(np.float64),
                                  X.astype(F32).astype(np.float64), g.astype(F32).astype(np.float64),
                                  r32.astype(np.float64)[:, None])
    scale = np.max(np.abs(ref), axis=1, keepdims=True)
    assert np.all(np.abs(host(dRf) - ref) <= 1e-5 * scale)
    within_bf16(host(dR), ref, 1e-5 * scale, "dR")


@pytest.mark.parametrize("n_seq,L,H,d", [(2, 5, 3, 8), (2, 64, 4, 128)])
def test_rope_split_merge(n_seq, L, H, d):
    T, C = n_seq * L, H * d
    rs = np.random.default_rng(L * H)
    x = rs.standard_normal((T, C)).astype(F32)
    out = torch.empty(H, T, d, dtype=torch.bfloat16, device="cuda")
    uq.uniquan_rope_split(T, H, d, L, dev(x, torch.float32), out, rotate=True)
    torch.cuda.synchronize()
    ang = D.rope_angles(L, d)
    ref = D.rope(D.split_heads(x.astype(np.float64), n_seq, H), ang)     # [n_seq, H, L, d]
    ref_hm = ref.transpose(1, 0, 2, 3).reshape(H, T, d)
    within_bf16(host(out), ref_hm, 2e-6 * np.abs(ref_hm).max(), "rope split")
    # inverse rotation on fp32 head-major input, merged back to token-major
    y = rs.standard_normal((H, T, d)).astype(F32)
    back = torch.empty(T, C, dtype=torch.bfloat16, device="cuda")
    uq.uniquan_rope_merge(T, H, d, L, dev(y, torch.float32), back, rotate=True)
    torch.cuda.synchronize()
    yin = y.astype(np.float64).reshape(H, n_seq, L, d).transpose(1, 0, 2, 3)
    ref_back = D.merge_heads(D.rope(yin, ang, inverse=True))
    within_bf16(host(back), ref_back, 2e-6 * np.abs(ref_back).max(), "rope merge")
    # no rotation: pure layout moves of bf16 data, bit-exact round trip
    xb = bfr(x)
    hm = torch.empty(H, T, d, dtype=torch.bfloat16, device="cuda")
    tm = torch.empty(T, C, dtype=torch.bfloat16, device="cuda")
    uq.uniquan_rope_split(T, H, d, L, dev(xb, torch.bfloat16), hm, rotate=False)
    uq.uniquan_rope_merge(T, H, d, L, hm, tm, rotate=False)
    torch.cuda.synchronize()
    assert np.array_equal(host(hm), xb.reshape(T, H, d).transpose(1, 0, 2))
    assert np.array_equal(host(tm), xb)


@pytest.mark.parametrize("n_seq,L,H,d,G,nsum", [(3, 43, 5, 128, 1, 1), (2, 40, 6, 16, 3, 2), (1, 9, 2, 512, 2, 2),
                                                 (2, 21, 4, 64, 2, 3)])
def test_rope_vector_path_matches_pair_path(n_seq, L, H, d, G, nsum):
    """The 16-byte chunk kernels (d a multiple of 16, 16-byte aligned buffers)
    against the one-pair kernels, reached through buffers offset by one
    element: bit-identical outputs for every input type and rotation, on
    token counts that leave a partial workgroup."""
    T, C = n_seq * L, H * d
    rs = np.random.default_rng(T + H + d)

    def run(fn, x, n_out, **kw):
        outs = []
        for shift in (0, 1):   # 0: aligned (chunk kernel); 1: offset by one element (pair kernel)
            xin = torch.empty(x.numel() + 8, dtype=x.dtype, device="cuda")
            xin[shift:shift + x.numel()] = x.reshape(-1)
            o = torch.empty(n_out + 8, dtype=torch.bfloat16, device="cuda")
            fn(T, H, d, L, xin[shift:shift + x.numel()], o[shift:shift + n_out], **kw)
            torch.cuda.synchronize()
            outs.append(o[shift:shift + n_out].clone())
        assert torch.equal(outs[0], outs[1]), (fn.__name__, kw)

    x32 = dev(rs.standard_normal((T, C)).astype(F32), torch.float32)
    xb = dev(bfr(rs.standard_normal((T, C))), torch.bfloat16)
    for x in (x32, xb):
        for rot in (True, False):
            run(uq.uniquan_rope_split, x, T * C, rotate=rot, group=G)
    y32 = dev(rs.standard_normal((nsum, H, T, d)).astype(F32), torch.float32)
    yb = dev(bfr(rs.standard_normal((nsum, H, T, d))), torch.bfloat16)
    for y in (y32, yb):
        for rot in (True, False):
            run(uq.uniquan_rope_merge, y, T * C, rotate=rot, group=G, nsum=nsum)


@pytest.mark.parametrize("n_seq,L,H,d,nsum", [(2, 64, 8, 128, 4), (1, 40, 3, 16, 2)])
def test_rope_merge_strided_output(n_seq, L, H, d, nsum):
    """Two merges writing side by side into one [T, 2 H d] array (rows 2 H d
    apart: the key and value gradients of grouped-query attention) equal the
    merges into contiguous [T, H d] arrays, bit for bit, on the chunk kernel
    (16-byte aligned halves) and the pair kernel (d = 16 with H = 3: odd halves)."""
    T, C = n_seq * L, H * d
    rs = np.random.default_rng(T + H + d + nsum)
    yk = dev(rs.standard_normal((nsum, H, T, d)).astype(F32), torch.float32)
    yv = dev(rs.standard_normal((nsum, H, T, d)).astype(F32), torch.float32)
    both = torch.full((T, 2 * C), float("nan"), dtype=torch.bfloat16, device="cuda")
    uq.uniquan_rope_merge(T, H, d, L, yk, both[:, :C], rotate=True, nsum=nsum, ld_out=2 * C)
    uq.uniquan_rope_merge(T, H, d, L, yv, both[:, C:], rotate=False, nsum=nsum, ld_out=2 * C)
    rk = torch.empty(T, C, dtype=torch.bfloat16, device="cuda")
    rv = torch.empty(T, C, dtype=torch.bfloat16, device="cuda")
    uq.uniquan_rope_merge(T, H, d, L, yk, rk, rotate=True, nsum=nsum)
    uq.uniquan_rope_merge(T, H, d, L, yv, rv, rotate=False, nsum=nsum)
    torch.cuda.synchronize()
    bits = lambda t: t.contiguous().view(torch.int16)
    assert torch.equal(bits(both[:, :C]), bits(rk)) and torch.equal(bits(both[:, C:]), bits(rv))


@pytest.mark.parametrize("R,C", [(8, 8), (72, 200), (2048, 136), (136, 4096)])
def test_transpose_2d_edges(R, C):
    """uniquan_transpose_bf16 on shapes with partial 64 x 64 tiles: bit-exact."""
    x = bfr(np.random.default_rng(R + C).standard_normal((R, C)))
    out = torch.empty(C, R, dtype=torch.bfloat16, device="cuda")
    uq.uniquan_transpose_bf16(R, C, dev(x, torch.bfloat16), out)
    torch.cuda.synchronize()
    assert np.array_equal(host(out), x.T)


@pytest.mark.parametrize("B,L", [(3, 7), (4, 130), (2, 2048), (1, 2100)])   # 2100: rows past the register path
def test_softmax_causal(B, L):
    rs = np.random.default_rng(B * L)
    S = (3.0 * rs.standard_normal((B, L, L))).astype(F32)
    P = torch.empty(B, L, L, dtype=torch.bfloat16, device="cuda")
    uq.uniquan_softmax_causal(B * L, L, dev(S, torch.float32), P)
    torch.cuda.synchronize()
    ref = D.causal_softmax(S.astype(np.float64))
    got = host(P)
    assert np.all(got[:, np.triu_indices(L, 1)[0], np.triu_indices(L, 1)[1]] == 0.0)
    within_bf16(got, ref, 1e-6, "P")
    # backward on a probability matrix and upstream gradient generated here
    Pin = bfr(ref)
    dP = rs.standard_normal((B, L, L)).astype(F32)
    dS = torch.empty_like(P)
    uq.uniquan_softmax_causal_bwd(B * L, L, dev(dP, torch.float32), dev(Pin, torch.bfloat16), dS)
    torch.cuda.synchronize()
    mask = np.tril(np.ones((L, L)))
    dpm = dP.astype(np.float64) * mask
    ref_ds = Pin * (dpm - np.sum(Pin * dpm, axis=-1, keepdims=True))
    # the fp32 row dot product errs by ~1e-5 of the row's largest |dP|; dS carries it times P
    scale = np.max(np.abs(dpm), axis=-1, keepdims=True)
    within_bf16(host(dS), ref_ds, 1e-5 * scale * Pin + 1e-7, "dS")


@pytest.mark.parametrize("B,R,C", [(1, 5, 7), (3, 64, 130), (2, 300, 64), (3, 68, 132), (2, 2048, 128)])
def test_transpose_batched(B, R, C):
    x = bfr(np.random.default_rng(R * C).standard_normal((B, R, C)))
    out = torch.empty(B, C, R, dtype=torch.bfloat16, device="cuda")
    uq.uniquan_transpose_bf16_batched(B, R, C, dev(x, torch.bfloat16), out)
    torch.cuda.synchronize()
    assert np.array_equal(host(out), x.transpose(0, 2, 1))


@pytest.mark.parametrize("n", [8, 1000, 3 * 2 ** 20 + 24])
def test_block_loss(n):
    rs = np.random.default_rng(n)
    R, M, Y = (rs.standard_normal(n).astype(F32) for _ in range(3))
    E = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    part = torch.empty(uq.uniquan_block_loss_ws(), device="cuda")
    loss = torch.zeros(1, device="cuda")
    uq.uniquan_block_loss(n, dev(R, torch.float32), dev(M, torch.float32), dev(Y, torch.float32), E, part, loss)
    torch.cuda.synchronize()
    e = ((R + M) - Y).astype(F32)
    assert np.array_equal(host(E), bfr(e))
    ref = float(np.sum(e.astype(np.float64) ** 2))
    assert abs(float(loss.item()) - ref) <= 1e-5 * ref


@pytest.mark.parametrize("T,C,K", [(264, 520, 96), (600, 1032, 160), (8192, 4096, 256)])
def test_gemm_block_loss_matches_product_then_loss(T, C, K):
    """The output product with the block loss in its store: E bit for bit the
    product (fp32) followed by uniquan_block_loss; the loss (partials grouped
    by tile) within 1e-6 of it and within 1e-5 of the fp64 sum of the same
    e^2 (ragged multi-tile shapes, the 7B width)."""
    rs = np.random.default_rng(T + C + K + 5)
    Hh = dev(bfr(rs.standard_normal((T, K))), torch.bfloat16)
    Wd = dev(bfr(rs.standard_normal((C, K)) * 0.1), torch.bfloat16)
    R = dev(rs.standard_normal((T, C)), torch.float32)
    Y = dev(rs.standard_normal((T, C)), torch.float32)
    E = torch.full((T, C), float("nan"), device="cuda", dtype=torch.bfloat16)
    part = torch.empty(uq.uniquan_gemm_block_loss_ws(T, C), device="cuda")
    loss = torch.zeros(1, device="cuda")
    uq.uniquan_gemm_block_loss(T, C, K, Hh, Wd, R, Y, E, part, loss)
    M = torch.empty(T, C, device="cuda")
    uq.uniquan_gemm_nt(T, C, K, Hh, Wd, M)
    E0 = torch.empty(T, C, device="cuda", dtype=torch.bfloat16)
    part0 = torch.empty(uq.uniquan_block_loss_ws(), device="cuda")
    loss0 = torch.zeros(1, device="cuda")
    uq.uniquan_block_loss(T * C, R, M, Y, E0, part0, loss0)
    torch.cuda.synchronize()
    assert torch.equal(E.view(torch.int16), E0.view(torch.int16))
    e = ((R.cpu().numpy() + M.cpu().numpy()) - Y.cpu().numpy()).astype(np.float64)
    ref = float(np.sum(e * e))
    assert abs(float(loss.item()) - float(loss0.item())) <= 1e-6 * ref
    assert abs(float(loss.item()) - ref) <= 1e-5 * ref


@pytest.mark.parametrize("L,N,batch", [(96, 64, 3), (256, 128, 2), (2048, 128, 2)])
def test_gemm_nt_batched_causal(L, N, batch):
    """Causal modes against the full product: mode 1 on j <= i; modes 2 and 3
    (operands zero above / below the diagonal) bit-identical everywhere."""
    rs = np.random.default_rng(L + N)
    full32 = lambda M_, N_, K_, a, b, o, causal: uq.uniquan_gemm_nt_batched(  # noqa: E731
        M_, N_, K_, batch, a, M_ * K_, b, N_ * K_, o, M_ * N_, 1.0, causal)
    # mode 1: scores, M == N == L, K = 128
    Q = torch.from_numpy(bfr(rs.standard_normal((batch, L, 128))).astype(F32)).to("cuda").to(torch.bfloat16)
    Kt = torch.from_numpy(bfr(rs.standard_normal((batch, L, 128))).astype(F32)).to("cuda").to(torch.bfloat16)
    S0 = torch.zeros(batch, L, L, device="cuda")
    S1 = torch.full((batch, L, L), 7.0, device="cuda")
    full32(L, L, 128, Q, Kt, S0, 0)
    full32(L, L, 128, Q, Kt, S1, 1)
    torch.cuda.synchronize()
    low = np.tril(np.ones((L, L), dtype=bool))
    assert np.array_equal(host(S1)[:, low], host(S0)[:, low])
    # modes 2 and 3: A [L, L] triangular, B [N, L]
    Bm = torch.from_numpy(bfr(rs.standard_normal((batch, N, L))).astype(F32)).to("cuda").to(torch.bfloat16)
    for mode, tri in ((2, np.tril), (3, np.triu)):
        A = torch.from_numpy(tri(bfr(rs.standard_normal((batch, L, L)))).astype(F32)).to("cuda").to(torch.bfloat16)
        O0 = torch.zeros(batch, L, N, device="cuda")
        O1 = torch.full((batch, L, N), 7.0, device="cuda")
        full32(L, N, L, A, Bm, O0, 0)
        full32(L, N, L, A, Bm, O1, mode)
        torch.cuda.synchronize()
        assert np.array_equal(host(O1), host(O0)), mode


def _bf16_dev(rs, shape, tri=None):
    a = bfr(rs.standard_normal(shape))
    if tri is not None:
        a = tri(a)
    return a, torch.from_numpy(a.astype(F32)).to("cuda").to(torch.bfloat16)


def test_gemm_pp_scores_causal_vs_fp64():
    """The attention's score products at the 7B block's sequence length on
    the shapes that select the ping-pong kernel (256 x 256 tiles: L = 2048,
    4 batches): mode 0 against an fp64 product for every batch, mode 1 against
    the same reference on every entry j <= i."""
    L, d, batch = 2048, 128, 4
    rs = np.random.default_rng(2048 + 4)
    Q, dQ = _bf16_dev(rs, (batch, L, d))
    Kk, dK = _bf16_dev(rs, (batch, L, d))
    S0 = torch.zeros(batch, L, L, device="cuda")
    S1 = torch.full((batch, L, L), 7.0, device="cuda")
    uq.uniquan_gemm_nt_batched(L, L, d, batch, dQ, L * d, dK, L * d, S0, L * L, 0.125, 0)
    uq.uniquan_gemm_nt_batched(L, L, d, batch, dQ, L * d, dK, L * d, S1, L * L, 0.125, 1)
    torch.cuda.synchronize()
    g0, g1 = host(S0), host(S1)
    low = np.tril(np.ones((L, L), dtype=bool))
    for b in range(batch):
        ref = 0.125 * Q[b] @ Kk[b].T
        mag = 0.125 * np.abs(Q[b]) @ np.abs(Kk[b]).T
        assert np.all(np.abs(g0[b] - ref) <= 1e-5 * mag), b
        assert np.all(np.abs(g1[b][low] - ref[low]) <= 1e-5 * mag[low]), b


@pytest.mark.parametrize("mode,tri", [(2, np.tril), (3, np.triu)])
def test_gemm_pp_triangular_vs_fp64(mode, tri):
    """P V and its transposed counterpart at L = 2048, d = 128 with 32 batches
    (256 x 128 tiles, 64-deep stages of the ping-pong kernel): modes 0 and 2 / 3
    against an fp64 product for every batch."""
    L, N, batch = 2048, 128, 32
    rs = np.random.default_rng(2048 + mode)
    A, dA = _bf16_dev(rs, (batch, L, L), tri)
    B, dB = _bf16_dev(rs, (batch, N, L))
    O0 = torch.zeros(batch, L, N, device="cuda")
    O1 = torch.full((batch, L, N), 7.0, device="cuda")
    uq.uniquan_gemm_nt_batched(L, N, L, batch, dA, L * L, dB, N * L, O0, L * N, 1.0, 0)
    uq.uniquan_gemm_nt_batched(L, N, L, batch, dA, L * L, dB, N * L, O1, L * N, 1.0, mode)
    torch.cuda.synchronize()
    g0, g1 = host(O0), host(O1)
    for b in range(batch):
        ref = A[b] @ B[b].T
        mag = np.abs(A[b]) @ np.abs(B[b]).T
        assert np.all(np.abs(g0[b] - ref) <= 1e-5 * mag + 1e-30), (mode, b)
        assert np.all(np.abs(g1[b] - ref) <= 1e-5 * mag + 1e-30), (mode, b)


@pytest.mark.parametrize("n_seq,L,H,G,nsum", [(2, 8, 4, 2, 2), (2, 64, 8, 4, 4)])
def test_rope_grouped_slots_and_partial_sums(n_seq, L, H, G, nsum):
    """Grouped slot order (head h at (h mod G) (H / G) + h / G) and the merge
    of nsum stacked partials with the inverse rotation."""
    d = 16 if L == 8 else 128
    T, C = n_seq * L, H * d
    rs = np.random.default_rng(H * G)
    slot = [(h % G) * (H // G) + h // G for h in range(H)]
    xb = bfr(rs.standard_normal((T, C)))
    hm = torch.empty(H, T, d, dtype=torch.bfloat16, device="cuda")
    uq.uniquan_rope_split(T, H, d, L, dev(xb, torch.bfloat16), hm, rotate=False, group=G)
    torch.cuda.synchronize()
    got = host(hm)
    for h in range(H):
        assert np.array_equal(got[slot[h]], xb[:, h * d:(h + 1) * d]), h
    # merge: sum of nsum partials, unpermute, inverse rotation
    y = rs.standard_normal((nsum, H, T, d)).astype(F32)
    out = torch.empty(T, C, dtype=torch.bfloat16, device="cuda")
    uq.uniquan_rope_merge(T, H, d, L, dev(y, torch.float32), out, rotate=True, group=G, nsum=nsum)
    torch.cuda.synchronize()
    ysum = y.astype(np.float64).sum(axis=0)                       # [H(slot), T, d]
    yh = np.stack([ysum[slot[h]] for h in range(H)])              # [H(head), T, d]
    yin = yh.reshape(H, n_seq, L, d).transpose(1, 0, 2, 3)
    ref = D.merge_heads(D.rope(yin, D.rope_angles(L, d), inverse=True))
    within_bf16(host(out), ref, 4e-6 * np.abs(ref).max(), "grouped merge")
