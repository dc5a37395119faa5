"""Kernel-level parity of the building blocks (GEMM, attention, LayerNorm)
against the fp64 oracle / plain definitions, through the C ABI."""
import numpy as np
import pytest

import oracle as O
from helpers import TOL, check, dev, host

pytestmark = pytest.mark.gpu

R = np.random.default_rng(4242)
CODE = {"f32": 0, "bf16": 1}


def _mat(shape, dtype, scale=1.0):
    import synth
    a = (R.standard_normal(shape) * scale).astype(np.float32)
    return synth.bf16_round(a) if dtype == "bf16" else a


GEMM_SHAPES = [(37, 40, 24), (200, 136, 72), (130, 264, 520), (1, 48, 64), (300, 16, 1000), (64, 64, 16384),
               (24, 520, 200), (48, 1032, 40), (60, 264, 136),
               (257, 129 * 8, 8),
               # direct-to-LDS kernel: ragged tiles, odd stage counts, split-K
               (300, 520, 256), (520, 1032, 1024), (1000, 264, 4096), (264, 2048, 544),
               (1024, 512, 2048), (2048, 1024, 1024), (776, 392, 1056),
               # short reductions on the two-blocks-per-CU DMA tile
               (300, 200, 64), (520, 264, 32),
               # few columns, long reduction (64x64 tiles)
               (300, 16, 8192)]


LAYOUTS = {"KN": (1, 0), "KK": (1, 1), "MM": (0, 0)}


def _gemm_cases():
    # the ABI requires the contiguous dimension of each operand to be a
    # multiple of 8; other layout/shape pairs are rejected (tests/test_abi.py)
    for shape in GEMM_SHAPES:
        M, N, K = shape
        for layout, (a_k, b_k) in LAYOUTS.items():
            if (not a_k and M % 8) or (b_k and K % 8) or (not b_k and N % 8) or (a_k and K % 8):
                continue
            yield pytest.param(layout, shape, id=f"{layout}-{M}x{N}x{K}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("layout,shape", list(_gemm_cases()))
def test_gemm(lib, dtype, layout, shape):
    import torch
    M, N, K = shape
    a_k, b_k = LAYOUTS[layout]
    A = _mat((M, K), dtype)
    B = _mat((K, N), dtype)
    bias = _mat((N,), dtype)
    Adev = dev(A if a_k else A.T.copy(), dtype)
    Bdev = dev(B.T.copy() if b_k else B, dtype)
    lda = K if a_k else M
    ldb = K if b_k else N
    for c_f32 in ([1] if dtype == "f32" else [0, 1]):
        C = torch.zeros(M, N, dtype=torch.float32 if c_f32 else torch.bfloat16, device="cuda")
        nb = lib.orbit_gemm_workspace_bytes(CODE[dtype], M, N, K, a_k, b_k)
        ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
        lib.orbit_gemm(CODE[dtype], M, N, K, Adev, lda, a_k, Bdev, ldb, b_k, C, N, c_f32, 0.5, dev(bias, dtype),
                       0, ws)
        torch.cuda.synchronize()
        ref = 0.5 * (A.astype(np.float64) @ B.astype(np.float64)) + bias
        tol = TOL[dtype] if dtype == "f32" else 1e-2
        check(f"gemm {layout} {shape} c_f32={c_f32}", host(C), ref, tol)
    # accumulate into float32
    C = torch.ones(M, N, dtype=torch.float32, device="cuda")
    lib.orbit_gemm(CODE[dtype], M, N, K, Adev, lda, a_k, Bdev, ldb, b_k, C, N, 1, 1.0, None, 1, ws)
    torch.cuda.synchronize()
    check(f"gemm acc {layout} {shape}", host(C), 1.0 + A.astype(np.float64) @ B, TOL[dtype] if dtype == "f32"
          else 1e-2)


STRIDED_SHAPES = [(200, 136, 72), (304, 520, 256), (520, 1032, 1024), (1000, 264, 4096), (2048, 1024, 1024)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("layout", list(LAYOUTS))
@pytest.mark.parametrize("shape", STRIDED_SHAPES, ids=[f"{m}x{n}x{k}" for m, n, k in STRIDED_SHAPES])
def test_gemm_strided(lib, dtype, layout, shape):
    """Operands and output as row slices of wider buffers (row strides past
    the contiguous dimension, as the block's q/k/v views of one QKV buffer
    are), the columns past each matrix filled with NaN: a read of them
    would reach the product, a write past N would overwrite them. Covers
    the direct-to-LDS tiles, split K and the register-staged kernel."""
    import torch
    M, N, K = shape
    a_k, b_k = LAYOUTS[layout]
    A = _mat((M, K), dtype)
    B = _mat((K, N), dtype)
    lda = (K if a_k else M) + 24
    ldb = (K if b_k else N) + 40
    ldc = N + 8

    def padded(x, ld):
        full = np.full((x.shape[0], ld), np.nan, np.float32)
        full[:, :x.shape[1]] = x
        return dev(full, dtype)

    Adev = padded(A if a_k else A.T.copy(), lda)
    Bdev = padded(B.T.copy() if b_k else B, ldb)
    for c_f32 in ([1] if dtype == "f32" else [0, 1]):
        C = torch.full((M, ldc), float("nan"), dtype=torch.float32 if c_f32 else torch.bfloat16, device="cuda")
        C[:, :N] = 0
        nb = lib.orbit_gemm_workspace_bytes(CODE[dtype], M, N, K, a_k, b_k)
        ws = torch.empty(max(nb, 256), dtype=torch.uint8, device="cuda")
        lib.orbit_gemm(CODE[dtype], M, N, K, Adev, lda, a_k, Bdev, ldb, b_k, C, ldc, c_f32, 1.0, None, c_f32, ws)
        torch.cuda.synchronize()
        got = host(C)
        assert np.isnan(got[:, N:]).all(), "columns past N were written"
        tol = TOL[dtype] if dtype == "f32" else 1e-2
        check(f"gemm strided {layout} {shape} c_f32={c_f32}", got[:, :N], A.astype(np.float64) @ B, tol)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dh", [32, 64, 128])
@pytest.mark.parametrize("L", [1, 37, 130])
def test_attention(lib, dtype, dh, L):
    _attention_case(lib, dtype, dh, L, 1.0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dh", [64, 128])
def test_attention_wide_logits(lib, dtype, dh):
    """Queries and keys scaled by 2: the logits of every row spread over more
    than 16 log2 units, twice the margin past which the online softmax raises
    its running maximum and rescales the output, so that path runs on later
    key tiles too, not only on the first."""
    _attention_case(lib, dtype, dh, 300, 2.0)


@pytest.mark.parametrize("dh", [192, 256])
@pytest.mark.parametrize("L", [1, 37, 300])
def test_attention_wide_heads(lib, dh, L):
    """The paper's head widths: 192 (1B: 3072 / 16 heads; 113B: 12288 / 64)
    and 256 (10B: 8192 / 32), bf16."""
    _attention_case(lib, "bf16", dh, L, 1.0)


@pytest.mark.parametrize("dtype,dh", [("bf16", 64), ("bf16", 128), ("bf16", 192), ("bf16", 256), ("f32", 64)])
def test_attention_split_backward(lib, dtype, dh):
    """2 samples x 3 heads x 600 positions is a grid of 30 blocks: the bf16
    backward splits its sweeps over two blocks each and merges the float32
    partials; 600 leaves partial key and query tiles in the second split.
    Two runs give bitwise-identical gradients (the merges add in a fixed
    order)."""
    _attention_case(lib, dtype, dh, 600, 1.0, repeat=True)


@pytest.mark.parametrize("dh", [64, 128, 192])
def test_attention_separate_strides(lib, dh):
    """q, k, v, dO and the gradients in separate buffers with five different
    row strides (all multiples of 8), columns past each matrix's heads
    filled with NaN: the tiles copied into LDS take each matrix's own
    stride and read no padding (a NaN there would reach the results); 130
    positions leave a partial last tile. bf16."""
    import torch
    B, H, L = 2, 3, 130
    A = H * dh
    T = B * L
    ld = {"q": A + 8, "k": A + 24, "v": 2 * A, "dO": A + 40, "g": A + 16}
    data = {n: _mat((T, A), "bf16", 1.0) for n in ("q", "k", "v", "dO")}
    buf = {}
    for n, a in data.items():
        full = np.full((T, ld[n]), np.nan, np.float32)
        full[:, :A] = a
        buf[n] = dev(full, "bf16")
    o = torch.zeros(T, A, dtype=torch.bfloat16, device="cuda")
    o32 = torch.zeros(T, A, dtype=torch.float32, device="cuda")
    lse = torch.zeros(B, H, L, dtype=torch.float32, device="cuda")
    lib.orbit_attention_fwd(1, B, H, L, dh, buf["q"], ld["q"], buf["k"], ld["k"], buf["v"], ld["v"], o, A, lse,
                            o32, A)
    grads = {n: torch.full((T, ld["g"]), float("nan"), dtype=torch.bfloat16, device="cuda") for n in ("q", "k", "v")}
    ws = torch.zeros(lib.orbit_attention_bwd_workspace_bytes(B, H, L, dh), dtype=torch.uint8, device="cuda")
    lib.orbit_attention_bwd(1, B, H, L, dh, buf["q"], ld["q"], buf["k"], ld["k"], buf["v"], ld["v"], o32, A, 1, lse,
                            buf["dO"], ld["dO"], grads["q"], grads["k"], grads["v"], ld["g"], ws)
    torch.cuda.synchronize()
    hd = lambda x: x.reshape(B, L, H, dh).transpose(0, 2, 1, 3)
    un = lambda x: x.transpose(0, 2, 1, 3).reshape(T, A)
    Q, K_, V_ = hd(data["q"]), hd(data["k"]), hd(data["v"])
    ref_o, P = O.attention_fwd(Q, K_, V_)
    dq, dk, dv = O.attention_bwd(hd(data["dO"]), Q, K_, V_, P)
    tol = TOL["bf16"]
    check("o", host(o), un(ref_o), tol)
    for n, ref in (("q", dq), ("k", dk), ("v", dv)):
        gh = host(grads[n])
        check("d" + n, gh[:, :A], un(ref), tol)
        assert np.isnan(gh[:, A:]).all(), f"d{n}: columns past the heads were written"


def _attention_case(lib, dtype, dh, L, qk_scale, repeat=False):
    import torch
    B, H = 2, 3
    A = H * dh
    # q, k, v live in one [T, 3A] buffer (as in the block), scaled like QK-normalised rows
    qkv = _mat((B * L, 3 * A), dtype, 1.0)
    if qk_scale != 1.0:
        qkv[:, :2 * A] *= np.float32(qk_scale)   # a power of two: bf16 values stay exact
    dO = _mat((B * L, A), dtype, 1.0)
    t = dev(qkv, dtype)
    e = t.element_size()
    q, k, v = t.data_ptr(), t.data_ptr() + A * e, t.data_ptr() + 2 * A * e
    o = torch.zeros(B * L, A, dtype=t.dtype, device="cuda")
    lse = torch.zeros(B, H, L, dtype=torch.float32, device="cuda")
    o32 = torch.zeros(B * L, A, dtype=torch.float32, device="cuda")
    lib.orbit_attention_fwd(CODE[dtype], B, H, L, dh, q, 3 * A, k, 3 * A, v, 3 * A, o, A, lse, o32, A)
    g = torch.zeros(B * L, 3 * A, dtype=t.dtype, device="cuda")
    ge = g.data_ptr()
    Dws = torch.zeros(lib.orbit_attention_bwd_workspace_bytes(B, H, L, dh), dtype=torch.uint8, device="cuda")
    dOd = dev(dO, dtype)
    lib.orbit_attention_bwd(CODE[dtype], B, H, L, dh, q, 3 * A, k, 3 * A, v, 3 * A, o32, A, 1, lse, dOd, A, ge,
                            ge + A * e, ge + 2 * A * e, 3 * A, Dws)
    torch.cuda.synchronize()
    if repeat:
        # a second run on the same inputs into a fresh buffer: bitwise equal
        g2 = torch.zeros_like(g)
        g2e = g2.data_ptr()
        lib.orbit_attention_bwd(CODE[dtype], B, H, L, dh, q, 3 * A, k, 3 * A, v, 3 * A, o32, A, 1, lse, dOd, A, g2e,
                                g2e + A * e, g2e + 2 * A * e, 3 * A, Dws)
        torch.cuda.synchronize()
        assert torch.equal(g, g2), "attention backward is not bitwise reproducible"
    hd = lambda x: x.reshape(B, L, H, dh).transpose(0, 2, 1, 3)
    Q, K_, V_ = hd(qkv[:, :A]), hd(qkv[:, A:2 * A]), hd(qkv[:, 2 * A:])
    ref_o, P = O.attention_fwd(Q, K_, V_)
    dq, dk, dv = O.attention_bwd(hd(dO), Q, K_, V_, P)
    un = lambda x: x.transpose(0, 2, 1, 3).reshape(B * L, A)
    tol = TOL[dtype]
    check("o", host(o), un(ref_o), tol)
    check("o32", host(o32), un(ref_o), tol)
    S_ = (Q @ np.swapaxes(K_, -1, -2)) / np.sqrt(dh)
    if qk_scale != 1.0:
        assert (S_.max(-1) - S_.min(-1)).min() * np.log2(np.e) > 16, "logits not spread widely enough"
    mx = S_.max(-1, keepdims=True)
    lse_ref = (mx + np.log(np.exp(S_ - mx).sum(-1, keepdims=True)))[..., 0]
    check("lse", host(lse), lse_ref, tol)
    gh = host(g)
    check("dq", gh[:, :A], un(dq), tol)
    check("dk", gh[:, A:2 * A], un(dk), tol)
    check("dv", gh[:, 2 * A:], un(dv), tol)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("rows,n", [(1, 8), (37, 128), (300, 1032), (5, 16384)])
def test_layernorm(lib, dtype, rows, n):
    import torch
    x = _mat((rows, n), dtype, 3.0) + (np.float32(2.0) if dtype == "f32" else 0)
    if dtype == "bf16":
        import synth
        x = synth.bf16_round(x)
    g = _mat((n,), dtype, 0.3) + np.float32(1.0)
    b = _mat((n,), dtype, 0.3)
    if dtype == "bf16":
        import synth
        g = synth.bf16_round(g)
    y = torch.zeros(rows, n, dtype=torch.bfloat16 if dtype == "bf16" else torch.float32, device="cuda")
    mean = torch.zeros(rows, dtype=torch.float32, device="cuda")
    rstd = torch.zeros(rows, dtype=torch.float32, device="cuda")
    lib.orbit_layernorm_fwd(CODE[dtype], rows, n, dev(x, dtype), dev(g, dtype), dev(b, dtype), 1e-5, y, mean, rstd)
    torch.cuda.synchronize()
    ref, (xhat, r) = O.layer_norm_fwd(x, g, b, 1e-5)
    check("ln y", host(y), ref, TOL[dtype])
    check("ln rstd", host(rstd), r[:, 0], 1e-4)
    check("ln mean", host(mean), x.astype(np.float64).mean(-1), 1e-4)


def _probe_pattern(seed, lane, i):
    """The probe's operand pattern, from its definition in include/orbit.h."""
    h = ((seed ^ (8 * lane + i)) * 0x9E3779B1) & 0xFFFFFFFF
    h ^= h >> 15
    h = (h * 0x85EBCA77) & 0xFFFFFFFF
    h ^= h >> 13
    return ((h & 255) - 128) / 64.0


@pytest.mark.gpu
@pytest.mark.parametrize("blocks,iters,seed,x", [(1, 1, 0, 1.0), (256, 64, 0, 1.0), (37, 1000, 0, 0.5),
                                                  (1024, 3, 0, -2.0), (3, 16, 12345, 1.0), (64, 8, 7, 0.25)])
def test_mfma_probe(lib, blocks, iters, seed, x):
    """The matrix-core probe computes what its contract states: per wave,
    8 iters times the summed squares of lanes 0 and 32's operand fragments
    (16 iters x^2 per accumulator element when seed is 0; exact there)."""
    import torch
    out = torch.full((blocks * 4,), float("nan"), dtype=torch.float32, device="cuda")
    lib.orbit_mfma_probe(blocks, iters, seed, x, out)
    torch.cuda.synchronize()
    if seed == 0:
        assert bool((out == 128.0 * x * x * iters).all())
    else:
        sq = sum((x * _probe_pattern(seed, l, i)) ** 2 for l in (0, 32) for i in range(8))
        want = 8.0 * iters * sq
        assert np.allclose(out.cpu().numpy(), want, rtol=1e-6, atol=0), (out[:4], want)
