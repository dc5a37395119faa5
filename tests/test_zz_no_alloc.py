"""The allocation-free attention backward (orbit_attention_bwd_noalloc)
against orbit_attention_bwd, the entry point whose kernels it shares: two
calls in a row, the second on a smaller input (the library's per-device
scratch array keeps the first call's contents), each bitwise equal to the
workspace entry point and within the bf16 / fp32 bound of the oracle."""
import numpy as np
import pytest

import oracle as O
from helpers import TOL, check, dev, host

pytestmark = pytest.mark.gpu

CODE = {"f32": 0, "bf16": 1}


def _case(lib, dtype, B, H, L, dh, seed):
    import torch

    import synth
    r = np.random.default_rng(seed)
    A = H * dh
    qkv = r.standard_normal((B * L, 3 * A)).astype(np.float32)
    dO = r.standard_normal((B * L, A)).astype(np.float32)
    if dtype == "bf16":
        qkv, dO = synth.bf16_round(qkv), synth.bf16_round(dO)
    t = dev(qkv, dtype)
    e = t.element_size()
    q, k, v = t.data_ptr(), t.data_ptr() + A * e, t.data_ptr() + 2 * A * e
    o = torch.empty(B * L, A, dtype=t.dtype, device="cuda")
    lse = torch.empty(B, H, L, dtype=torch.float32, device="cuda")
    o32 = torch.empty(B * L, A, dtype=torch.float32, device="cuda")
    c = CODE[dtype]
    lib.orbit_attention_fwd(c, B, H, L, dh, q, 3 * A, k, 3 * A, v, 3 * A, o, A, lse, o32, A)
    dOd = dev(dO, dtype)
    # the entry point with a caller workspace
    g_ws = torch.full((B * L, 3 * A), 7.0, dtype=t.dtype, device="cuda")
    ws = torch.empty(lib.orbit_attention_bwd_workspace_bytes(B, H, L, dh), dtype=torch.uint8, device="cuda")
    gw = g_ws.data_ptr()
    lib.orbit_attention_bwd(c, B, H, L, dh, q, 3 * A, k, 3 * A, v, 3 * A, o32, A, 1, lse, dOd, A, gw, gw + A * e,
                            gw + 2 * A * e, 3 * A, ws)
    # the allocation-free entry point
    g_na = torch.full((B * L, 3 * A), -3.0, dtype=t.dtype, device="cuda")
    gn = g_na.data_ptr()
    lib.orbit_attention_bwd_noalloc(c, B, H, L, dh, q, 3 * A, k, 3 * A, v, 3 * A, o32, A, 1, lse, dOd, A, gn,
                                    gn + A * e, gn + 2 * A * e, 3 * A)
    torch.cuda.synchronize()
    assert torch.equal(g_ws, g_na), f"noalloc differs from the workspace entry point (B={B} H={H} L={L} dh={dh})"
    hd = lambda x: x.reshape(B, L, H, dh).transpose(0, 2, 1, 3)
    un = lambda x: x.transpose(0, 2, 1, 3).reshape(B * L, A)
    Q, K_, V_ = hd(qkv[:, :A]), hd(qkv[:, A:2 * A]), hd(qkv[:, 2 * A:])
    _, P = O.attention_fwd(Q, K_, V_)
    dq, dk, dv = O.attention_bwd(hd(dO), Q, K_, V_, P)
    gh = host(g_na)
    tol = TOL[dtype]
    check("noalloc dq", gh[:, :A], un(dq), tol)
    check("noalloc dk", gh[:, A:2 * A], un(dk), tol)
    check("noalloc dv", gh[:, 2 * A:], un(dv), tol)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_two_calls_second_smaller(lib, dtype):
    print(f"noalloc {dtype}: call 1 B=2 H=8 L=700 dh=128; call 2 B=1 H=3 L=130 dh=64", flush=True)
    _case(lib, dtype, 2, 8, 700, 128, 1)
    _case(lib, dtype, 1, 3, 130, 64, 2)


def test_noalloc_rejects_sizes_beyond_its_scratch(lib):
    from paper_2404_14712_amd._lib import ORBIT_E_UNSUPPORTED
    B, H, L, dh = 128, 64, 8192, 128
    assert lib.orbit_attention_bwd_workspace_bytes(B, H, L, dh) > (160 << 20)
    st = lib.lib.orbit_attention_bwd_noalloc(1, B, H, L, dh, 0x1000, H * dh, 0x2000, H * dh, 0x3000, H * dh, 0x4000,
                                             H * dh, 1, 0x5000, 0x6000, H * dh, 0x7000, 0x8000, 0x9000, H * dh, None)
    assert st == ORBIT_E_UNSUPPORTED and "scratch" in lib.last_error()
