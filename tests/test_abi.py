"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every entry point include/orbit.h declares, and rejects bad arguments with
the documented status before enqueuing anything."""
import ctypes
import os
import re

import pytest

from paper_2404_14712_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    return L.OrbitLib()


def _declared():
    src = open(os.path.join(ROOT, "include", "orbit.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(orbit_[a-z0-9_]+)\s*\(", src)))


def test_header_and_binding_agree():
    assert _declared() == sorted(L.EXPORTS)


def test_every_declared_symbol_is_exported(lib):
    for name in _declared():
        assert hasattr(lib.lib, name), name


def test_abi_version_and_strings(lib):
    assert lib.lib.orbit_abi_version() == L.ABI_VERSION == 2
    assert lib.lib.orbit_status_string(0) == b"ok"
    assert lib.lib.orbit_status_string(1) == b"invalid argument"


def _bdesc(**kw):
    v = dict(B=2, L=128, d=128, heads=4, head_dim=32, mlp=512, qk_norm=1, eps=1e-5, dtype=0)
    v.update(kw)
    return L.BlockDesc(*[v[f] for f, _ in L.BlockDesc._fields_])


def test_size_queries_are_deterministic_and_reject_bad_descs(lib):
    d = _bdesc()
    s1 = lib.orbit_vit_block_saved_bytes(d)
    assert s1 > 0 and s1 == lib.orbit_vit_block_saved_bytes(d)
    assert lib.orbit_vit_block_workspace_bytes(d) > 0
    assert lib.orbit_vit_block_saved_bytes(_bdesc(head_dim=48)) == 0
    assert "head_dim" in lib.last_error()
    # the paper's head widths 192 and 256 run in bf16 only
    assert lib.orbit_vit_block_saved_bytes(_bdesc(heads=2, head_dim=192, d=384, dtype=1)) > 0
    assert lib.orbit_vit_block_saved_bytes(_bdesc(heads=2, head_dim=256, d=512, dtype=1)) > 0
    assert lib.orbit_vit_block_saved_bytes(_bdesc(heads=2, head_dim=192, d=384, dtype=0)) == 0
    assert "head_dim 192" in lib.last_error()
    assert lib.orbit_vit_block_saved_bytes(_bdesc(d=100)) == 0
    assert lib.orbit_vit_block_saved_bytes(_bdesc(dtype=7)) == 0
    assert lib.orbit_vit_block_saved_bytes(_bdesc(L=0)) == 0
    # bf16 intermediates are half the size of f32 ones (statistics stay f32)
    assert lib.orbit_vit_block_saved_bytes(_bdesc(dtype=1)) < s1


def _call_block_fwd(lib, desc, x=0x1000, y=0x2000, ws=0x3000, ws_bytes=1 << 40, params=None):
    p = L.BlockParams(*[0x4000 + 0x100 * i for i in range(16)]) if params is None else params
    return lib.lib.orbit_vit_block_fwd(ctypes.byref(desc), ctypes.byref(p), x, y, None, ws, ws_bytes, None)


def test_block_fwd_validation(lib):
    d = _bdesc()
    assert _call_block_fwd(lib, d, x=None) == L.ORBIT_E_ARG and "x is NULL" in lib.last_error()
    assert _call_block_fwd(lib, d, x=0x1001) == L.ORBIT_E_ARG and "aligned" in lib.last_error()
    assert _call_block_fwd(lib, d, y=0x1000) == L.ORBIT_E_ARG and "alias" in lib.last_error()
    assert _call_block_fwd(lib, d, ws_bytes=16) == L.ORBIT_E_ARG and "workspace" in lib.last_error()
    assert _call_block_fwd(lib, _bdesc(head_dim=96)) == L.ORBIT_E_UNSUPPORTED
    # the attention's 32-bit slice offsets: L x 3A bytes must stay well below 2^31
    big = _bdesc(L=1 << 17, heads=16, head_dim=128)
    assert lib.orbit_vit_block_workspace_bytes(big) == 0 and "32-bit" in lib.last_error()
    assert _call_block_fwd(lib, big) == L.ORBIT_E_UNSUPPORTED
    bad = L.BlockParams(*[0x4000 + 0x100 * i for i in range(16)])
    bad.w_fc1 = None
    assert _call_block_fwd(lib, d, params=bad) == L.ORBIT_E_ARG and "w_fc1" in lib.last_error()
    assert lib.lib.orbit_vit_block_fwd(None, None, 0, 0, None, 0, 0, None) == L.ORBIT_E_ARG


def test_other_entry_validation(lib):
    e = L.EmbedDesc(2, 3, 8, 12, 3, 40, 0)  # patch 3 unsupported
    assert lib.lib.orbit_patch_embed(ctypes.byref(e), 0x100, 0x200, 0x300, None, 0x400, None) == \
        L.ORBIT_E_UNSUPPORTED
    e = L.EmbedDesc(2, 3, 10, 12, 4, 40, 0)  # H not a multiple of 4
    assert lib.lib.orbit_patch_embed(ctypes.byref(e), 0x100, 0x200, 0x300, None, 0x400, None) == L.ORBIT_E_ARG
    a = L.AggDesc(1, 4, 5, 64, 4, 16, 1)  # 4 heads in bf16: rows of heads values are not 16 bytes
    assert lib.orbit_var_aggregate_saved_bytes(a) == 0
    a = L.AggDesc(1, 4, 5, 192, 24, 8, 1)  # 24 heads do not divide 64
    assert lib.orbit_var_aggregate_saved_bytes(a) == 0
    a = L.AggDesc(1, 4, 5, 256, 32, 8, 1)
    assert lib.orbit_var_aggregate_saved_bytes(a) > 0
    h = L.HeadDesc(1, 4, 64, 60, 1, 1e-5, 0, 0)  # out not a multiple of 8
    assert lib.orbit_head_saved_bytes(h) == 0
    h = L.HeadDesc(1, 4, 64, 64, 1, 1e-5, 0, 9)  # more than 8 hidden layers
    assert lib.orbit_head_saved_bytes(h) == 0 and "hidden" in lib.last_error()
    # two hidden layers keep their pre-activations and outputs: 4 more [T, d] tensors
    h0 = L.HeadDesc(1, 4, 64, 64, 1, 1e-5, 0, 0)
    h2 = L.HeadDesc(1, 4, 64, 64, 1, 1e-5, 0, 2)
    assert lib.orbit_head_saved_bytes(h2) >= lib.orbit_head_saved_bytes(h0) + 4 * 4 * 64 * 4
    w = L.WmseDesc(2, 128, 256, 48, 4)
    assert lib.orbit_wmse_workspace_bytes(w) >= 2 * 2048 * 4
    assert lib.orbit_wmse_workspace_bytes(L.WmseDesc(2, 130, 256, 48, 4)) == 0 and "multiples" in lib.last_error()
    assert lib.lib.orbit_wmse_loss(ctypes.byref(L.WmseDesc(2, 128, 256, 48, 3)), 0x100, 0x200, 1.0, 0x300, None,
                                   0x400, 1 << 20, None) == L.ORBIT_E_UNSUPPORTED
    assert lib.lib.orbit_mse_loss(0x100, 0x200, 0, 1.0, 0x300, None, 0x400, 1024, None) == L.ORBIT_E_ARG
    assert lib.lib.orbit_gemm(1, 16, 16, 16, 0x100, 16, 0, 0x200, 16, 1, 0x300, 16, 1, 1.0, None, 0, None, 0,
                              None) == L.ORBIT_E_UNSUPPORTED
    # B stored N-major with N = 12: its contiguous dimension is not a multiple of 8
    assert lib.lib.orbit_gemm(1, 16, 12, 16, 0x100, 16, 1, 0x200, 16, 0, 0x300, 16, 1, 1.0, None, 0, None, 0,
                              None) == L.ORBIT_E_ARG and "multiple of 8" in lib.last_error()
    assert lib.lib.orbit_attention_fwd(1, 1, 1, 8, 96, 0x100, 96, 0x200, 96, 0x300, 96, 0x400, 96, 0x500,
                                       None, 0, None) == L.ORBIT_E_UNSUPPORTED
    # the matrix-core probe validates its sizes and output before launching
    assert lib.lib.orbit_mfma_probe(0, 16, 0, 1.0, 0x100, None) == L.ORBIT_E_ARG and "blocks" in lib.last_error()
    assert lib.lib.orbit_mfma_probe(16, (1 << 20) + 1, 0, 1.0, 0x100, None) == L.ORBIT_E_ARG and \
        "iters" in lib.last_error()
    assert lib.lib.orbit_mfma_probe(16, 16, 7, 1.0, None, None) == L.ORBIT_E_ARG and "out" in lib.last_error()


def test_workspace_sizes_cover_the_configs(lib):
    import synth
    for c in synth.CONFIGS.values():
        d = L.BlockDesc(c.B, c.L, c.d, c.heads, c.head_dim, c.mlp, c.qk_norm, c.eps, 1 if c.dtype == "bf16" else 0)
        assert lib.orbit_vit_block_saved_bytes(d) > 0, c.name
        assert lib.orbit_vit_block_workspace_bytes(d) > 0, c.name
        if c.V:
            a = L.AggDesc(c.B, c.L, c.V, c.d, c.agg_heads, c.agg_head_dim, 1 if c.dtype == "bf16" else 0)
            assert lib.orbit_var_aggregate_saved_bytes(a) > 0, (c.name, lib.last_error())
