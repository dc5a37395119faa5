"""ctypes binding of include/orbit.h: argument marshalling only.

Every function named ``orbit_*`` here calls the C entry point of the same name
with raw device pointers taken from torch tensors and the current HIP stream;
no computation happens in Python. Missing libraries raise immediately — there
is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_float, c_int, c_int32, c_int64, c_size_t, c_void_p
from typing import Dict, Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liborbit.so")

ORBIT_OK, ORBIT_E_ARG, ORBIT_E_UNSUPPORTED, ORBIT_E_DEVICE = 0, 1, 2, 3
ORBIT_F32, ORBIT_BF16 = 0, 1
ABI_VERSION = 2

BLOCK_PARAMS = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "qn_g", "qn_b", "kn_g", "kn_b",
                "w_proj", "b_proj", "ln2_g", "ln2_b", "w_fc1", "b_fc1", "w_fc2", "b_fc2")
AGG_PARAMS = ("q0", "w_q", "b_q", "w_k", "b_k", "w_v", "b_v", "w_o", "b_o", "pos")
HEAD_PARAMS = ("lnf_g", "lnf_b", "w_h", "b_h", "w_hid", "b_hid")


class BlockDesc(ctypes.Structure):
    _fields_ = [("B", c_int32), ("L", c_int32), ("d", c_int32), ("heads", c_int32),
                ("head_dim", c_int32), ("mlp", c_int32), ("qk_norm", c_int32), ("eps", c_float),
                ("dtype", c_int32)]


class BlockParams(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in BLOCK_PARAMS]


class BlockGrads(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in BLOCK_PARAMS]


class EmbedDesc(ctypes.Structure):
    _fields_ = [("B", c_int32), ("V", c_int32), ("H", c_int32), ("W", c_int32), ("patch", c_int32),
                ("d", c_int32), ("dtype", c_int32)]


class AggDesc(ctypes.Structure):
    _fields_ = [("B", c_int32), ("L", c_int32), ("V", c_int32), ("d", c_int32), ("heads", c_int32),
                ("head_dim", c_int32), ("dtype", c_int32)]


class AggParams(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in AGG_PARAMS]


class AggGrads(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in AGG_PARAMS]


class HeadDesc(ctypes.Structure):
    _fields_ = [("B", c_int32), ("L", c_int32), ("d", c_int32), ("out", c_int32), ("final_ln", c_int32),
                ("eps", c_float), ("dtype", c_int32), ("hidden", c_int32)]


class WmseDesc(ctypes.Structure):
    _fields_ = [("B", c_int32), ("H", c_int32), ("W", c_int32), ("V", c_int32), ("patch", c_int32)]


class HeadParams(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in HEAD_PARAMS]


class HeadGrads(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in HEAD_PARAMS]


class OrbitError(RuntimeError):
    def __init__(self, fn: str, status: int, detail: str):
        super().__init__(f"{fn} failed with status {status}: {detail}")
        self.status = status
        self.detail = detail


# C prototypes: name -> (restype, argtypes)
P = c_void_p
_PROTOS = {
    "orbit_vit_block_saved_bytes": (c_size_t, [POINTER(BlockDesc)]),
    "orbit_vit_block_workspace_bytes": (c_size_t, [POINTER(BlockDesc)]),
    "orbit_vit_block_fwd": (c_int, [POINTER(BlockDesc), POINTER(BlockParams), P, P, P, P, c_size_t, P]),
    "orbit_vit_block_bwd": (c_int, [POINTER(BlockDesc), POINTER(BlockParams), P, P, P, P, POINTER(BlockGrads),
                                    c_int, P, c_size_t, P]),
    "orbit_patch_embed": (c_int, [POINTER(EmbedDesc), P, P, P, P, P, P]),
    "orbit_patch_embed_workspace_bytes": (c_size_t, [POINTER(EmbedDesc)]),
    "orbit_patch_embed_bwd": (c_int, [POINTER(EmbedDesc), P, P, P, P, P, c_int, P, c_size_t, P]),
    "orbit_var_aggregate_saved_bytes": (c_size_t, [POINTER(AggDesc)]),
    "orbit_var_aggregate_workspace_bytes": (c_size_t, [POINTER(AggDesc)]),
    "orbit_var_aggregate": (c_int, [POINTER(AggDesc), P, POINTER(AggParams), P, P, P, c_size_t, P]),
    "orbit_var_aggregate_bwd": (c_int, [POINTER(AggDesc), P, POINTER(AggParams), P, P, P, POINTER(AggGrads),
                                        c_int, P, c_size_t, P]),
    "orbit_head_saved_bytes": (c_size_t, [POINTER(HeadDesc)]),
    "orbit_head_workspace_bytes": (c_size_t, [POINTER(HeadDesc)]),
    "orbit_head_fwd": (c_int, [POINTER(HeadDesc), P, POINTER(HeadParams), P, P, P, c_size_t, P]),
    "orbit_head_bwd": (c_int, [POINTER(HeadDesc), P, POINTER(HeadParams), P, P, P, POINTER(HeadGrads), c_int, P,
                               c_size_t, P]),
    "orbit_mse_workspace_bytes": (c_size_t, [c_int64]),
    "orbit_mse_loss": (c_int, [P, P, c_int64, c_float, P, P, P, c_size_t, P]),
    "orbit_wmse_workspace_bytes": (c_size_t, [POINTER(WmseDesc)]),
    "orbit_wmse_loss": (c_int, [POINTER(WmseDesc), P, P, c_float, P, P, P, c_size_t, P]),
    "orbit_gemm_workspace_bytes": (c_size_t, [c_int32] * 6),
    "orbit_gemm": (c_int, [c_int32, c_int32, c_int32, c_int32, P, c_int64, c_int32, P, c_int64, c_int32, P,
                           c_int64, c_int32, c_float, P, c_int32, P, c_size_t, P]),
    "orbit_attention_fwd": (c_int, [c_int32] * 5 + [P, c_int64, P, c_int64, P, c_int64, P, c_int64, P, P, c_int64,
                                                    P]),
    "orbit_attention_bwd_workspace_bytes": (c_size_t, [c_int32] * 4),
    "orbit_attention_bwd": (c_int, [c_int32] * 5 + [P, c_int64, P, c_int64, P, c_int64, P, c_int64, c_int32, P, P,
                                                    c_int64, P, P, P, c_int64, P, c_size_t, P]),
    "orbit_attention_bwd_noalloc": (c_int, [c_int32] * 5 + [P, c_int64, P, c_int64, P, c_int64, P, c_int64, c_int32,
                                                            P, P, c_int64, P, P, P, c_int64, P]),
    "orbit_layernorm_fwd": (c_int, [c_int32, c_int32, c_int32, P, P, P, c_float, P, P, P, P]),
    "orbit_status_string": (c_char_p, [c_int]),
    "orbit_last_error": (c_char_p, []),
    "orbit_abi_version": (c_int, []),
    "orbit_timing_enable": (c_int, [c_int]),
    "orbit_timing_filter": (c_int, [c_char_p]),
    "orbit_timing_summary": (c_int, [c_char_p, POINTER(c_int64), POINTER(c_double), POINTER(c_double),
                                     POINTER(c_double)]),
    "orbit_timing_kernel_name": (c_char_p, [c_int]),
    "orbit_mfma_probe": (c_int, [c_int32, c_int32, ctypes.c_uint32, c_float, P, P]),
}

EXPORTS = tuple(_PROTOS)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


class OrbitLib:
    """The loaded library. Methods mirror the C entry points."""

    def __init__(self, path: str = LIB_PATH):
        if not os.path.exists(path):
            raise RuntimeError(f"HIP library {path} is missing: build it with "
                               "`python -m paper_2404_14712_amd.build` (no CPU fallback exists)")
        self.path = path
        self.lib = ctypes.CDLL(path)
        for name, (res, args) in _PROTOS.items():
            f = getattr(self.lib, name)
            f.restype = res
            f.argtypes = args
        v = self.lib.orbit_abi_version()
        if v != ABI_VERSION:
            raise RuntimeError(f"{path}: ABI version {v}, expected {ABI_VERSION}")

    # -- helpers --------------------------------------------------------
    def _check(self, fn: str, st: int):
        if st != ORBIT_OK:
            raise OrbitError(fn, st, self.lib.orbit_last_error().decode())

    @staticmethod
    def _struct(cls, tensors: Dict[str, object]):
        s = cls()
        for n, _ in cls._fields_:
            setattr(s, n, _ptr(tensors.get(n)))
        return s

    def last_error(self) -> str:
        return self.lib.orbit_last_error().decode()

    # -- block ---------------------------------------------------------------
    def orbit_vit_block_saved_bytes(self, desc: BlockDesc) -> int:
        return self.lib.orbit_vit_block_saved_bytes(ctypes.byref(desc))

    def orbit_vit_block_workspace_bytes(self, desc: BlockDesc) -> int:
        return self.lib.orbit_vit_block_workspace_bytes(ctypes.byref(desc))

    def orbit_vit_block_fwd(self, desc, params, x, y, saved, ws, stream=None):
        p = self._struct(BlockParams, params)
        self._check("orbit_vit_block_fwd", self.lib.orbit_vit_block_fwd(
            ctypes.byref(desc), ctypes.byref(p), _ptr(x), _ptr(y), _ptr(saved), _ptr(ws),
            ws.numel() * ws.element_size(), _stream(stream)))

    def orbit_vit_block_bwd(self, desc, params, x, saved, dy, dx, grads, accumulate, ws, stream=None):
        p = self._struct(BlockParams, params)
        g = self._struct(BlockGrads, grads)
        self._check("orbit_vit_block_bwd", self.lib.orbit_vit_block_bwd(
            ctypes.byref(desc), ctypes.byref(p), _ptr(x), _ptr(saved), _ptr(dy), _ptr(dx), ctypes.byref(g),
            int(accumulate), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))

    # -- patch embedding -------------------------------------------------------
    def orbit_patch_embed(self, desc, img, w_pe, b_pe, ve, tok, stream=None):
        self._check("orbit_patch_embed", self.lib.orbit_patch_embed(
            ctypes.byref(desc), _ptr(img), _ptr(w_pe), _ptr(b_pe), _ptr(ve), _ptr(tok), _stream(stream)))

    def orbit_patch_embed_workspace_bytes(self, desc) -> int:
        return self.lib.orbit_patch_embed_workspace_bytes(ctypes.byref(desc))

    def orbit_patch_embed_bwd(self, desc, img, dtok, dw_pe, db_pe, dve, accumulate, ws, stream=None):
        self._check("orbit_patch_embed_bwd", self.lib.orbit_patch_embed_bwd(
            ctypes.byref(desc), _ptr(img), _ptr(dtok), _ptr(dw_pe), _ptr(db_pe), _ptr(dve), int(accumulate),
            _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))

    # -- aggregation -----------------------------------------------------------
    def orbit_var_aggregate_saved_bytes(self, desc) -> int:
        return self.lib.orbit_var_aggregate_saved_bytes(ctypes.byref(desc))

    def orbit_var_aggregate_workspace_bytes(self, desc) -> int:
        return self.lib.orbit_var_aggregate_workspace_bytes(ctypes.byref(desc))

    def orbit_var_aggregate(self, desc, tok, params, z, saved, ws, stream=None):
        p = self._struct(AggParams, params)
        self._check("orbit_var_aggregate", self.lib.orbit_var_aggregate(
            ctypes.byref(desc), _ptr(tok), ctypes.byref(p), _ptr(z), _ptr(saved), _ptr(ws),
            ws.numel() * ws.element_size(), _stream(stream)))

    def orbit_var_aggregate_bwd(self, desc, tok, params, saved, dz, dtok, grads, accumulate, ws, stream=None):
        p = self._struct(AggParams, params)
        g = self._struct(AggGrads, grads)
        self._check("orbit_var_aggregate_bwd", self.lib.orbit_var_aggregate_bwd(
            ctypes.byref(desc), _ptr(tok), ctypes.byref(p), _ptr(saved), _ptr(dz), _ptr(dtok), ctypes.byref(g),
            int(accumulate), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))

    # -- head ------------------------------------------------------------------
    def orbit_head_saved_bytes(self, desc) -> int:
        return self.lib.orbit_head_saved_bytes(ctypes.byref(desc))

    def orbit_head_workspace_bytes(self, desc) -> int:
        return self.lib.orbit_head_workspace_bytes(ctypes.byref(desc))

    def orbit_head_fwd(self, desc, x, params, pred, saved, ws, stream=None):
        p = self._struct(HeadParams, params)
        self._check("orbit_head_fwd", self.lib.orbit_head_fwd(
            ctypes.byref(desc), _ptr(x), ctypes.byref(p), _ptr(pred), _ptr(saved), _ptr(ws),
            ws.numel() * ws.element_size(), _stream(stream)))

    def orbit_head_bwd(self, desc, x, params, saved, dpred, dx, grads, accumulate, ws, stream=None):
        p = self._struct(HeadParams, params)
        g = self._struct(HeadGrads, grads)
        self._check("orbit_head_bwd", self.lib.orbit_head_bwd(
            ctypes.byref(desc), _ptr(x), ctypes.byref(p), _ptr(saved), _ptr(dpred), _ptr(dx), ctypes.byref(g),
            int(accumulate), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))

    # -- loss ------------------------------------------------------------------
    def orbit_mse_workspace_bytes(self, n: int) -> int:
        return self.lib.orbit_mse_workspace_bytes(int(n))

    def orbit_mse_loss(self, pred, tgt, n, scale, loss, dpred, ws, stream=None):
        self._check("orbit_mse_loss", self.lib.orbit_mse_loss(
            _ptr(pred), _ptr(tgt), int(n), float(scale), _ptr(loss), _ptr(dpred), _ptr(ws),
            ws.numel() * ws.element_size(), _stream(stream)))

    def orbit_wmse_workspace_bytes(self, desc) -> int:
        return self.lib.orbit_wmse_workspace_bytes(ctypes.byref(desc))

    def orbit_wmse_loss(self, desc, pred, tgt, scale, loss, dpred, ws, stream=None):
        self._check("orbit_wmse_loss", self.lib.orbit_wmse_loss(
            ctypes.byref(desc), _ptr(pred), _ptr(tgt), float(scale), _ptr(loss), _ptr(dpred), _ptr(ws),
            ws.numel() * ws.element_size(), _stream(stream)))

    # -- building blocks -------------------------------------------------------
    def orbit_gemm_workspace_bytes(self, dtype, M, N, K, a_kmajor, b_kmajor) -> int:
        return self.lib.orbit_gemm_workspace_bytes(dtype, M, N, K, int(a_kmajor), int(b_kmajor))

    def orbit_gemm(self, dtype, M, N, K, A, lda, a_kmajor, B, ldb, b_kmajor, C, ldc, c_f32, alpha=1.0,
                   bias=None, accumulate=0, ws=None, stream=None):
        nb = 0 if ws is None else ws.numel() * ws.element_size()
        self._check("orbit_gemm", self.lib.orbit_gemm(
            dtype, M, N, K, _ptr(A), lda, int(a_kmajor), _ptr(B), ldb, int(b_kmajor), _ptr(C), ldc, int(c_f32),
            float(alpha), _ptr(bias), int(accumulate), _ptr(ws), nb, _stream(stream)))

    def orbit_attention_fwd(self, dtype, B, H, L, dh, q, ldq, k, ldk, v, ldv, o, ldo, lse, o32=None, ldo32=0,
                            stream=None):
        self._check("orbit_attention_fwd", self.lib.orbit_attention_fwd(
            dtype, B, H, L, dh, _ptr(q), ldq, _ptr(k), ldk, _ptr(v), ldv, _ptr(o), ldo, _ptr(lse), _ptr(o32),
            ldo32, _stream(stream)))

    def orbit_attention_bwd_workspace_bytes(self, B, H, L, dh) -> int:
        return self.lib.orbit_attention_bwd_workspace_bytes(B, H, L, dh)

    def orbit_attention_bwd(self, dtype, B, H, L, dh, q, ldq, k, ldk, v, ldv, o, ldo, o_f32, lse, dO, lddo, dq, dk,
                            dv, ldg, ws, stream=None):
        self._check("orbit_attention_bwd", self.lib.orbit_attention_bwd(
            dtype, B, H, L, dh, _ptr(q), ldq, _ptr(k), ldk, _ptr(v), ldv, _ptr(o), ldo, int(o_f32), _ptr(lse),
            _ptr(dO), lddo, _ptr(dq), _ptr(dk), _ptr(dv), ldg, _ptr(ws), ws.numel() * ws.element_size(),
            _stream(stream)))

    def orbit_attention_bwd_noalloc(self, dtype, B, H, L, dh, q, ldq, k, ldk, v, ldv, o, ldo, o_f32, lse, dO, lddo,
                                    dq, dk, dv, ldg, stream=None):
        self._check("orbit_attention_bwd_noalloc", self.lib.orbit_attention_bwd_noalloc(
            dtype, B, H, L, dh, _ptr(q), ldq, _ptr(k), ldk, _ptr(v), ldv, _ptr(o), ldo, int(o_f32), _ptr(lse),
            _ptr(dO), lddo, _ptr(dq), _ptr(dk), _ptr(dv), ldg, _stream(stream)))

    def orbit_layernorm_fwd(self, dtype, rows, n, x, g, b, eps, y, mean, rstd, stream=None):
        self._check("orbit_layernorm_fwd", self.lib.orbit_layernorm_fwd(
            dtype, rows, n, _ptr(x), _ptr(g), _ptr(b), float(eps), _ptr(y), _ptr(mean), _ptr(rstd),
            _stream(stream)))

    # -- measurement aid -------------------------------------------------------
    def orbit_mfma_probe(self, blocks, iters, seed, x, out, stream=None):
        self._check("orbit_mfma_probe", self.lib.orbit_mfma_probe(int(blocks), int(iters), int(seed), float(x),
                                                                  _ptr(out), _stream(stream)))

    # -- timing ----------------------------------------------------------------
    def orbit_timing_enable(self, on: bool):
        self._check("orbit_timing_enable", self.lib.orbit_timing_enable(1 if on else 0))

    def orbit_timing_filter(self, prefix: Optional[str]):
        self._check("orbit_timing_filter", self.lib.orbit_timing_filter(prefix.encode() if prefix else None))

    def orbit_timing_summary(self, prefix: Optional[str] = None):
        n, ms, fl, by = c_int64(), c_double(), c_double(), c_double()
        self._check("orbit_timing_summary", self.lib.orbit_timing_summary(
            prefix.encode() if prefix else None, ctypes.byref(n), ctypes.byref(ms), ctypes.byref(fl),
            ctypes.byref(by)))
        return {"launches": n.value, "ms": ms.value, "flops": fl.value, "bytes": by.value}

    def orbit_timing_kernel_names(self):
        out, i = [], 0
        while True:
            s = self.lib.orbit_timing_kernel_name(i)
            if s is None:
                return out
            out.append(s.decode())
            i += 1
