"""ctypes binding of libsr (include/sr.h): the same names, argument marshalling only.

Tensor arguments are torch tensors on the GPU (their ``data_ptr()`` is passed) or
raw integer device addresses; ``stream=None`` uses torch's current stream.  A
non-OK status raises ``SrError`` carrying ``sr_last_error()``.  If libsr.so has
not been built, ``lib()`` raises ``SrLibraryMissing``: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsr.so")

SR_OK, SR_EINVAL, SR_ESHAPE, SR_EDTYPE, SR_EALIGN, SR_EWORKSPACE, SR_EUNSUPPORTED, SR_EHIP = range(8)
SR_F32, SR_BF16 = 0, 1
SR_BLOCK_PRELN, SR_BLOCK_ADALN = 0, 1
SR_SEL_RANDOM, SR_SEL_TOPK_DIFFNORM = 0, 1

PARAM_FIELDS = ("ln1_w", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o", "ln2_w", "ln2_b",
                "w_fc1", "b_fc1", "w_fc2", "b_fc2", "w_ada", "b_ada")

EXPORTS = ("sr_last_error", "sr_version", "sr_workspace_bytes", "sr_select_scratch_bytes",
           "sr_select_indices", "sr_select_indices_noalloc", "sr_gather", "sr_scatter_delta", "sr_sparse_blocks_fwd",
           "sr_sparse_blocks_bwd", "sr_dense_blocks_fwd", "sr_dense_blocks_bwd", "sr_validate_indices",
           "sr_attention_colsums", "sr_select_topk_scores", "sr_routed_blocks_fwd", "sr_routed_blocks_bwd",
           "sr_cross_attention_fwd", "sr_cross_attention_bwd",
           "sr_edm_workspace_bytes", "sr_edm_blocks_fwd", "sr_edm_blocks_bwd",
           "sr_profile_start", "sr_profile_stop", "sr_probe_mfma_rate")


class SrLibraryMissing(RuntimeError):
    pass


class SrError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"libsr status {status}: {msg}")
        self.status = status


class SrConfig(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("L", ctypes.c_int32), ("D", ctypes.c_int32),
                ("H", ctypes.c_int32), ("F", ctypes.c_int32), ("n_blocks", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("kind", ctypes.c_int32), ("ln_eps", ctypes.c_float),
                ("idx_shared", ctypes.c_int32)]


class SrBlockParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in PARAM_FIELDS]


class SrBlockGrads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in PARAM_FIELDS]


EDM_PARAM_FIELDS = ("w_film", "b_film", "w_qkv", "b_qkv", "w_o", "b_o",
                    "lnc_w", "lnc_b", "w_q", "b_q", "w_kv", "b_kv", "w_oc", "b_oc", "w_g", "b_g",
                    "ln2_w", "ln2_b", "w_fc1", "b_fc1", "w_fc2", "b_fc2")


class SrEdmBlockParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in EDM_PARAM_FIELDS]


class SrEdmBlockGrads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in EDM_PARAM_FIELDS]


_lib = None


def lib(path: str = LIB_PATH):
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise SrLibraryMissing(f"{path} is not built; run `python -m paper_2607_02829_amd.build`")
    L = ctypes.CDLL(path)
    P = ctypes.c_void_p
    I32, U64, SZ = ctypes.c_int32, ctypes.c_uint64, ctypes.c_size_t
    CP = ctypes.POINTER(SrConfig)
    sig = {
        "sr_last_error": ([], ctypes.c_char_p),
        "sr_version": ([], ctypes.c_char_p),
        "sr_workspace_bytes": ([CP, I32, ctypes.POINTER(SZ), ctypes.POINTER(SZ)], I32),
        "sr_select_scratch_bytes": ([CP, I32, ctypes.POINTER(SZ)], I32),
        "sr_select_indices": ([CP, I32, I32, U64, U64, P, P, P, P, SZ, P], I32),
        "sr_select_indices_noalloc": ([CP, I32, I32, U64, U64, P, P, P, P], I32),
        "sr_gather": ([CP, I32, P, P, P, P], I32),
        "sr_scatter_delta": ([CP, I32, P, P, P, P, P], I32),
        "sr_sparse_blocks_fwd": ([CP, I32, P, P, P, P, P, SZ, P, SZ, P], I32),
        "sr_sparse_blocks_bwd": ([CP, I32, P, P, P, SZ, P, P, P, P, P, SZ, P], I32),
        "sr_dense_blocks_fwd": ([CP, P, P, P, P, P, SZ, P, SZ, P], I32),
        "sr_dense_blocks_bwd": ([CP, P, P, P, SZ, P, P, P, P, P, SZ, P], I32),
        "sr_validate_indices": ([CP, I32, P, P, P], I32),
        "sr_attention_colsums": ([CP, I32, P, SZ, I32, P, P], I32),
        "sr_routed_blocks_fwd": ([CP, I32, P, P, P, P, P, SZ, P], I32),
        "sr_cross_attention_fwd": ([CP, I32, I32, P, P, P, P, P], I32),
        "sr_cross_attention_bwd": ([CP, I32, I32, P, P, P, P, P, P, P, P, P], I32),
        "sr_routed_blocks_bwd": ([CP, I32, P, P, P, P, SZ, P, P, P, P, SZ, P], I32),
        "sr_select_topk_scores": ([CP, I32, P, I32, P, P], I32),
        "sr_edm_workspace_bytes": ([CP, I32, ctypes.POINTER(SZ), ctypes.POINTER(SZ)], I32),
        "sr_edm_blocks_fwd": ([CP, I32, P, P, P, P, P, P, SZ, P], I32),
        "sr_edm_blocks_bwd": ([CP, I32, P, P, P, P, SZ, P, P, P, P, P, P, SZ, P], I32),
        "sr_profile_start": ([ctypes.c_char_p], I32),
        "sr_profile_stop": ([ctypes.c_char_p, SZ, ctypes.POINTER(SZ)], I32),
        "sr_probe_mfma_rate": ([P, ctypes.POINTER(ctypes.c_double), P], I32),
    }
    for name, (args, res) in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = res
    _lib = L
    return L


def _p(t):
    """torch tensor -> data_ptr; (address, nbytes) -> address; int -> int; None -> NULL."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if isinstance(t, tuple):
        return t[0]
    return t.data_ptr()


def _nbytes(t):
    """Size in bytes of a buffer argument (0 for NULL or a bare address)."""
    if t is None or isinstance(t, int):
        return 0
    if isinstance(t, tuple):
        return t[1]
    return t.numel() * t.element_size()


def _stream(stream):
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _check(status: int):
    if status != SR_OK:
        raise SrError(status, lib().sr_last_error().decode())


def sr_version() -> str:
    return lib().sr_version().decode()


def sr_last_error() -> str:
    return lib().sr_last_error().decode()


def sr_workspace_bytes(cfg: SrConfig, S: int) -> tuple[int, int]:
    a, b = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib().sr_workspace_bytes(ctypes.byref(cfg), S, ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


def sr_select_scratch_bytes(cfg: SrConfig, select_kind: int) -> int:
    a = ctypes.c_size_t()
    _check(lib().sr_select_scratch_bytes(ctypes.byref(cfg), select_kind, ctypes.byref(a)))
    return a.value


def sr_select_indices(cfg, K, select_kind, seed, step, x_t, x_prev, idx, scratch=None, stream=None):
    _check(lib().sr_select_indices(ctypes.byref(cfg), K, select_kind, seed, step, _p(x_t), _p(x_prev),
                                   _p(idx), _p(scratch), _nbytes(scratch), _stream(stream)))


def sr_select_indices_noalloc(cfg, K, select_kind, seed, step, x_t, x_prev, idx, stream=None):
    _check(lib().sr_select_indices_noalloc(ctypes.byref(cfg), K, select_kind, seed, step, _p(x_t), _p(x_prev),
                                           _p(idx), _stream(stream)))


SR_SELECT_NOALLOC_MAX_TOKENS = 1 << 20


def sr_gather(cfg, K, x, idx, h0, stream=None):
    _check(lib().sr_gather(ctypes.byref(cfg), K, _p(x), _p(idx), _p(h0), _stream(stream)))


def sr_scatter_delta(cfg, K, x, h, h0, idx, stream=None):
    _check(lib().sr_scatter_delta(ctypes.byref(cfg), K, _p(x), _p(h), _p(h0), _p(idx), _stream(stream)))


def sr_sparse_blocks_fwd(cfg, S, params, cond, h_in, h_out, saved, scratch=None, stream=None):
    _check(lib().sr_sparse_blocks_fwd(ctypes.byref(cfg), S, params, _p(cond), _p(h_in), _p(h_out),
                                      _p(saved), _nbytes(saved), _p(scratch), _nbytes(scratch),
                                      _stream(stream)))


def sr_sparse_blocks_bwd(cfg, S, params, cond, saved, dh_out, dh_in, grads, dcond, scratch, stream=None):
    _check(lib().sr_sparse_blocks_bwd(ctypes.byref(cfg), S, params, _p(cond), _p(saved), _nbytes(saved),
                                      _p(dh_out), _p(dh_in), grads, _p(dcond), _p(scratch),
                                      _nbytes(scratch), _stream(stream)))


def sr_dense_blocks_fwd(cfg, params, cond, x_in, x_out, saved, scratch=None, stream=None):
    _check(lib().sr_dense_blocks_fwd(ctypes.byref(cfg), params, _p(cond), _p(x_in), _p(x_out), _p(saved),
                                     _nbytes(saved), _p(scratch), _nbytes(scratch), _stream(stream)))


def sr_dense_blocks_bwd(cfg, params, cond, saved, dx_out, dx_in, grads, dcond, scratch, stream=None):
    _check(lib().sr_dense_blocks_bwd(ctypes.byref(cfg), params, _p(cond), _p(saved), _nbytes(saved),
                                     _p(dx_out), _p(dx_in), grads, _p(dcond), _p(scratch), _nbytes(scratch),
                                     _stream(stream)))


def sr_validate_indices(cfg, K, idx, ok_dev, stream=None):
    _check(lib().sr_validate_indices(ctypes.byref(cfg), K, _p(idx), _p(ok_dev), _stream(stream)))


def sr_routed_blocks_fwd(cfg, K, idx, params, cond, x, saved, stream=None):
    _check(lib().sr_routed_blocks_fwd(ctypes.byref(cfg), K, _p(idx), params, _p(cond), _p(x), _p(saved),
                                      _nbytes(saved), _stream(stream)))


def sr_routed_blocks_bwd(cfg, K, idx, params, cond, saved, g, grads, dcond, scratch, stream=None):
    _check(lib().sr_routed_blocks_bwd(ctypes.byref(cfg), K, _p(idx), params, _p(cond), _p(saved), _nbytes(saved),
                                      _p(g), grads, _p(dcond), _p(scratch), _nbytes(scratch), _stream(stream)))


def sr_cross_attention_fwd(cfg, Sq, Skv, q, kv, O, lse, stream=None):
    _check(lib().sr_cross_attention_fwd(ctypes.byref(cfg), Sq, Skv, _p(q), _p(kv), _p(O), _p(lse), _stream(stream)))


def sr_cross_attention_bwd(cfg, Sq, Skv, q, kv, O, dO, lse, dq, dkv, delta, stream=None):
    _check(lib().sr_cross_attention_bwd(ctypes.byref(cfg), Sq, Skv, _p(q), _p(kv), _p(O), _p(dO), _p(lse), _p(dq),
                                        _p(dkv), _p(delta), _stream(stream)))


def sr_edm_workspace_bytes(cfg: SrConfig, S: int) -> tuple[int, int]:
    a, b = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib().sr_edm_workspace_bytes(ctypes.byref(cfg), S, ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


def sr_edm_blocks_fwd(cfg, S, params, e, zc, h_in, h_out, saved, stream=None):
    _check(lib().sr_edm_blocks_fwd(ctypes.byref(cfg), S, params, _p(e), _p(zc), _p(h_in), _p(h_out), _p(saved),
                                   _nbytes(saved), _stream(stream)))


def sr_edm_blocks_bwd(cfg, S, params, e, zc, saved, dh_out, dh_in, grads, dzc, de, scratch, stream=None):
    _check(lib().sr_edm_blocks_bwd(ctypes.byref(cfg), S, params, _p(e), _p(zc), _p(saved), _nbytes(saved),
                                   _p(dh_out), _p(dh_in), grads, _p(dzc), _p(de), _p(scratch), _nbytes(scratch),
                                   _stream(stream)))


def sr_attention_colsums(cfg, S, saved, block, colsum, stream=None):
    _check(lib().sr_attention_colsums(ctypes.byref(cfg), S, _p(saved), _nbytes(saved), block, _p(colsum),
                                      _stream(stream)))


def sr_select_topk_scores(cfg, K, planes, parts, idx, stream=None):
    _check(lib().sr_select_topk_scores(ctypes.byref(cfg), K, _p(planes), parts, _p(idx), _stream(stream)))


def sr_profile_start(name_filter: str = "") -> None:
    _check(lib().sr_profile_start(name_filter.encode()))


def sr_profile_stop() -> dict[str, dict[str, float]]:
    """Stop recording; returns {name: {launches, ms, flops, bytes}} (totals)."""
    buf = ctypes.create_string_buffer(1 << 20)
    need = ctypes.c_size_t()
    _check(lib().sr_profile_stop(buf, len(buf), ctypes.byref(need)))
    return _parse_profile(buf.value.decode())


def sr_probe_mfma_rate(sink, stream=None) -> float:
    """Sustained dense bf16 MFMA TFLOP/s of the current device (sink: >= 4 bytes of device memory)."""
    out = ctypes.c_double()
    _check(lib().sr_probe_mfma_rate(_p(sink), ctypes.byref(out), _stream(stream)))
    return out.value


def _parse_profile(text: str) -> dict[str, dict[str, float]]:
    out = {}
    for line in text.strip().splitlines():
        name, n, ms, fl, by = line.split()
        out[name] = {"launches": float(n), "ms": float(ms), "flops": float(fl), "bytes": float(by)}
    return out
