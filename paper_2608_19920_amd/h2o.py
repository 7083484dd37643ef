"""ctypes binding of libh2o.so (the C ABI in include/h2o.h).

Argument marshalling only: shapes and dtypes are read off torch tensors,
pointers and the current HIP stream are passed through, and a non-OK status
raises ``H2OError``. Every step of the computation runs in the library's HIP
kernels; there is no fallback. If the library is not built, the first call
raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libh2o.so")

H2O_OK, H2O_EINVAL, H2O_ESHAPE, H2O_EDTYPE, H2O_EALIGN, H2O_EWORKSPACE, \
    H2O_ENODEVICE, H2O_ELAUNCH = range(8)
H2O_F32, H2O_BF16 = 0, 1
STATUS_NAMES = ["H2O_OK", "H2O_EINVAL", "H2O_ESHAPE", "H2O_EDTYPE", "H2O_EALIGN",
                "H2O_EWORKSPACE", "H2O_ENODEVICE", "H2O_ELAUNCH"]
EXPORTED = ["h2o_workspace_bytes", "h2o_sdpa_chunk", "h2o_accumulate_scores",
            "h2o_evict_insert", "h2o_evict_workspace_bytes", "h2o_evict_insert_policy",
            "h2o_chunk_step", "h2o_chunk_step_attend", "h2o_chunk_step_evict",
            "h2o_noalloc_scratch_bytes", "h2o_chunk_step_noalloc",
            "h2o_cache_workspace_bytes", "h2o_sdpa_cache", "h2o_backward_workspace_bytes",
            "h2o_sdpa_chunk_backward", "h2o_kv_gather", "h2o_kv_scatter",
            "h2o_chunk_step_insert_first", "h2o_bottomk", "h2o_last_error", "h2o_debug_force_path",
            "h2o_debug_timing", "h2o_debug_kernel_time", "h2o_version"]
KERNEL_IDS = {"generic_lse": 0, "generic_main": 1, "mfma_lse": 2, "mfma_main": 3,
              "split_reduce": 4, "colsum_reduce": 5, "accumulate": 6, "bottomk": 7,
              "insert": 8, "decode_split": 9, "decode_combine": 10,
              "argmin_insert": 11, "decode_finish": 12, "variant_keys": 13,
              "bwd_dq": 14, "bwd_dkdv": 15, "kv_copy": 16, "bwd_dot": 17,
              "bwd_dq_reduce": 18, "bottomk_insert": 19}
# eviction rankings (Sec. "Variants of Heavy-Hitter Oracle"), as h2o_policy
POLICIES = {"h2o": 0, "h2o_norm": 1, "h2o_orig": 2}


class H2OError(RuntimeError):
    def __init__(self, status: int, msg: str):
        self.status = status
        name = STATUS_NAMES[status] if 0 <= status < len(STATUS_NAMES) else str(status)
        super().__init__(f"{name}: {msg}")


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library with argument types set (loads on first use)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built: run `python -m "
                           "paper_2608_19920_amd.build` (no fallback exists)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i, f, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    L.h2o_workspace_bytes.argtypes = [i] * 7
    L.h2o_workspace_bytes.restype = sz
    L.h2o_sdpa_chunk.argtypes = [vp] * 9 + [sz] + [i] * 6 + [f, i, vp]
    L.h2o_sdpa_chunk.restype = i
    L.h2o_accumulate_scores.argtypes = [vp, vp, i, i, i, i, vp]
    L.h2o_accumulate_scores.restype = i
    L.h2o_evict_insert.argtypes = [vp] * 8 + [i] * 6 + [ctypes.c_int32, i, vp]
    L.h2o_evict_insert.restype = i
    L.h2o_evict_workspace_bytes.argtypes = [i] * 5
    L.h2o_evict_workspace_bytes.restype = sz
    L.h2o_evict_insert_policy.argtypes = [vp] * 8 + [i] * 6 + [ctypes.c_int32, i, i, vp, sz,
                                                               vp]
    L.h2o_evict_insert_policy.restype = i
    L.h2o_chunk_step.argtypes = [vp] * 12 + [sz] + [i] * 6 + [f, ctypes.c_int32, i, vp]
    L.h2o_chunk_step.restype = i
    for name in ("h2o_chunk_step_attend", "h2o_chunk_step_evict"):
        getattr(L, name).argtypes = L.h2o_chunk_step.argtypes
        getattr(L, name).restype = i
    L.h2o_noalloc_scratch_bytes.argtypes = []
    L.h2o_noalloc_scratch_bytes.restype = sz
    L.h2o_chunk_step_noalloc.argtypes = [vp] * 11 + [i] * 6 + [f, ctypes.c_int32, i, vp]
    L.h2o_chunk_step_noalloc.restype = i
    L.h2o_cache_workspace_bytes.argtypes = [i] * 8
    L.h2o_cache_workspace_bytes.restype = sz
    L.h2o_sdpa_cache.argtypes = [vp] * 8 + [sz] + [i] * 6 + [f, ctypes.c_int32, i, vp]
    L.h2o_sdpa_cache.restype = i
    L.h2o_chunk_step_insert_first.argtypes = [vp] * 12 + [sz] + [i] * 6 + \
        [f, ctypes.c_int32, i, i, vp]
    L.h2o_chunk_step_insert_first.restype = i
    L.h2o_backward_workspace_bytes.argtypes = [i] * 7
    L.h2o_backward_workspace_bytes.restype = sz
    L.h2o_sdpa_chunk_backward.argtypes = [vp] * 14 + [sz] + [i] * 6 + [f, ctypes.c_int32, i, vp]
    L.h2o_sdpa_chunk_backward.restype = i
    for name in ("h2o_kv_gather", "h2o_kv_scatter"):
        getattr(L, name).argtypes = [vp] * 3 + [i] * 6 + [vp]
        getattr(L, name).restype = i
    L.h2o_bottomk.argtypes = [vp, i, i, i, vp, vp]
    L.h2o_bottomk.restype = i
    L.h2o_last_error.argtypes = []
    L.h2o_last_error.restype = ctypes.c_char_p
    L.h2o_debug_force_path.argtypes = [i]
    L.h2o_debug_force_path.restype = i
    L.h2o_debug_timing.argtypes = [i]
    L.h2o_debug_timing.restype = i
    L.h2o_debug_kernel_time.argtypes = [i, ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_long)]
    L.h2o_debug_kernel_time.restype = i
    L.h2o_version.argtypes = []
    L.h2o_version.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(status: int) -> None:
    if status != H2O_OK:
        raise H2OError(status, lib().h2o_last_error().decode())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return H2O_F32
    if t.dtype == torch.bfloat16:
        return H2O_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _dev(t: Optional[torch.Tensor], name: str):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def h2o_version() -> str:
    return lib().h2o_version().decode()


def h2o_debug_force_path(path: int) -> None:
    _check(lib().h2o_debug_force_path(int(path)))


def h2o_debug_timing(on: bool) -> None:
    _check(lib().h2o_debug_timing(1 if on else 0))


def h2o_debug_kernel_time(kernel) -> tuple:
    """(total milliseconds, launch count) of a kernel since h2o_debug_timing."""
    kid = KERNEL_IDS[kernel] if isinstance(kernel, str) else int(kernel)
    ms, n = ctypes.c_double(0.0), ctypes.c_long(0)
    _check(lib().h2o_debug_kernel_time(kid, ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def h2o_workspace_bytes(B, Hq, Hkv, T, M, d, dtype) -> int:
    code = dtype if isinstance(dtype, int) else _dtype_code(torch.empty(0, dtype=dtype))
    return int(lib().h2o_workspace_bytes(B, Hq, Hkv, T, M, d, code))


def h2o_sdpa_chunk(q, k_cache, v_cache, k_new, v_new, out, lse, wsum, workspace,
                   scale: Optional[float] = None, stream=None) -> None:
    """q [B,Hq,T,d]; caches [B,Hkv,M,d]; new [B,Hkv,T,d]; out like q;
    lse [B,Hq,T] f32; wsum [B,Hkv,M+T] f32; workspace uint8 of
    h2o_workspace_bytes(...) bytes."""
    B, Hq, T, d = q.shape
    Hkv, M = k_cache.shape[1], k_cache.shape[2]
    dt = _dtype_code(q)
    for name, t in (("k_cache", k_cache), ("v_cache", v_cache), ("k_new", k_new),
                    ("v_new", v_new), ("out", out)):
        if t.dtype != q.dtype:
            raise TypeError(f"{name} dtype {t.dtype} != q dtype {q.dtype}")
    if tuple(k_cache.shape) != (B, Hkv, M, d) or tuple(v_cache.shape) != (B, Hkv, M, d):
        raise ValueError("cache shape mismatch")
    if tuple(k_new.shape) != (B, Hkv, T, d) or tuple(v_new.shape) != (B, Hkv, T, d):
        raise ValueError("k_new/v_new shape mismatch")
    if tuple(out.shape) != (B, Hq, T, d):
        raise ValueError("out shape mismatch")
    if tuple(lse.shape) != (B, Hq, T) or lse.dtype != torch.float32:
        raise ValueError("lse must be float32 [B,Hq,T]")
    if tuple(wsum.shape) != (B, Hkv, M + T) or wsum.dtype != torch.float32:
        raise ValueError("wsum must be float32 [B,Hkv,M+T]")
    if scale is None:
        scale = d ** -0.5
    nbytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(lib().h2o_sdpa_chunk(
        _dev(q, "q"), _dev(k_cache, "k_cache"), _dev(v_cache, "v_cache"),
        _dev(k_new, "k_new"), _dev(v_new, "v_new"), _dev(out, "out"), _dev(lse, "lse"),
        _dev(wsum, "wsum"), _dev(workspace, "workspace"), nbytes,
        B, Hq, Hkv, T, M, d, float(scale), dt, _stream(stream)))


def h2o_accumulate_scores(scores, wsum, stream=None) -> None:
    """scores [B,Hkv,M] f32 (in-out) += wsum[..., :M]; wsum [B,Hkv,M+T]."""
    B, Hkv, M = scores.shape
    T = wsum.shape[2] - M
    if scores.dtype != torch.float32 or wsum.dtype != torch.float32:
        raise TypeError("scores and wsum must be float32")
    if tuple(wsum.shape[:2]) != (B, Hkv) or T < 0:
        raise ValueError("wsum shape mismatch")
    _check(lib().h2o_accumulate_scores(_dev(scores, "scores"), _dev(wsum, "wsum"),
                                       B, Hkv, M, T, _stream(stream)))


def _evict_args(k_cache, v_cache, scores, token_pos, k_new, v_new, wsum, evict_idx):
    B, Hkv, M, d = k_cache.shape
    T = k_new.shape[2]
    k = evict_idx.shape[2]
    dt = _dtype_code(k_cache)
    if v_cache.dtype != k_cache.dtype or k_new.dtype != k_cache.dtype or \
            v_new.dtype != k_cache.dtype:
        raise TypeError("cache and chunk tensors must share one dtype")
    if tuple(v_cache.shape) != (B, Hkv, M, d) or tuple(k_new.shape) != (B, Hkv, T, d) or \
            tuple(v_new.shape) != (B, Hkv, T, d):
        raise ValueError("shape mismatch")
    if tuple(scores.shape) != (B, Hkv, M) or scores.dtype != torch.float32:
        raise ValueError("scores must be float32 [B,Hkv,M]")
    if tuple(wsum.shape) != (B, Hkv, M + T) or wsum.dtype != torch.float32:
        raise ValueError("wsum must be float32 [B,Hkv,M+T]")
    if evict_idx.dtype != torch.int32 or tuple(evict_idx.shape[:2]) != (B, Hkv):
        raise ValueError("evict_idx must be int32 [B,Hkv,k]")
    if token_pos is not None and (token_pos.dtype != torch.int32 or
                                  tuple(token_pos.shape) != (B, Hkv, M)):
        raise ValueError("token_pos must be int32 [B,Hkv,M]")
    ptrs = (_dev(k_cache, "k_cache"), _dev(v_cache, "v_cache"), _dev(scores, "scores"),
            _dev(token_pos, "token_pos"), _dev(k_new, "k_new"), _dev(v_new, "v_new"),
            _dev(wsum, "wsum"), _dev(evict_idx, "evict_idx"))
    return ptrs, (B, Hkv, M, T, d, k), dt


def h2o_evict_insert(k_cache, v_cache, scores, token_pos, k_new, v_new, wsum, evict_idx,
                     pos0: int, stream=None) -> None:
    """Bottom-k eviction of the accumulated scores and insert of the chunk."""
    ptrs, sizes, dt = _evict_args(k_cache, v_cache, scores, token_pos, k_new, v_new, wsum,
                                  evict_idx)
    _check(lib().h2o_evict_insert(*ptrs, *sizes, int(pos0), dt, _stream(stream)))


def _policy_code(policy) -> int:
    if isinstance(policy, str):
        if policy not in POLICIES:
            raise ValueError(f"unknown policy {policy!r}")
        return POLICIES[policy]
    return int(policy)


def h2o_evict_workspace_bytes(B, Hkv, M, k, policy) -> int:
    return int(lib().h2o_evict_workspace_bytes(B, Hkv, M, k, _policy_code(policy)))


def h2o_evict_insert_policy(k_cache, v_cache, scores, token_pos, k_new, v_new, wsum,
                            evict_idx, pos0: int, policy, workspace=None, stream=None) -> None:
    """h2o_evict_insert with the ranking of ``policy`` ("h2o", "h2o_norm",
    "h2o_orig"); workspace is a uint8 tensor of h2o_evict_workspace_bytes()."""
    ptrs, sizes, dt = _evict_args(k_cache, v_cache, scores, token_pos, k_new, v_new, wsum,
                                  evict_idx)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().h2o_evict_insert_policy(*ptrs, *sizes, int(pos0), dt, _policy_code(policy),
                                         _dev(workspace, "workspace"), nbytes,
                                         _stream(stream)))


def h2o_chunk_step(q, k_cache, v_cache, scores, token_pos, k_new, v_new, out, lse, wsum,
                   evict_idx, workspace, pos0: int, scale: Optional[float] = None,
                   stream=None, part: str = "all") -> None:
    """h2o_sdpa_chunk + h2o_accumulate_scores + h2o_evict_insert (k = T) in one
    call; shapes as there. ``part`` "attend" / "evict" calls one half
    (h2o_chunk_step_attend / h2o_chunk_step_evict)."""
    fn = {"all": "h2o_chunk_step", "attend": "h2o_chunk_step_attend",
          "evict": "h2o_chunk_step_evict"}[part]
    B, Hq, T, d = q.shape
    Hkv, M = k_cache.shape[1], k_cache.shape[2]
    dt = _dtype_code(q)
    for name, t in (("k_cache", k_cache), ("v_cache", v_cache), ("k_new", k_new),
                    ("v_new", v_new), ("out", out)):
        if t.dtype != q.dtype:
            raise TypeError(f"{name} dtype {t.dtype} != q dtype {q.dtype}")
    if tuple(k_cache.shape) != (B, Hkv, M, d) or tuple(v_cache.shape) != (B, Hkv, M, d) or \
            tuple(k_new.shape) != (B, Hkv, T, d) or tuple(v_new.shape) != (B, Hkv, T, d) or \
            tuple(out.shape) != (B, Hq, T, d):
        raise ValueError("shape mismatch")
    if tuple(lse.shape) != (B, Hq, T) or lse.dtype != torch.float32:
        raise ValueError("lse must be float32 [B,Hq,T]")
    if tuple(wsum.shape) != (B, Hkv, M + T) or wsum.dtype != torch.float32:
        raise ValueError("wsum must be float32 [B,Hkv,M+T]")
    if tuple(scores.shape) != (B, Hkv, M) or scores.dtype != torch.float32:
        raise ValueError("scores must be float32 [B,Hkv,M]")
    if tuple(evict_idx.shape) != (B, Hkv, T) or evict_idx.dtype != torch.int32:
        raise ValueError("evict_idx must be int32 [B,Hkv,T]")
    if token_pos is not None and (token_pos.dtype != torch.int32 or
                                  tuple(token_pos.shape) != (B, Hkv, M)):
        raise ValueError("token_pos must be int32 [B,Hkv,M]")
    if scale is None:
        scale = d ** -0.5
    nbytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(getattr(lib(), fn)(
        _dev(q, "q"), _dev(k_cache, "k_cache"), _dev(v_cache, "v_cache"),
        _dev(scores, "scores"), _dev(token_pos, "token_pos"), _dev(k_new, "k_new"),
        _dev(v_new, "v_new"), _dev(out, "out"), _dev(lse, "lse"), _dev(wsum, "wsum"),
        _dev(evict_idx, "evict_idx"), _dev(workspace, "workspace"), nbytes,
        B, Hq, Hkv, T, M, d, float(scale), int(pos0), dt, _stream(stream)))


def h2o_cache_workspace_bytes(B, Hq, Hkv, T, M, d, dtype, policy="h2o") -> int:
    code = dtype if isinstance(dtype, int) else _dtype_code(torch.empty(0, dtype=dtype))
    return int(lib().h2o_cache_workspace_bytes(B, Hq, Hkv, T, M, d, code,
                                               _policy_code(policy)))


def _cache_args(q, k_cache, v_cache, token_pos, out, lse, wsum):
    B, Hq, T, d = q.shape
    Hkv, M = k_cache.shape[1], k_cache.shape[2]
    for name, t in (("k_cache", k_cache), ("v_cache", v_cache), ("out", out)):
        if t.dtype != q.dtype:
            raise TypeError(f"{name} dtype {t.dtype} != q dtype {q.dtype}")
    if tuple(k_cache.shape) != (B, Hkv, M, d) or tuple(v_cache.shape) != (B, Hkv, M, d) or \
            tuple(out.shape) != (B, Hq, T, d):
        raise ValueError("shape mismatch")
    if token_pos is None or token_pos.dtype != torch.int32 or \
            tuple(token_pos.shape) != (B, Hkv, M):
        raise ValueError("token_pos must be int32 [B,Hkv,M]")
    if tuple(lse.shape) != (B, Hq, T) or lse.dtype != torch.float32:
        raise ValueError("lse must be float32 [B,Hq,T]")
    if tuple(wsum.shape) != (B, Hkv, M) or wsum.dtype != torch.float32:
        raise ValueError("wsum must be float32 [B,Hkv,M]")
    return B, Hq, Hkv, T, M, d


def h2o_sdpa_cache(q, k_cache, v_cache, token_pos, out, lse, wsum, workspace, pos0: int,
                   scale: Optional[float] = None, stream=None) -> None:
    """Attention of the T queries (positions pos0..) over the cache slots,
    masked by token_pos; wsum [B,Hkv,M] f32; workspace uint8 of
    h2o_cache_workspace_bytes(...) bytes."""
    B, Hq, Hkv, T, M, d = _cache_args(q, k_cache, v_cache, token_pos, out, lse, wsum)
    if scale is None:
        scale = d ** -0.5
    nbytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(lib().h2o_sdpa_cache(
        _dev(q, "q"), _dev(k_cache, "k_cache"), _dev(v_cache, "v_cache"),
        _dev(token_pos, "token_pos"), _dev(out, "out"), _dev(lse, "lse"), _dev(wsum, "wsum"),
        _dev(workspace, "workspace"), nbytes, B, Hq, Hkv, T, M, d, float(scale), int(pos0),
        _dtype_code(q), _stream(stream)))


def h2o_noalloc_scratch_bytes() -> int:
    return int(lib().h2o_noalloc_scratch_bytes())


def h2o_chunk_step_noalloc(q, k_cache, v_cache, scores, token_pos, k_new, v_new, out, lse, wsum,
                           evict_idx, pos0: int, scale: Optional[float] = None,
                           stream=None) -> None:
    """h2o_chunk_step without a workspace: the library's own scratch array
    (h2o_noalloc_scratch_bytes) serves instead; shapes as in h2o_chunk_step."""
    B, Hq, T, d = q.shape
    Hkv, M = k_cache.shape[1], k_cache.shape[2]
    if tuple(wsum.shape) != (B, Hkv, M + T) or tuple(evict_idx.shape) != (B, Hkv, T) or \
            tuple(scores.shape) != (B, Hkv, M) or tuple(out.shape) != (B, Hq, T, d) or \
            tuple(k_new.shape) != (B, Hkv, T, d) or tuple(v_new.shape) != (B, Hkv, T, d) or \
            tuple(lse.shape) != (B, Hq, T):
        raise ValueError("shape mismatch")
    if scale is None:
        scale = d ** -0.5
    _check(lib().h2o_chunk_step_noalloc(
        _dev(q, "q"), _dev(k_cache, "k_cache"), _dev(v_cache, "v_cache"),
        _dev(scores, "scores"), _dev(token_pos, "token_pos"), _dev(k_new, "k_new"),
        _dev(v_new, "v_new"), _dev(out, "out"), _dev(lse, "lse"), _dev(wsum, "wsum"),
        _dev(evict_idx, "evict_idx"), B, Hq, Hkv, T, M, d, float(scale), int(pos0),
        _dtype_code(q), _stream(stream)))


def h2o_chunk_step_insert_first(q, k_cache, v_cache, scores, token_pos, k_new, v_new, out, lse,
                                wsum, evict_idx, workspace, pos0: int,
                                scale: Optional[float] = None, policy="h2o",
                                stream=None) -> None:
    """Evict by ``policy`` (scores after pos0 tokens), insert the chunk, attend
    with the token-position mask, accumulate; wsum [B,Hkv,M]."""
    B, Hq, Hkv, T, M, d = _cache_args(q, k_cache, v_cache, token_pos, out, lse, wsum)
    if k_new.dtype != q.dtype or v_new.dtype != q.dtype or \
            tuple(k_new.shape) != (B, Hkv, T, d) or tuple(v_new.shape) != (B, Hkv, T, d):
        raise ValueError("k_new/v_new must be [B,Hkv,T,d] in q's dtype")
    if tuple(scores.shape) != (B, Hkv, M) or scores.dtype != torch.float32:
        raise ValueError("scores must be float32 [B,Hkv,M]")
    if tuple(evict_idx.shape) != (B, Hkv, T) or evict_idx.dtype != torch.int32:
        raise ValueError("evict_idx must be int32 [B,Hkv,T]")
    if scale is None:
        scale = d ** -0.5
    nbytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(lib().h2o_chunk_step_insert_first(
        _dev(q, "q"), _dev(k_cache, "k_cache"), _dev(v_cache, "v_cache"),
        _dev(scores, "scores"), _dev(token_pos, "token_pos"), _dev(k_new, "k_new"),
        _dev(v_new, "v_new"), _dev(out, "out"), _dev(lse, "lse"), _dev(wsum, "wsum"),
        _dev(evict_idx, "evict_idx"), _dev(workspace, "workspace"), nbytes,
        B, Hq, Hkv, T, M, d, float(scale), int(pos0), _dtype_code(q), _policy_code(policy),
        _stream(stream)))


def h2o_backward_workspace_bytes(B, Hq, Hkv, T, M, d, dtype) -> int:
    code = dtype if isinstance(dtype, int) else _dtype_code(torch.empty(0, dtype=dtype))
    return int(lib().h2o_backward_workspace_bytes(B, Hq, Hkv, T, M, d, code))


def h2o_sdpa_chunk_backward(q, k_cache, v_cache, k_new, v_new, lse, dout, dq, dk_cache,
                            dv_cache, dk_new, dv_new, workspace, scale: Optional[float] = None,
                            token_pos=None, pos0: int = 0, stream=None) -> None:
    """Gradients of sum(dout * out) for the chunk attention (token_pos None)
    or the cache attention with the token-position mask (token_pos given;
    k_new, v_new, dk_new, dv_new unused). Gradients in q's dtype."""
    B, Hq, T, d = q.shape
    Hkv, M = k_cache.shape[1], k_cache.shape[2]
    cache = token_pos is not None
    for name, t in (("k_cache", k_cache), ("v_cache", v_cache), ("dout", dout),
                    ("dq", dq), ("dk_cache", dk_cache), ("dv_cache", dv_cache)):
        if t.dtype != q.dtype:
            raise TypeError(f"{name} dtype {t.dtype} != q dtype {q.dtype}")
    for name, t in (("dout", dout), ("dq", dq)):
        if tuple(t.shape) != (B, Hq, T, d):
            raise ValueError(f"{name} must be [B,Hq,T,d]")
    for name, t in (("k_cache", k_cache), ("v_cache", v_cache), ("dk_cache", dk_cache),
                    ("dv_cache", dv_cache)):
        if tuple(t.shape) != (B, Hkv, M, d):
            raise ValueError(f"{name} must be [B,Hkv,M,d]")
    if not cache:
        for name, t in (("k_new", k_new), ("v_new", v_new), ("dk_new", dk_new),
                        ("dv_new", dv_new)):
            if t is None or t.dtype != q.dtype or tuple(t.shape) != (B, Hkv, T, d):
                raise ValueError(f"{name} must be [B,Hkv,T,d] in q's dtype")
    elif token_pos.dtype != torch.int32 or tuple(token_pos.shape) != (B, Hkv, M):
        raise ValueError("token_pos must be int32 [B,Hkv,M]")
    if tuple(lse.shape) != (B, Hq, T) or lse.dtype != torch.float32:
        raise ValueError("lse must be float32 [B,Hq,T]")
    if scale is None:
        scale = d ** -0.5
    nbytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    n = (lambda t, name: None) if cache else _dev
    _check(lib().h2o_sdpa_chunk_backward(
        _dev(q, "q"), _dev(k_cache, "k_cache"), _dev(v_cache, "v_cache"), n(k_new, "k_new"),
        n(v_new, "v_new"), _dev(token_pos, "token_pos"), _dev(lse, "lse"),
        _dev(dout, "dout"), _dev(dq, "dq"), _dev(dk_cache, "dk_cache"),
        _dev(dv_cache, "dv_cache"), n(dk_new, "dk_new"), n(dv_new, "dv_new"),
        _dev(workspace, "workspace"), nbytes, B, Hq, Hkv, T, M, d, float(scale), int(pos0),
        _dtype_code(q), _stream(stream)))


def _kv_rows(cache, idx, rows):
    B, Hkv, M, d = cache.shape
    k = idx.shape[2]
    if idx.dtype != torch.int32 or tuple(idx.shape) != (B, Hkv, k):
        raise ValueError("idx must be int32 [B,Hkv,k]")
    if rows.dtype != cache.dtype or tuple(rows.shape) != (B, Hkv, k, d):
        raise ValueError("rows must be [B,Hkv,k,d] in the cache's dtype")
    return B, Hkv, M, k, d


def h2o_kv_gather(cache, idx, delta, stream=None) -> None:
    """delta[b,h,i] = cache[b,h,idx[b,h,i]]."""
    B, Hkv, M, k, d = _kv_rows(cache, idx, delta)
    _check(lib().h2o_kv_gather(_dev(cache, "cache"), _dev(idx, "idx"), _dev(delta, "delta"),
                               B, Hkv, M, k, d, _dtype_code(cache), _stream(stream)))


def h2o_kv_scatter(cache, idx, src, stream=None) -> None:
    """cache[b,h,idx[b,h,i]] = src[b,h,i]."""
    B, Hkv, M, k, d = _kv_rows(cache, idx, src)
    _check(lib().h2o_kv_scatter(_dev(cache, "cache"), _dev(idx, "idx"), _dev(src, "src"),
                                B, Hkv, M, k, d, _dtype_code(cache), _stream(stream)))


def h2o_bottomk(scores, k: int, idx_out, stream=None) -> None:
    """scores [..., M] f32; idx_out [..., k] int32 (ascending indices)."""
    M = scores.shape[-1]
    rows = scores.numel() // max(M, 1)
    if scores.dtype != torch.float32 or idx_out.dtype != torch.int32:
        raise TypeError("scores must be float32, idx_out int32")
    if idx_out.numel() != rows * k:
        raise ValueError("idx_out size mismatch")
    _check(lib().h2o_bottomk(_dev(scores, "scores"), rows, M, int(k), _dev(idx_out, "idx_out"),
                             _stream(stream)))


# ------------------------------------------------------------ conveniences
def alloc_step(B, Hq, Hkv, T, M, d, dtype, device="cuda", policy="h2o",
               insert_first: bool = False):
    """Output and scratch tensors for one chunk step (``policy``'s eviction
    workspace included); ``insert_first``: for the paper's order
    (h2o_chunk_step_insert_first / h2o_sdpa_cache, wsum of M columns)."""
    code = _dtype_code(torch.empty(0, dtype=dtype))
    if insert_first:
        ws = h2o_cache_workspace_bytes(B, Hq, Hkv, T, M, d, code, policy)
    else:
        ws = h2o_workspace_bytes(B, Hq, Hkv, T, M, d, code)
    ews = h2o_evict_workspace_bytes(B, Hkv, M, T, policy)
    return dict(
        evict_workspace=torch.empty(max(ews, 16), dtype=torch.uint8, device=device),
        out=torch.empty(B, Hq, T, d, dtype=dtype, device=device),
        lse=torch.empty(B, Hq, T, dtype=torch.float32, device=device),
        wsum=torch.empty(B, Hkv, M + (0 if insert_first else T), dtype=torch.float32,
                         device=device),
        workspace=torch.empty(max(ws, 16), dtype=torch.uint8, device=device),
        evict_idx=torch.empty(B, Hkv, T, dtype=torch.int32, device=device),
    )


def step(state, q, k_new, v_new, bufs, pos0: int, scale=None, stream=None,
         fused: bool = True, policy: str = "h2o") -> None:
    """One chunk step in place: attend, accumulate, evict + insert, through
    h2o_chunk_step (``fused``, the h2o ranking) or the three separate calls
    (the eviction ranks by ``policy``).

    ``state`` holds k_cache, v_cache, scores, token_pos (token_pos may be None
    except for h2o_norm).
    """
    if policy != "h2o":
        h2o_sdpa_chunk(q, state["k_cache"], state["v_cache"], k_new, v_new, bufs["out"],
                       bufs["lse"], bufs["wsum"], bufs["workspace"], scale, stream)
        h2o_accumulate_scores(state["scores"], bufs["wsum"], stream)
        h2o_evict_insert_policy(state["k_cache"], state["v_cache"], state["scores"],
                                state.get("token_pos"), k_new, v_new, bufs["wsum"],
                                bufs["evict_idx"], pos0, policy, bufs["evict_workspace"],
                                stream)
        return
    if fused:
        h2o_chunk_step(q, state["k_cache"], state["v_cache"], state["scores"],
                       state.get("token_pos"), k_new, v_new, bufs["out"], bufs["lse"],
                       bufs["wsum"], bufs["evict_idx"], bufs["workspace"], pos0, scale, stream)
        return
    h2o_sdpa_chunk(q, state["k_cache"], state["v_cache"], k_new, v_new, bufs["out"],
                   bufs["lse"], bufs["wsum"], bufs["workspace"], scale, stream)
    h2o_accumulate_scores(state["scores"], bufs["wsum"], stream)
    h2o_evict_insert(state["k_cache"], state["v_cache"], state["scores"], state.get("token_pos"),
                     k_new, v_new, bufs["wsum"], bufs["evict_idx"], pos0, stream)
