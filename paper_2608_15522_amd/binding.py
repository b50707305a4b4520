"""ctypes binding of libsa.so: argument marshalling only.

Each function has the name of the C entry point it calls.  Torch tensors
supply device pointers; ``torch.cuda.current_stream()`` supplies the HIP
stream; outputs and the workspace that the caller does not pass are allocated
with ``torch.empty`` (PyTorch is the device-memory allocator here).  All
arithmetic runs in the library's kernels.  There is no fallback: if
``libsa.so`` is missing or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

from .srcid import source_id

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsa.so")

SA_OK, SA_ERR_INVALID_ARG, SA_ERR_UNSUPPORTED, SA_ERR_WORKSPACE, SA_ERR_HIP = range(5)
SA_BF16, SA_F32 = 0, 1
(SA_CALL_CROSS_SCORES, SA_CALL_BUILD_BLOCK_MASK, SA_CALL_SPARSE_ATTENTION,
 SA_CALL_SELECT_PROTECTED, SA_CALL_CACHE_INDICATOR, SA_CALL_TOKEN_ATTENTION,
 SA_CALL_CROSS_ATTENTION) = range(7)

# Every symbol the C header declares, with its ctypes signature.
_VP, _I, _F, _SZ = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
SIGNATURES = {
    "sa_cross_scores": (_I, [_VP, _VP, _VP, _VP, _I, _I, _I, _I, _I, _I, _F, _I,
                             _VP, _VP, _VP, _I, _VP, _SZ, _VP]),
    "sa_select_protected": (_I, [_VP, _I, _I, _I, _VP, _VP, _VP]),
    "sa_build_block_mask": (_I, [_VP, _VP, _I, _I, _I, _I, _I, _F, _I, _I, _VP,
                                 _VP, _VP, _VP, _VP, _VP, _SZ, _VP]),
    "sa_sparse_attention": (_I, [_VP, _VP, _VP, _VP, _VP, _I, _I, _I, _I, _I, _F,
                                 _I, _VP, _VP, _VP, _SZ, _VP]),
    "sa_sparse_attention_noalloc": (_I, [_VP, _VP, _VP, _VP, _VP, _I, _I, _I, _I, _I, _F,
                                         _I, _VP, _VP, _VP]),
    "sa_saliency_ema": (_I, [_VP, _VP, _SZ, _F, _VP]),
    "sa_select_protected_tokens": (_I, [_VP, _I, _I, _I, _VP, _VP, _VP]),
    "sa_protected_token_attention": (_I, [_VP, _VP, _VP, _VP, _VP, _I, _I, _I, _I, _I,
                                          _F, _VP, _I, _VP, _SZ, _VP]),
    "sa_cache_indicator": (_I, [_VP, _VP, _VP, _VP, _VP, _VP, _VP, _I, _I, _I, _I, _I,
                                _F, _F, _F, _F, _VP, _VP, _SZ, _VP]),
    "sa_cross_attention": (_I, [_VP, _VP, _VP, _VP, _VP, _I, _I, _I, _I, _I, _I, _F, _VP,
                                _SZ, _VP]),
    "sa_cross_scores_from_lse": (_I, [_VP, _VP, _VP, _VP, _VP, _VP, _I, _I, _I, _I, _I, _I,
                                      _F, _I, _VP, _VP, _VP, _I, _VP, _SZ, _VP]),
    "sa_pool_columns": (_I, [_I]),
    "sa_cross_scores_pooled": (_I, [_VP, _VP, _VP, _VP, _VP, _VP, _I, _I, _I, _I, _I, _I,
                                    _F, _I, _VP, _VP, _VP, _I, _VP, _VP, _VP, _SZ, _VP]),
    "sa_build_block_mask_pooled": (_I, [_VP, _VP, _I, _I, _I, _I, _F, _I, _I, _VP, _VP, _VP,
                                        _VP, _VP, _VP]),
    "sa_workspace_size": (_SZ, [_I, _I, _I, _I, _I, _I, _I]),
    "sa_last_error": (ctypes.c_char_p, []),
    "sa_version": (_I, []),
    "sa_build_id": (ctypes.c_char_p, []),
}


class SaError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"[sa error {code}] {message}")
        self.code = code


_lib_handle = None


def lib():
    """The loaded library (loaded on first use; raises if it is not built)."""
    global _lib_handle
    if _lib_handle is None:
        if not os.path.exists(LIB_PATH):
            raise SaError(-1, f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2608_15522_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        built = handle.sa_build_id().decode()
        want = source_id()
        if want is not None and built != want:
            raise SaError(-1, f"{LIB_PATH} was built from other sources (build id "
                              f"{built}, sources {want}): rebuild it with "
                              "`python -m paper_2608_15522_amd.build`")
        _lib_handle = handle
    return _lib_handle


def sa_last_error() -> str:
    return lib().sa_last_error().decode()


def sa_version() -> int:
    return lib().sa_version()


def sa_build_id() -> str:
    return lib().sa_build_id().decode()


def _check(rc: int):
    if rc != SA_OK:
        raise SaError(rc, sa_last_error())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return SA_BF16
    if t.dtype == torch.float32:
        return SA_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensors must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return t.data_ptr()


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _expect(t, name, shape, dtype):
    """The library sees only pointers: a tensor of another shape or dtype than
    the call implies would be read or written out of bounds, so refuse it."""
    if t is None:
        return
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.dtype != dtype:
        raise TypeError(f"{name}: dtype {t.dtype}, expected {dtype}")


def _nbytes(ws):
    return ws.numel() * ws.element_size()


def sa_workspace_size(call: int, B: int, H: int, L_v: int, L_a: int, d: int,
                      block: int) -> int:
    return int(lib().sa_workspace_size(call, B, H, L_v, L_a, d, block))


def _workspace(call, B, H, L_v, L_a, d, block, device, ws):
    need = sa_workspace_size(call, B, H, L_v, L_a, d, block)
    if ws is None:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=device)
    return ws


def sa_cross_scores(q_a, k_v, q_v, k_a, scale, block, *, sal_v_tok=None,
                    sal_v_blk=None, sal_a_tok=None, accumulate=False,
                    want_tok=True, ws=None):
    """Token/block saliency; returns (sal_v_tok, sal_v_blk, sal_a_tok)."""
    B, H, L_a, d = q_a.shape
    L_v = k_v.shape[2]
    n_b = -(-L_v // block)
    dev = q_a.device
    _expect(k_v, "k_v", (B, H, L_v, d), q_a.dtype)
    _expect(q_v, "q_v", (B, H, L_v, d), q_a.dtype)
    _expect(k_a, "k_a", (B, H, L_a, d), q_a.dtype)
    _expect(sal_v_tok, "sal_v_tok", (B, L_v), torch.float32)
    _expect(sal_v_blk, "sal_v_blk", (B, n_b), torch.float32)
    _expect(sal_a_tok, "sal_a_tok", (B, L_a), torch.float32)
    if sal_v_blk is None:
        sal_v_blk = torch.empty(B, n_b, dtype=torch.float32, device=dev)
    if sal_v_tok is None and want_tok:
        sal_v_tok = torch.empty(B, L_v, dtype=torch.float32, device=dev)
    if q_v is not None and sal_a_tok is None:
        sal_a_tok = torch.empty(B, L_a, dtype=torch.float32, device=dev)
    ws = _workspace(SA_CALL_CROSS_SCORES, B, H, L_v, L_a, d, block, dev, ws)
    _check(lib().sa_cross_scores(
        _ptr(q_a), _ptr(k_v), _ptr(q_v), _ptr(k_a), B, H, L_v, L_a, d,
        _dtype_code(q_a), float(scale), block, _ptr(sal_v_tok), _ptr(sal_v_blk),
        _ptr(sal_a_tok), int(bool(accumulate)), _ptr(ws), _nbytes(ws), _stream()))
    return sal_v_tok, sal_v_blk, sal_a_tok


def sa_select_protected(sal_blk, k_prot, *, prot_idx=None, prot_flag=None,
                        want_idx=True):
    """Protected blocks; returns (prot_idx [B,k_prot] i32, prot_flag [B,n_b] u8)."""
    B, n_b = sal_blk.shape
    dev = sal_blk.device
    _expect(sal_blk, "sal_blk", (B, n_b), torch.float32)
    _expect(prot_idx, "prot_idx", (B, max(k_prot, 0)), torch.int32)
    _expect(prot_flag, "prot_flag", (B, n_b), torch.uint8)
    if prot_idx is None and want_idx:
        prot_idx = torch.empty(B, max(k_prot, 0), dtype=torch.int32, device=dev)
    if prot_flag is None:
        prot_flag = torch.empty(B, n_b, dtype=torch.uint8, device=dev)
    _check(lib().sa_select_protected(_ptr(sal_blk), B, n_b, int(k_prot),
                                     _ptr(prot_idx) if k_prot > 0 else None,
                                     _ptr(prot_flag), _stream()))
    return prot_idx, prot_flag


def sa_build_block_mask(q_v, k_v, scale, block, k_keep, prot_flag=None, *,
                        kv_idx=None, kv_cnt=None, want_mask=False,
                        want_scores=False, mask=None, scores=None, ws=None):
    """Compacted protected block mask; returns (kv_idx, kv_cnt, mask, scores)."""
    B, H, L_v, d = q_v.shape
    n_b = -(-L_v // block)
    dev = q_v.device
    _expect(k_v, "k_v", (B, H, L_v, d), q_v.dtype)
    _expect(prot_flag, "prot_flag", (B, n_b), torch.uint8)
    _expect(kv_idx, "kv_idx", (B, H, n_b, n_b), torch.int32)
    _expect(kv_cnt, "kv_cnt", (B, H, n_b), torch.int32)
    _expect(mask, "mask", (B, H, n_b, n_b), torch.uint8)
    _expect(scores, "scores", (B, H, n_b, n_b), torch.float32)
    if kv_idx is None:
        kv_idx = torch.empty(B, H, n_b, n_b, dtype=torch.int32, device=dev)
    if kv_cnt is None:
        kv_cnt = torch.empty(B, H, n_b, dtype=torch.int32, device=dev)
    if mask is None and want_mask:
        mask = torch.empty(B, H, n_b, n_b, dtype=torch.uint8, device=dev)
    if scores is None and want_scores:
        scores = torch.empty(B, H, n_b, n_b, dtype=torch.float32, device=dev)
    ws = _workspace(SA_CALL_BUILD_BLOCK_MASK, B, H, L_v, 1, d, block, dev, ws)
    _check(lib().sa_build_block_mask(
        _ptr(q_v), _ptr(k_v), B, H, L_v, d, _dtype_code(q_v), float(scale), block,
        int(k_keep), _ptr(prot_flag), _ptr(kv_idx), _ptr(kv_cnt), _ptr(mask),
        _ptr(scores), _ptr(ws), _nbytes(ws), _stream()))
    return kv_idx, kv_cnt, mask, scores


def sa_sparse_attention(q, k, v, scale, block, kv_idx, kv_cnt, *, o=None,
                        lse=None, want_lse=False, ws=None):
    """Block-sparse attention; returns (o, lse)."""
    B, H, L, d = q.shape
    dev = q.device
    n_b = -(-L // block)
    for name, t in (("k", k), ("v", v), ("o", o)):
        _expect(t, name, (B, H, L, d), q.dtype)
    _expect(lse, "lse", (B, H, L), torch.float32)
    _expect(kv_idx, "kv_idx", (B, H, n_b, n_b), torch.int32)
    _expect(kv_cnt, "kv_cnt", (B, H, n_b), torch.int32)
    if o is None:
        o = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty(B, H, L, dtype=torch.float32, device=dev)
    ws = _workspace(SA_CALL_SPARSE_ATTENTION, B, H, L, 1, d, block, dev, ws)
    _check(lib().sa_sparse_attention(
        _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, H, L, d, _dtype_code(q),
        float(scale), block, _ptr(kv_idx), _ptr(kv_cnt), _ptr(ws), _nbytes(ws),
        _stream()))
    return o, lse


def sa_sparse_attention_noalloc(q, k, v, scale, block, kv_idx, kv_cnt, o, lse=None):
    """Block-sparse attention into the caller's o (and lse), with the
    library's own per-device scratch: nothing is allocated.  Returns (o, lse)."""
    B, H, L, d = q.shape
    n_b = -(-L // block)
    for name, t in (("k", k), ("v", v), ("o", o)):
        _expect(t, name, (B, H, L, d), q.dtype)
    _expect(lse, "lse", (B, H, L), torch.float32)
    _expect(kv_idx, "kv_idx", (B, H, n_b, n_b), torch.int32)
    _expect(kv_cnt, "kv_cnt", (B, H, n_b), torch.int32)
    _check(lib().sa_sparse_attention_noalloc(
        _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, H, L, d, _dtype_code(q),
        float(scale), block, _ptr(kv_idx), _ptr(kv_cnt), _stream()))
    return o, lse


def sa_cross_attention(q, k, v, scale, *, o=None, lse=None, want_lse=False, ws=None):
    """Dense cross-modal attention of q [B,H,Lq,d] over k, v [B,H,Lk,d];
    returns (o, lse) with lse the natural-log row LSE (or None)."""
    B, H, Lq, d = q.shape
    Lk = k.shape[2]
    dev = q.device
    _expect(k, "k", (B, H, Lk, d), q.dtype)
    _expect(v, "v", (B, H, Lk, d), q.dtype)
    _expect(o, "o", (B, H, Lq, d), q.dtype)
    _expect(lse, "lse", (B, H, Lq), torch.float32)
    if o is None:
        o = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty(B, H, Lq, dtype=torch.float32, device=dev)
    ws = _workspace(SA_CALL_CROSS_ATTENTION, B, H, Lq, Lk, d, 0, dev, ws)
    _check(lib().sa_cross_attention(
        _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, H, Lq, Lk, d, _dtype_code(q),
        float(scale), _ptr(ws), _nbytes(ws), _stream()))
    return o, lse


def sa_cross_scores_from_lse(q_a, k_v, q_v, k_a, lse_a, lse_v, scale, block, *,
                             sal_v_tok=None, sal_v_blk=None, sal_a_tok=None,
                             accumulate=False, want_tok=True, ws=None):
    """Saliency from the row LSEs of the two cross-attention forwards;
    returns (sal_v_tok, sal_v_blk, sal_a_tok)."""
    B, H, L_a, d = q_a.shape
    L_v = k_v.shape[2]
    n_b = -(-L_v // block)
    dev = q_a.device
    _expect(k_v, "k_v", (B, H, L_v, d), q_a.dtype)
    _expect(q_v, "q_v", (B, H, L_v, d), q_a.dtype)
    _expect(k_a, "k_a", (B, H, L_a, d), q_a.dtype)
    _expect(lse_a, "lse_a", (B, H, L_a), torch.float32)
    _expect(lse_v, "lse_v", (B, H, L_v), torch.float32)
    _expect(sal_v_tok, "sal_v_tok", (B, L_v), torch.float32)
    _expect(sal_v_blk, "sal_v_blk", (B, n_b), torch.float32)
    _expect(sal_a_tok, "sal_a_tok", (B, L_a), torch.float32)
    if sal_v_blk is None:
        sal_v_blk = torch.empty(B, n_b, dtype=torch.float32, device=dev)
    if sal_v_tok is None and want_tok:
        sal_v_tok = torch.empty(B, L_v, dtype=torch.float32, device=dev)
    if sal_a_tok is None and q_v is not None:
        sal_a_tok = torch.empty(B, L_a, dtype=torch.float32, device=dev)
    ws = _workspace(SA_CALL_CROSS_SCORES, B, H, L_v, L_a, d, block, dev, ws)
    _check(lib().sa_cross_scores_from_lse(
        _ptr(q_a), _ptr(k_v), _ptr(q_v), _ptr(k_a), _ptr(lse_a), _ptr(lse_v), B, H, L_v,
        L_a, d, _dtype_code(q_a), float(scale), block, _ptr(sal_v_tok), _ptr(sal_v_blk),
        _ptr(sal_a_tok), int(bool(accumulate)), _ptr(ws), _nbytes(ws), _stream()))
    return sal_v_tok, sal_v_blk, sal_a_tok


def sa_pool_columns(n_b: int) -> int:
    """Columns n_pad of the pooled block means (0 for an unsupported n_b)."""
    return int(lib().sa_pool_columns(int(n_b)))


def sa_cross_scores_pooled(q_a, k_v, q_v, k_a, scale, block, *, lse_a=None, lse_v=None,
                           sal_v_tok=None, sal_v_blk=None, sal_a_tok=None, qbar=None,
                           kbar=None, accumulate=False, want_tok=True, ws=None):
    """The saliency of both directions (standalone, or from the forwards' row
    LSEs when lse_a and lse_v are given) plus the block means of Q^v and K^v;
    returns (sal_v_tok, sal_v_blk, sal_a_tok, qbar, kbar), the means as
    [B,H,d,n_pad] float64."""
    B, H, L_a, d = q_a.shape
    L_v = k_v.shape[2]
    n_b = -(-L_v // block)
    n_pad = sa_pool_columns(n_b)
    dev = q_a.device
    _expect(k_v, "k_v", (B, H, L_v, d), q_a.dtype)
    _expect(q_v, "q_v", (B, H, L_v, d), q_a.dtype)
    _expect(k_a, "k_a", (B, H, L_a, d), q_a.dtype)
    _expect(lse_a, "lse_a", (B, H, L_a), torch.float32)
    _expect(lse_v, "lse_v", (B, H, L_v), torch.float32)
    _expect(sal_v_tok, "sal_v_tok", (B, L_v), torch.float32)
    _expect(sal_v_blk, "sal_v_blk", (B, n_b), torch.float32)
    _expect(sal_a_tok, "sal_a_tok", (B, L_a), torch.float32)
    _expect(qbar, "qbar", (B, H, d, n_pad), torch.float64)
    _expect(kbar, "kbar", (B, H, d, n_pad), torch.float64)
    if sal_v_blk is None:
        sal_v_blk = torch.empty(B, n_b, dtype=torch.float32, device=dev)
    if sal_v_tok is None and want_tok:
        sal_v_tok = torch.empty(B, L_v, dtype=torch.float32, device=dev)
    if sal_a_tok is None:
        sal_a_tok = torch.empty(B, L_a, dtype=torch.float32, device=dev)
    if qbar is None:
        qbar = torch.empty(B, H, d, n_pad, dtype=torch.float64, device=dev)
    if kbar is None:
        kbar = torch.empty(B, H, d, n_pad, dtype=torch.float64, device=dev)
    ws = _workspace(SA_CALL_CROSS_SCORES, B, H, L_v, L_a, d, block, dev, ws)
    _check(lib().sa_cross_scores_pooled(
        _ptr(q_a), _ptr(k_v), _ptr(q_v), _ptr(k_a), _ptr(lse_a), _ptr(lse_v), B, H, L_v,
        L_a, d, _dtype_code(q_a), float(scale), block, _ptr(sal_v_tok), _ptr(sal_v_blk),
        _ptr(sal_a_tok), int(bool(accumulate)), _ptr(qbar), _ptr(kbar), _ptr(ws),
        _nbytes(ws), _stream()))
    return sal_v_tok, sal_v_blk, sal_a_tok, qbar, kbar


def sa_build_block_mask_pooled(qbar, kbar, L_v, scale, block, k_keep, prot_flag=None, *,
                               kv_idx=None, kv_cnt=None, want_mask=False,
                               want_scores=False, mask=None, scores=None):
    """sa_build_block_mask from the means of sa_cross_scores_pooled; returns
    (kv_idx, kv_cnt, mask, scores)."""
    B, H, d, n_pad = qbar.shape
    n_b = -(-L_v // block)
    dev = qbar.device
    _expect(qbar, "qbar", (B, H, d, sa_pool_columns(n_b)), torch.float64)
    _expect(kbar, "kbar", (B, H, d, n_pad), torch.float64)
    _expect(prot_flag, "prot_flag", (B, n_b), torch.uint8)
    _expect(kv_idx, "kv_idx", (B, H, n_b, n_b), torch.int32)
    _expect(kv_cnt, "kv_cnt", (B, H, n_b), torch.int32)
    _expect(mask, "mask", (B, H, n_b, n_b), torch.uint8)
    _expect(scores, "scores", (B, H, n_b, n_b), torch.float32)
    if kv_idx is None:
        kv_idx = torch.empty(B, H, n_b, n_b, dtype=torch.int32, device=dev)
    if kv_cnt is None:
        kv_cnt = torch.empty(B, H, n_b, dtype=torch.int32, device=dev)
    if mask is None and want_mask:
        mask = torch.empty(B, H, n_b, n_b, dtype=torch.uint8, device=dev)
    if scores is None and want_scores:
        scores = torch.empty(B, H, n_b, n_b, dtype=torch.float32, device=dev)
    _check(lib().sa_build_block_mask_pooled(
        _ptr(qbar), _ptr(kbar), B, H, L_v, d, float(scale), block, int(k_keep),
        _ptr(prot_flag), _ptr(kv_idx), _ptr(kv_cnt), _ptr(mask), _ptr(scores), _stream()))
    return kv_idx, kv_cnt, mask, scores


def sa_saliency_ema(sal_bar, sal, alpha):
    """Lagged saliency update in place: sal_bar = alpha*sal_bar + (1-alpha)*sal."""
    if sal_bar.dtype != torch.float32 or sal.dtype != torch.float32:
        raise TypeError("saliency maps are float32")
    if sal_bar.numel() != sal.numel():
        raise ValueError("sal_bar and sal differ in size")
    _check(lib().sa_saliency_ema(_ptr(sal_bar), _ptr(sal), sal_bar.numel(),
                                 float(alpha), _stream()))
    return sal_bar


def sa_select_protected_tokens(sal_tok, k_tok, *, tok_idx=None, tok_flag=None,
                               want_flag=True):
    """Protected tokens; returns (tok_idx [B,k_tok] i32 ascending, tok_flag [B,L] u8)."""
    B, L = sal_tok.shape
    dev = sal_tok.device
    _expect(sal_tok, "sal_tok", (B, L), torch.float32)
    _expect(tok_idx, "tok_idx", (B, max(k_tok, 0)), torch.int32)
    _expect(tok_flag, "tok_flag", (B, L), torch.uint8)
    if tok_idx is None:
        tok_idx = torch.empty(B, max(k_tok, 0), dtype=torch.int32, device=dev)
    if tok_flag is None and want_flag:
        tok_flag = torch.empty(B, L, dtype=torch.uint8, device=dev)
    _check(lib().sa_select_protected_tokens(_ptr(sal_tok), B, L, int(k_tok),
                                            _ptr(tok_idx) if k_tok > 0 else None,
                                            _ptr(tok_flag), _stream()))
    return tok_idx, tok_flag


def sa_protected_token_attention(q, k, v, scale, tok_idx, o, lse=None, *, ws=None):
    """Dense rows of the protected tokens written over o (and lse); returns (o, lse)."""
    B, H, L, d = q.shape
    k_tok = tok_idx.shape[1]
    for name, t in (("k", k), ("v", v), ("o", o)):
        _expect(t, name, (B, H, L, d), q.dtype)
    _expect(lse, "lse", (B, H, L), torch.float32)
    _expect(tok_idx, "tok_idx", (B, k_tok), torch.int32)
    ws = _workspace(SA_CALL_TOKEN_ATTENTION, B, H, L, k_tok, d, 0, q.device, ws)
    _check(lib().sa_protected_token_attention(
        _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, H, L, d, _dtype_code(q),
        float(scale), _ptr(tok_idx) if k_tok > 0 else None, int(k_tok), _ptr(ws),
        _nbytes(ws), _stream()))
    return o, lse


def sa_cache_indicator(y_v, y_v_hat, *, prot_flag=None, y_a=None, y_a_hat=None,
                       s_bar=None, s_hat=None, lambda_p=0.5, lambda_s=0.1, tau=0.2,
                       eps=1e-6, out=None, ws=None):
    """Cache-reuse indicator; returns out [6] f32 (device): dv, da, dp, ds,
    sync, reuse."""
    B, L_v, C = y_v.shape
    L_a = y_a.shape[1] if y_a is not None else 0
    dev = y_v.device
    _expect(y_v_hat, "y_v_hat", (B, L_v, C), y_v.dtype)
    _expect(prot_flag, "prot_flag", (B, L_v), torch.uint8)
    _expect(y_a, "y_a", (B, L_a, C), y_v.dtype)
    _expect(y_a_hat, "y_a_hat", (B, L_a, C), y_v.dtype)
    _expect(s_bar, "s_bar", (B, L_v), torch.float32)
    _expect(s_hat, "s_hat", (B, L_v), torch.float32)
    _expect(out, "out", (6,), torch.float32)
    if out is None:
        out = torch.empty(6, dtype=torch.float32, device=dev)
    need = sa_workspace_size(SA_CALL_CACHE_INDICATOR, B, 1, L_v, L_a, 128, 128)
    if ws is None:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    _check(lib().sa_cache_indicator(
        _ptr(y_v), _ptr(y_v_hat), _ptr(prot_flag), _ptr(y_a), _ptr(y_a_hat),
        _ptr(s_bar), _ptr(s_hat), B, L_v, L_a, C, _dtype_code(y_v), float(lambda_p),
        float(lambda_s), float(tau), float(eps), _ptr(out), _ptr(ws), _nbytes(ws),
        _stream()))
    return out


# ---- measurement helper library (libsa_bench.so, include/sa_bench.h) --------
BENCH_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)),
                              "libsa_bench.so")
BENCH_SIGNATURES = {
    "sa_bench_mfma_peak": (_I, [_I, _I, _I, ctypes.POINTER(_F), ctypes.POINTER(_F)]),
}
_bench_handle = None


def bench_lib():
    """The loaded measurement helper library (raises if it is not built)."""
    global _bench_handle
    if _bench_handle is None:
        if not os.path.exists(BENCH_LIB_PATH):
            raise SaError(-1, f"{BENCH_LIB_PATH} is missing: build it with "
                              "`python -m paper_2608_15522_amd.build`")
        handle = ctypes.CDLL(BENCH_LIB_PATH)
        for name, (res, args) in BENCH_SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _bench_handle = handle
    return _bench_handle


def sa_bench_mfma_peak(random_operands: bool = True, iters: int = 4096,
                       reps: int = 3):
    """Sustained bf16 MFMA throughput of the current device: (TFLOP/s, GHz),
    best of `reps` runs."""
    tf, ghz = _F(0.0), _F(0.0)
    rc = bench_lib().sa_bench_mfma_peak(int(bool(random_operands)), int(iters), int(reps),
                                        ctypes.byref(tf), ctypes.byref(ghz))
    if rc != 0:
        raise SaError(rc, "sa_bench_mfma_peak failed")
    return float(tf.value), float(ghz.value)
