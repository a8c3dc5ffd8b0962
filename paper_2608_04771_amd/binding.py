"""Thin Python binding of libreco.so (argument marshalling only).

Each function has the name of the C entry point it calls and forwards device
pointers (``tensor.data_ptr()``) and the current HIP stream of torch.  Every
step of the computation runs in the HIP kernels of the library; nothing here
computes a result.  The library must have been built in-tree
(``python -m paper_2608_04771_amd.build``); importing it otherwise fails.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libreco.so")

RECO_OK = 0
RECO_ERR_INVALID_ARG = 1
RECO_ERR_UNSUPPORTED = 2
RECO_ERR_WORKSPACE = 3
RECO_ERR_HIP = 4
RECO_F32 = 0
RECO_BF16 = 1
RECO_SCORE_CAUSAL = 1
RECO_POOL_MAX = 0
RECO_POOL_MEAN = 1
DEV_ERRORS = {0: "ok", 1: "append overflow", 2: "bad retention", 3: "bad score", 4: "bad token id",
              5: "bad length", 6: "bad logit row"}

EXPORTED = [
    "reco_score_workspace_size", "reco_score", "reco_select_compact_workspace_size", "reco_select_compact",
    "reco_pool_scores", "reco_layer_retention",
    "reco_decode_attn_workspace_size", "reco_decode_attn", "reco_decode_attn_noalloc", "reco_logit_penalty",
    "reco_penalty_sample_workspace_size", "reco_penalty_sample",
    "reco_answer_ppl_workspace_size", "reco_answer_ppl", "reco_retention_from_reward", "reco_retention_eq1",
    "reco_kept_count", "reco_status_str", "reco_abi_version",
]


class RecoKVCache(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("len", ctypes.c_void_p),
                ("n_layers", ctypes.c_int32), ("batch", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("capacity", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32)]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libreco.so; raises if it has not been built (no fallback exists)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"HIP library missing: {path} (build it with `python -m paper_2608_04771_amd.build`)")
    lib = ctypes.CDLL(path)
    P, I32, I64, F32, F64, SZ, U32, U64 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                                           ctypes.c_double, ctypes.c_size_t, ctypes.c_uint32, ctypes.c_uint64)
    C = ctypes.POINTER(RecoKVCache)
    sig = {
        "reco_score_workspace_size": (SZ, [C, I32, I32, I32]),
        "reco_score": (I32, [C, I32, I32, P, I32, I32, F32, U32, P, P, P, SZ, P, P]),
        "reco_select_compact_workspace_size": (SZ, [C, I32]),
        "reco_select_compact": (I32, [C, I32, I32, P, P, I64, I32, P, P, SZ, P, P]),
        "reco_pool_scores": (I32, [C, I32, I32, I32, P, P, I32, I32, P, P]),
        "reco_layer_retention": (F64, [F64, I32, I32, F64]),
        "reco_decode_attn_workspace_size": (SZ, [C, I32, I32]),
        "reco_decode_attn": (I32, [C, I32, I32, P, I32, F32, P, P, P, P, P, P, SZ, P, P]),
        "reco_decode_attn_noalloc": (I32, [C, I32, I32, P, I32, F32, P, P, P, P, P, P, P]),
        "reco_logit_penalty": (I32, [P, I32, I32, I64, P, I32, P, F32, F32, F32, F32, F32, P, P]),
        "reco_penalty_sample_workspace_size": (SZ, [I32, I32]),
        "reco_penalty_sample": (I32, [P, I32, I32, I64, P, I32, P, F32, F32, F32, F32, F32, F32, U64, U64, P, P, SZ,
                                      P, P]),
        "reco_answer_ppl_workspace_size": (SZ, [I32, I32, I32]),
        "reco_answer_ppl": (I32, [P, P, I32, I32, I32, F32, P, P, P, SZ, P, P]),
        "reco_retention_from_reward": (F64, [F64, F64, F64]),
        "reco_retention_eq1": (F64, [ctypes.POINTER(ctypes.c_double), I32, F64, F64]),
        "reco_kept_count": (I32, [I32, I32, F64]),
        "reco_status_str": (ctypes.c_char_p, [I32]),
        "reco_abi_version": (I32, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


# torch's current-stream handle without building a Stream object (a few
# microseconds per call otherwise); the public call is the fallback.
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream(device) -> ctypes.c_void_p:
    if _raw_stream is not None:
        idx = device.index if device.index is not None else torch.cuda.current_device()
        return ctypes.c_void_p(_raw_stream(idx))
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _check(status: int, what: str):
    if status != RECO_OK:
        msg = load_library().reco_status_str(status).decode()
        raise RuntimeError(f"{what} failed: {msg} (status {status})")


def _need_cuda(*ts):
    """Every given tensor (None skipped) is a contiguous tensor on one GPU."""
    dev = None
    for t in ts:
        if t is not None:
            if not t.is_cuda:
                raise ValueError("tensors must live on the GPU")
            if not t.is_contiguous():
                raise ValueError("tensors must be contiguous")
            d = t.get_device()
            if dev is None:
                dev = d
            elif d != dev:
                raise ValueError("tensors of one call must live on the same GPU")


def _same_gpu(a: torch.Tensor, b: torch.Tensor):
    if not a.is_cuda or a.get_device() != b.get_device():
        raise ValueError("tensors of one call must live on the same GPU")


_DT = {torch.float32: "float32", torch.bfloat16: "bfloat16", torch.float64: "float64", torch.int32: "int32",
       torch.uint8: "uint8"}


def _expect(t: Optional[torch.Tensor], what: str, shape, dtype: torch.dtype):
    """The C ABI sees only pointers, so every tensor it indexes is checked here
    against the exact shape and dtype the call reads or writes: an undersized
    or mistyped buffer would otherwise be read or written out of bounds."""
    if t is None:
        return
    if tuple(t.shape) != tuple(shape) or t.dtype != dtype:
        raise ValueError(f"{what} must be {_DT.get(dtype, dtype)} {list(shape)}, "
                         f"got {_DT.get(t.dtype, t.dtype)} {list(t.shape)}")


def _expect_dev_err(dev_err: Optional[torch.Tensor]):
    if dev_err is not None and (dev_err.dtype != torch.int32 or dev_err.numel() < 1):
        raise ValueError("dev_err must be an int32 tensor with at least one element")


def _nbytes(t: torch.Tensor) -> int:
    return t.numel() * t.element_size()


class KVCache:
    """A KV cache in the library's layout: K and V ``[NL][B][H][Cap][D]``
    (fp32 or bf16), ``length`` ``[NL][B][H]`` int32, all on the GPU."""

    def __init__(self, k: torch.Tensor, v: torch.Tensor, length: torch.Tensor):
        if k.shape != v.shape or k.dim() != 5 or k.dtype != v.dtype:
            raise ValueError("k and v must share a [NL][B][H][Cap][D] shape and dtype")
        if k.dtype not in (torch.float32, torch.bfloat16):
            raise ValueError("cache dtype must be float32 or bfloat16")
        if length.dtype != torch.int32 or tuple(length.shape) != tuple(k.shape[:3]):
            raise ValueError("length must be int32 [NL][B][H]")
        _need_cuda(k, v, length)
        self.k, self.v, self.length = k, v, length
        NL, B, H, Cap, D = k.shape
        self.struct = RecoKVCache(k.data_ptr(), v.data_ptr(), length.data_ptr(), NL, B, H, Cap, D,
                                  RECO_F32 if k.dtype == torch.float32 else RECO_BF16)

    @property
    def shape(self):
        return tuple(self.k.shape)

    def ref(self):
        return ctypes.byref(self.struct)


def _layers(cache: KVCache, layer0: int, n_layers: Optional[int]):
    layer0 = int(layer0)
    nl = (cache.shape[0] - layer0) if n_layers is None else int(n_layers)
    if layer0 < 0 or nl < 1 or layer0 + nl > cache.shape[0]:
        raise ValueError(f"layers [{layer0}, {layer0 + nl}) outside the cache's {cache.shape[0]} layers")
    return layer0, nl


def score_workspace_size(cache: KVCache, n_q_heads: int, w: int, n_layers: Optional[int] = None) -> int:
    nl = cache.shape[0] if n_layers is None else n_layers
    return int(load_library().reco_score_workspace_size(cache.ref(), nl, n_q_heads, w))


def select_compact_workspace_size(cache: KVCache, n_layers: Optional[int] = None) -> int:
    nl = cache.shape[0] if n_layers is None else n_layers
    return int(load_library().reco_select_compact_workspace_size(cache.ref(), nl))


def decode_attn_workspace_size(cache: KVCache, n_q_heads: int, n_layers: Optional[int] = None) -> int:
    nl = cache.shape[0] if n_layers is None else n_layers
    return int(load_library().reco_decode_attn_workspace_size(cache.ref(), nl, n_q_heads))


def penalty_sample_workspace_size(rows: int, vocab: int) -> int:
    return int(load_library().reco_penalty_sample_workspace_size(rows, vocab))


def answer_ppl_workspace_size(batch: int, n: int, vocab: int) -> int:
    return int(load_library().reco_answer_ppl_workspace_size(batch, n, vocab))


def _ws(nbytes, device, ws: Optional[torch.Tensor]) -> torch.Tensor:
    """The caller's workspace, else a new one of nbytes() bytes (the library
    checks the size either way)."""
    if ws is not None:
        return ws
    return torch.empty(max(int(nbytes()), 1), dtype=torch.uint8, device=device)


def decode_workspace(cache: "KVCache", n_q_heads: int, n_layers: Optional[int] = None) -> torch.Tensor:
    """A decode workspace (contents need not be initialised).  Do not share
    one between overlapping calls."""
    return _ws(lambda: decode_attn_workspace_size(cache, n_q_heads, n_layers), cache.k.device, None)


def _score_shapes(cache: KVCache, nl: int, q_win: torch.Tensor, w: int, scores, row_stats):
    NL, B, H, Cap, D = cache.shape
    if q_win.dim() != 5 or q_win.shape[0] != nl or q_win.shape[1] != B or q_win.shape[3] != w or q_win.shape[4] != D:
        raise ValueError("q_win must be [n_layers][B][Hq][w][D]")
    if q_win.dtype != cache.k.dtype:
        raise ValueError("q_win must have the cache dtype")
    hq = q_win.shape[2]
    _expect(scores, "scores", (nl, B, H, Cap), torch.float32)
    _expect(row_stats, "row_stats", (nl, B, hq, w, 2), torch.float32)
    return hq


def reco_score(cache: KVCache, q_win: torch.Tensor, w: int, scale: Optional[float] = None, causal: bool = True,
               scores: Optional[torch.Tensor] = None, layer0: int = 0, n_layers: Optional[int] = None,
               ws: Optional[torch.Tensor] = None, dev_err: Optional[torch.Tensor] = None,
               row_stats: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Eq. 2 window attention mass; returns scores [n_layers][B][H][Cap] fp32.
    ``row_stats`` ([n_layers][B][Hq][w][2], from the window tokens' decode
    steps) replaces the normaliser pass over K."""
    layer0, nl = _layers(cache, layer0, n_layers)
    hq = _score_shapes(cache, nl, q_win, w, scores, row_stats)
    _expect_dev_err(dev_err)
    NL, B, H, Cap, D = cache.shape
    _need_cuda(cache.k, q_win, scores, ws, dev_err, row_stats)
    if scores is None:
        scores = torch.zeros((nl, B, H, Cap), dtype=torch.float32, device=cache.k.device)
    ws = _ws(lambda: score_workspace_size(cache, hq, w, nl), cache.k.device, ws)
    scale = 1.0 / math.sqrt(D) if scale is None else float(scale)
    st = load_library().reco_score(cache.ref(), layer0, nl, _ptr(q_win), hq, w, scale,
                                   RECO_SCORE_CAUSAL if causal else 0, _ptr(row_stats), _ptr(scores), _ptr(ws),
                                   _nbytes(ws), _ptr(dev_err), _stream(cache.k.device))
    _check(st, "reco_score")
    return scores


def _select_shapes(cache: KVCache, nl: int, scores: torch.Tensor, retention: torch.Tensor, kept_idx):
    NL, Bsz, H, Cap, D = cache.shape
    if retention.dtype != torch.float64:
        raise ValueError("retention must be float64")
    if tuple(retention.shape) == (Bsz,):
        stride = 0
    elif tuple(retention.shape) == (nl, Bsz):
        stride = Bsz
    else:
        raise ValueError("retention must be [B] or [n_layers][B]")
    _expect(scores, "scores", (nl, Bsz, H, Cap), torch.float32)
    _expect(kept_idx, "kept_idx", (nl, Bsz, H, Cap), torch.int32)
    return stride


def reco_select_compact(cache: KVCache, scores: torch.Tensor, retention: torch.Tensor, w: int,
                        kept_idx: Optional[torch.Tensor] = None, layer0: int = 0, n_layers: Optional[int] = None,
                        ws: Optional[torch.Tensor] = None, dev_err: Optional[torch.Tensor] = None):
    """Select the reward budget per unit and compact K/V in place (len <- m).
    ``retention`` is float64 [B] (one level per sequence) or [n_layers][B]
    (per-layer budgets)."""
    layer0, nl = _layers(cache, layer0, n_layers)
    stride = _select_shapes(cache, nl, scores, retention, kept_idx)
    _expect_dev_err(dev_err)
    _need_cuda(cache.k, scores, retention, kept_idx, ws, dev_err)
    ws = _ws(lambda: select_compact_workspace_size(cache, nl), cache.k.device, ws)
    st = load_library().reco_select_compact(cache.ref(), layer0, nl, _ptr(scores), _ptr(retention), stride, w,
                                            _ptr(kept_idx), _ptr(ws), _nbytes(ws), _ptr(dev_err),
                                            _stream(cache.k.device))
    _check(st, "reco_select_compact")
    return kept_idx


def reco_pool_scores(cache: KVCache, scores: torch.Tensor, w: int, kernel: int, mode: str = "max",
                     pooled: Optional[torch.Tensor] = None, layer0: int = 0, n_layers: Optional[int] = None,
                     dev_err: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Max / mean pooling of the prefix scores (window scores copied); returns
    pooled [n_layers][B][H][Cap] fp32 (entries at or beyond len unwritten)."""
    layer0, nl = _layers(cache, layer0, n_layers)
    NL, Bsz, H, Cap, D = cache.shape
    if mode not in ("max", "mean"):
        raise ValueError("mode must be 'max' or 'mean'")
    _expect(scores, "scores", (nl, Bsz, H, Cap), torch.float32)
    _expect(pooled, "pooled", (nl, Bsz, H, Cap), torch.float32)
    _expect_dev_err(dev_err)
    _need_cuda(cache.k, scores, pooled, dev_err)
    if pooled is None:
        pooled = torch.zeros_like(scores)
    st = load_library().reco_pool_scores(cache.ref(), layer0, nl, w, _ptr(scores), _ptr(pooled), kernel,
                                         RECO_POOL_MAX if mode == "max" else RECO_POOL_MEAN, _ptr(dev_err),
                                         _stream(cache.k.device))
    _check(st, "reco_pool_scores")
    return pooled


def _decode_shapes(cache: KVCache, nl: int, q: torch.Tensor, k_new, v_new, out, lse, row_stats):
    NL, B, H, Cap, D = cache.shape
    if q.dim() != 4 or q.shape[0] != nl or q.shape[1] != B or q.shape[3] != D or q.dtype != cache.k.dtype:
        raise ValueError("q must be [n_layers][B][Hq][D] in the cache dtype")
    hq = q.shape[2]
    if (k_new is None) != (v_new is None):
        raise ValueError("k_new and v_new must be given together")
    _expect(k_new, "k_new", (nl, B, H, D), cache.k.dtype)
    _expect(v_new, "v_new", (nl, B, H, D), cache.k.dtype)
    _expect(out, "out", (nl, B, hq, D), cache.k.dtype)
    _expect(lse, "lse", (nl, B, hq), torch.float32)
    _expect(row_stats, "row_stats", (nl, B, hq, 2), torch.float32)
    return hq


def reco_decode_attn(cache: KVCache, q: torch.Tensor, k_new: Optional[torch.Tensor] = None,
                     v_new: Optional[torch.Tensor] = None, scale: Optional[float] = None,
                     out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None, want_lse: bool = True,
                     layer0: int = 0, n_layers: Optional[int] = None, ws: Optional[torch.Tensor] = None,
                     dev_err: Optional[torch.Tensor] = None, row_stats: Optional[torch.Tensor] = None):
    """GQA decode attention (optionally appending the new token); returns (out, lse).
    ``row_stats`` ([n_layers][B][Hq][2] fp32) optionally receives each query's
    (max, sum) of the log2-domain logits."""
    layer0, nl = _layers(cache, layer0, n_layers)
    hq = _decode_shapes(cache, nl, q, k_new, v_new, out, lse, row_stats)
    _expect_dev_err(dev_err)
    _need_cuda(cache.k, q, k_new, v_new, out, lse, ws, dev_err, row_stats)
    NL, B, H, Cap, D = cache.shape
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty((nl, B, hq), dtype=torch.float32, device=q.device)
    ws = _ws(lambda: decode_attn_workspace_size(cache, hq, nl), q.device, ws)
    scale = 1.0 / math.sqrt(D) if scale is None else float(scale)
    st = load_library().reco_decode_attn(cache.ref(), layer0, nl, _ptr(q), hq, scale, _ptr(k_new), _ptr(v_new),
                                         _ptr(out), _ptr(lse), _ptr(row_stats), _ptr(ws), _nbytes(ws),
                                         _ptr(dev_err), _stream(q.device))
    _check(st, "reco_decode_attn")
    return out, lse


def reco_decode_attn_noalloc(cache: KVCache, q: torch.Tensor, out: torch.Tensor, lse: Optional[torch.Tensor] = None,
                             k_new: Optional[torch.Tensor] = None, v_new: Optional[torch.Tensor] = None,
                             scale: Optional[float] = None, layer0: int = 0, n_layers: Optional[int] = None,
                             dev_err: Optional[torch.Tensor] = None, row_stats: Optional[torch.Tensor] = None):
    """reco_decode_attn without a workspace and without any allocation: the
    caller passes ``out`` (and optionally ``lse``); the split partials live in
    the library's static per-device array.  Calls overlapping on one GPU race."""
    layer0, nl = _layers(cache, layer0, n_layers)
    if out is None:
        raise ValueError("out must be given (this entry point allocates nothing)")
    _decode_shapes(cache, nl, q, k_new, v_new, out, lse, row_stats)
    _expect_dev_err(dev_err)
    _need_cuda(cache.k, q, k_new, v_new, out, lse, dev_err, row_stats)
    D = cache.shape[4]
    scale = 1.0 / math.sqrt(D) if scale is None else float(scale)
    st = load_library().reco_decode_attn_noalloc(cache.ref(), layer0, nl, _ptr(q), q.shape[2], scale, _ptr(k_new),
                                                 _ptr(v_new), _ptr(out), _ptr(lse), _ptr(row_stats), _ptr(dev_err),
                                                 _stream(q.device))
    _check(st, "reco_decode_attn_noalloc")
    return out, lse


class PreparedDecode:
    """reco_decode_attn for a loop that calls it again and again with the same
    cache, outputs, workspace and error word (a decoder's per-token call):
    those are checked once here, and each call checks only the tensors that
    change from token to token (query, new K/V rows, statistics slot) against
    the shapes fixed at construction before passing their pointers on.  The
    library computes exactly what reco_decode_attn computes."""

    def __init__(self, cache: KVCache, n_q_heads: int, out: torch.Tensor, lse: Optional[torch.Tensor],
                 ws: torch.Tensor, dev_err: Optional[torch.Tensor] = None, scale: Optional[float] = None,
                 layer0: int = 0, n_layers: Optional[int] = None):
        layer0, nl = _layers(cache, layer0, n_layers)
        NL, Bsz, H, Cap, D = cache.shape
        hq = int(n_q_heads)
        if out is None or ws is None:
            raise ValueError("out and ws must be given")
        _expect(out, "out", (nl, Bsz, hq, D), cache.k.dtype)
        _expect(lse, "lse", (nl, Bsz, hq), torch.float32)
        _expect_dev_err(dev_err)
        _need_cuda(cache.k, out, lse, ws, dev_err)
        _same_gpu(out, cache.k)
        if _nbytes(ws) < decode_attn_workspace_size(cache, hq, nl):
            raise ValueError("ws is smaller than reco_decode_attn_workspace_size")
        self.cache, self.out, self.lse, self.ws, self.dev_err = cache, out, lse, ws, dev_err
        self._fn = load_library().reco_decode_attn
        self._dev = cache.k.device
        self._dt = cache.k.dtype
        self._q_shape = (nl, Bsz, hq, D)
        self._kv_shape = (nl, Bsz, H, D)
        self._st_shape = (nl, Bsz, hq, 2)
        self._fixed_head = (cache.ref(), layer0, nl)
        self._hq = hq
        self._scale = 1.0 / math.sqrt(D) if scale is None else float(scale)
        self._fixed_tail = (_ptr(out), _ptr(lse))
        self._ws = (_ptr(ws), _nbytes(ws), _ptr(dev_err))

    def _check_t(self, t: torch.Tensor, what: str, shape, dtype: torch.dtype):
        if (tuple(t.shape) != shape or t.dtype != dtype or t.device != self._dev or not t.is_contiguous()):
            raise ValueError(f"{what} must be a contiguous {_DT.get(dtype, dtype)} {list(shape)} tensor on "
                             f"{self._dev}")

    def __call__(self, q: torch.Tensor, k_new: Optional[torch.Tensor] = None, v_new: Optional[torch.Tensor] = None,
                 row_stats: Optional[torch.Tensor] = None):
        self._check_t(q, "q", self._q_shape, self._dt)
        if (k_new is None) != (v_new is None):
            raise ValueError("k_new and v_new must be given together")
        if k_new is not None:
            self._check_t(k_new, "k_new", self._kv_shape, self._dt)
            self._check_t(v_new, "v_new", self._kv_shape, self._dt)
        if row_stats is not None:
            self._check_t(row_stats, "row_stats", self._st_shape, torch.float32)
        cref, layer0, nl = self._fixed_head
        st = self._fn(cref, layer0, nl, _ptr(q), self._hq, self._scale, _ptr(k_new), _ptr(v_new),
                      *self._fixed_tail, _ptr(row_stats), *self._ws, _stream(self._dev))
        if st != RECO_OK:
            _check(st, "reco_decode_attn")
        return self.out, self.lse


def _logit_rows(logits: torch.Tensor):
    if logits.dtype != torch.float32 or logits.dim() != 2 or logits.stride(1) != 1 or \
            logits.stride(0) < logits.shape[1]:
        raise ValueError("logits must be fp32 [rows][vocab] with unit column stride and row stride >= vocab")
    return logits.shape


def reco_logit_penalty(logits: torch.Tensor, refl_ids: torch.Tensor, reward: torch.Tensor, tau_lo: float,
                       tau_hi: float, beta_lo: float, beta_mid: float, beta_hi: float,
                       dev_err: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Eq. 3-4 in place on fp32 logits [rows][vocab] (row stride may exceed vocab)."""
    rows, vocab = _logit_rows(logits)
    if refl_ids.dtype != torch.int32 or refl_ids.dim() != 1:
        raise ValueError("refl_ids must be a 1-D int32 tensor")
    _expect(reward, "reward", (rows,), torch.float32)
    _expect_dev_err(dev_err)
    _need_cuda(refl_ids, reward, dev_err)
    _same_gpu(logits, reward)
    st = load_library().reco_logit_penalty(_ptr(logits), rows, vocab, logits.stride(0), _ptr(refl_ids),
                                           refl_ids.numel(), _ptr(reward), tau_lo, tau_hi, beta_lo, beta_mid,
                                           beta_hi, _ptr(dev_err), _stream(logits.device))
    _check(st, "reco_logit_penalty")
    return logits


def reco_penalty_sample(logits: torch.Tensor, refl_ids: Optional[torch.Tensor], reward: torch.Tensor, tau_lo: float,
                        tau_hi: float, beta_lo: float, beta_mid: float, beta_hi: float, temperature: float,
                        seed: int, offset: int, tokens: Optional[torch.Tensor] = None,
                        ws: Optional[torch.Tensor] = None, dev_err: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Eq. 3-4 in place on fp32 logits [rows][vocab], then the next token of
    each row from softmax(z~ / T) (greedy when T = 0); returns tokens [rows] int32."""
    rows, vocab = _logit_rows(logits)
    if refl_ids is not None and (refl_ids.dtype != torch.int32 or refl_ids.dim() != 1):
        raise ValueError("refl_ids must be a 1-D int32 tensor")
    _expect(reward, "reward", (rows,), torch.float32)
    _expect(tokens, "tokens", (rows,), torch.int32)
    _expect_dev_err(dev_err)
    _need_cuda(reward, refl_ids, tokens, ws, dev_err)
    _same_gpu(logits, reward)
    if tokens is None:
        tokens = torch.empty(rows, dtype=torch.int32, device=logits.device)
    ws = _ws(lambda: penalty_sample_workspace_size(rows, vocab), logits.device, ws)
    n_refl = 0 if refl_ids is None else refl_ids.numel()
    st = load_library().reco_penalty_sample(_ptr(logits), rows, vocab, logits.stride(0), _ptr(refl_ids), n_refl,
                                            _ptr(reward), tau_lo, tau_hi, beta_lo, beta_mid, beta_hi,
                                            float(temperature), int(seed) & (2 ** 64 - 1),
                                            int(offset) & (2 ** 64 - 1), _ptr(tokens), _ptr(ws), _nbytes(ws),
                                            _ptr(dev_err), _stream(logits.device))
    _check(st, "reco_penalty_sample")
    return tokens


class PreparedPenaltySample:
    """reco_penalty_sample for a loop over logit rows of one shape (a
    decoder's per-token draw): the reflection ids, the per-row rewards, the
    token output, the workspace and the error word are checked once, and each
    call checks only the logit rows before passing their pointer on, with
    the temperature, seed and draw offset of that call."""

    def __init__(self, rows: int, vocab: int, refl_ids: Optional[torch.Tensor], reward: torch.Tensor,
                 tokens: torch.Tensor, ws: torch.Tensor, dev_err: Optional[torch.Tensor] = None):
        rows, vocab = int(rows), int(vocab)
        if refl_ids is not None and (refl_ids.dtype != torch.int32 or refl_ids.dim() != 1):
            raise ValueError("refl_ids must be a 1-D int32 tensor")
        if tokens is None or ws is None:
            raise ValueError("tokens and ws must be given")
        _expect(reward, "reward", (rows,), torch.float32)
        _expect(tokens, "tokens", (rows,), torch.int32)
        _expect_dev_err(dev_err)
        _need_cuda(reward, refl_ids, tokens, ws, dev_err)
        _same_gpu(tokens, reward)
        if _nbytes(ws) < penalty_sample_workspace_size(rows, vocab):
            raise ValueError("ws is smaller than reco_penalty_sample_workspace_size")
        self.tokens = tokens
        self._keep = (refl_ids, reward, ws, dev_err)
        self._fn = load_library().reco_penalty_sample
        self._dev = reward.device
        self._rows, self._vocab = rows, vocab
        self._ids = (_ptr(refl_ids), 0 if refl_ids is None else refl_ids.numel(), _ptr(reward))
        self._tail = (_ptr(tokens), _ptr(ws), _nbytes(ws), _ptr(dev_err))

    def __call__(self, logits: torch.Tensor, tau_lo: float, tau_hi: float, beta_lo: float, beta_mid: float,
                 beta_hi: float, temperature: float, seed: int, offset: int) -> torch.Tensor:
        if (logits.dtype != torch.float32 or logits.dim() != 2 or tuple(logits.shape) != (self._rows, self._vocab)
                or logits.stride(1) != 1 or logits.stride(0) < self._vocab or logits.device != self._dev):
            raise ValueError(f"logits must be fp32 [{self._rows}][{self._vocab}] with unit column stride on "
                             f"{self._dev}")
        st = self._fn(_ptr(logits), self._rows, self._vocab, logits.stride(0), *self._ids, tau_lo, tau_hi, beta_lo,
                      beta_mid, beta_hi, float(temperature), int(seed) & (2 ** 64 - 1), int(offset) & (2 ** 64 - 1),
                      *self._tail, _stream(self._dev))
        if st != RECO_OK:
            _check(st, "reco_penalty_sample")
        return self.tokens


def reco_answer_ppl(logits: torch.Tensor, tokens: torch.Tensor, tau_p: float, ppl: Optional[torch.Tensor] = None,
                    stop: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                    dev_err: Optional[torch.Tensor] = None):
    """Eq. 5-6: returns (ppl [B] fp32, stop [B] int32)."""
    if logits.dtype != torch.float32 or logits.dim() != 3:
        raise ValueError("logits must be fp32 [B][n][V]")
    B, n, V = logits.shape
    _expect(tokens, "tokens", (B, n), torch.int32)
    _expect(ppl, "ppl", (B,), torch.float32)
    _expect(stop, "stop", (B,), torch.int32)
    _expect_dev_err(dev_err)
    _need_cuda(logits, tokens, ppl, stop, ws, dev_err)
    if ppl is None:
        ppl = torch.empty(B, dtype=torch.float32, device=logits.device)
    if stop is None:
        stop = torch.empty(B, dtype=torch.int32, device=logits.device)
    ws = _ws(lambda: answer_ppl_workspace_size(B, n, V), logits.device, ws)
    st = load_library().reco_answer_ppl(_ptr(logits), _ptr(tokens), B, n, V, tau_p, _ptr(ppl), _ptr(stop),
                                        _ptr(ws), _nbytes(ws), _ptr(dev_err), _stream(logits.device))
    _check(st, "reco_answer_ppl")
    return ppl, stop


def reco_retention_from_reward(v: float, lo: float = 0.3, hi: float = 1.0) -> float:
    return float(load_library().reco_retention_from_reward(float(v), float(lo), float(hi)))


def reco_retention_eq1(v_hist: Sequence[float], lam: float = 0.25, delta: float = 0.1) -> float:
    arr = (ctypes.c_double * len(v_hist))(*[float(x) for x in v_hist])
    return float(load_library().reco_retention_eq1(arr, len(v_hist), float(lam), float(delta)))


def reco_layer_retention(r: float, layer: int, n_layers: int, spread: float) -> float:
    return float(load_library().reco_layer_retention(float(r), int(layer), int(n_layers), float(spread)))


def reco_kept_count(L: int, w: int, r: float) -> int:
    return int(load_library().reco_kept_count(int(L), int(w), float(r)))


def reco_abi_version() -> int:
    return int(load_library().reco_abi_version())
