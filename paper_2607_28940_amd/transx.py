"""Python binding of libtransx.so (the TransX serving path on MI355X).

Argument marshalling only: every step of the path runs in the library's HIP
kernels. PyTorch provides device memory (weights, the page pool, workspaces,
inputs, outputs) and the stream; the functions mirror the C ABI of
include/transx.h (kv_cache_build, kv_cache_append, score_candidates).
If the library has not been built, loading fails loudly: there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import List, Optional, Sequence

import numpy as np

from .inputs import ModelConfig

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtransx.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "transx.h")

TX_OK, TX_E_INVALID, TX_E_NOMEM, TX_E_NOCACHE, TX_E_HIP, TX_E_UNSUPPORTED = 0, -1, -2, -3, -4, -5
TX_F32, TX_BF16 = 0, 1
TX_OP_BUILD, TX_OP_APPEND, TX_OP_SCORE = 0, 1, 2
PAGE_TOKENS = 64
STATUS_NAMES = {0: "TX_OK", -1: "TX_E_INVALID", -2: "TX_E_NOMEM", -3: "TX_E_NOCACHE", -4: "TX_E_HIP",
                -5: "TX_E_UNSUPPORTED"}


class TxError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {msg}")
        self.code = code


class Config(ctypes.Structure):
    _fields_ = [("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32), ("d_ffn", ctypes.c_int32),
                ("n_enc_layers", ctypes.c_int32), ("n_dec_layers", ctypes.c_int32),
                ("rel_pos_buckets", ctypes.c_int32), ("ln_eps", ctypes.c_float), ("dtype", ctypes.c_int32),
                ("l_local", ctypes.c_int32), ("global_pool", ctypes.c_int32), ("n_actions", ctypes.c_int32)]

    @classmethod
    def of(cls, m: ModelConfig) -> "Config":
        return cls(m.d_model, m.n_heads, m.d_ffn, m.n_enc_layers, m.n_dec_layers, m.rel_pos_buckets,
                   float(m.ln_eps), TX_BF16 if m.dtype == "bf16" else TX_F32, int(m.l_local),
                   int(bool(m.global_pool)), int(m.n_actions))


_lib = None
VP = ctypes.c_void_p
I32P = ctypes.POINTER(ctypes.c_int32)
I64P = ctypes.POINTER(ctypes.c_int64)
CFGP = ctypes.POINTER(Config)

_SIGS = {
    "tx_last_error": (ctypes.c_char_p, []),
    "tx_num_weights": (ctypes.c_int32, [CFGP]),
    "tx_model_repack_bytes": (ctypes.c_size_t, [CFGP]),
    "tx_model_create": (ctypes.c_int, [CFGP, VP, ctypes.c_size_t, ctypes.c_uint64, ctypes.POINTER(VP)]),
    "tx_model_set_weights": (ctypes.c_int, [VP, ctypes.POINTER(VP), ctypes.c_int32, VP]),
    "tx_model_destroy": (None, [VP]),
    "tx_kv_page_bytes": (ctypes.c_size_t, [CFGP]),
    "tx_kv_pool_bytes": (ctypes.c_size_t, [CFGP, ctypes.c_int64, ctypes.c_int32, ctypes.c_int64]),
    "tx_kv_cache_create": (ctypes.c_int, [VP, VP, ctypes.c_size_t, ctypes.c_int64, ctypes.c_int32, ctypes.c_int64,
                                          ctypes.POINTER(VP)]),
    "tx_kv_cache_destroy": (None, [VP]),
    "tx_kv_cache_release": (ctypes.c_int, [VP, ctypes.c_int32, I32P]),
    "tx_kv_cache_length": (ctypes.c_int, [VP, ctypes.c_int32, I64P]),
    "tx_kv_cache_free_pages": (ctypes.c_int64, [VP]),
    "tx_kv_cache_model_id": (ctypes.c_uint64, [VP]),
    "tx_kv_cache_export": (ctypes.c_int, [VP, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, VP, VP]),
    "tx_workspace_bytes": (ctypes.c_size_t, [VP, ctypes.c_int32, ctypes.c_int32, I64P, I64P]),
    "tx_workspace_min_bytes": (ctypes.c_size_t, [VP, ctypes.c_int32, ctypes.c_int32, I64P, I64P]),
    "kv_cache_build": (ctypes.c_int, [VP, ctypes.c_int32, I32P, VP, I64P, VP, ctypes.c_size_t, VP]),
    "kv_cache_append": (ctypes.c_int, [VP, ctypes.c_int32, I32P, VP, I64P, VP, ctypes.c_size_t, VP]),
    "score_candidates": (ctypes.c_int, [VP, ctypes.c_int32, I32P, VP, I64P, VP, I64P, VP, VP, ctypes.c_size_t, VP]),
    "score_candidates_static": (ctypes.c_int, [VP, ctypes.c_int32, I32P, VP, I64P, VP, I64P, VP, VP]),
    "score_events": (ctypes.c_int, [VP, ctypes.c_int32, I32P, I64P, VP, I64P, VP, I64P, VP, VP, ctypes.c_size_t, VP]),
    "tx_profile_enable": (ctypes.c_int, [ctypes.c_int32]),
    "tx_profile_select": (ctypes.c_int, [ctypes.c_uint64]),
    "tx_profile_classes": (ctypes.c_int32, []),
    "tx_profile_class_name": (ctypes.c_char_p, [ctypes.c_int32]),
    "tx_profile_read": (ctypes.c_int, [ctypes.POINTER(ctypes.c_double), I64P, ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(ctypes.c_double)]),
}


def header_functions() -> List[str]:
    """Names of the functions include/transx.h declares."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"^\s*#.*$", "", text, flags=re.M)  # preprocessor lines (macros)
    return sorted(set(re.findall(r"\b([A-Za-z_][A-Za-z0-9_]*)\s*\(", text)) -
                  {"if", "defined", "sizeof", "TRANSX_H"})


def lib():
    """Load libtransx.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build the HIP library first "
                               "(python -c 'import __graft_entry__ as g; g.build()')")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def check(code: int):
    if code != TX_OK:
        msg = lib().tx_last_error().decode(errors="replace")
        raise TxError(code, msg)


def _i64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int64))


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _p(a: np.ndarray, t):
    return a.ctypes.data_as(t)


def _stream(stream) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def _torch_dtype(m: ModelConfig):
    import torch
    return torch.bfloat16 if m.dtype == "bf16" else torch.float32


class Model:
    """Model config + repacked device weights (owns the repack buffer)."""

    def __init__(self, mc: ModelConfig, weights: Sequence, model_id: int = 1, device: str = "cuda", stream=None):
        import torch
        self.mc = mc
        self.cfg = Config.of(mc)
        L = lib()
        nbytes = L.tx_model_repack_bytes(ctypes.byref(self.cfg))
        if nbytes == 0:
            raise TxError(TX_E_INVALID, "unsupported model config")
        self.repack = torch.empty(nbytes, dtype=torch.uint8, device=device)
        h = VP()
        check(L.tx_model_create(ctypes.byref(self.cfg), VP(self.repack.data_ptr()), nbytes, model_id,
                                ctypes.byref(h)))
        self.handle = h
        dt = _torch_dtype(mc)
        src = [torch.as_tensor(np.asarray(w, dtype=np.float32)).to(dt).to(device).contiguous() for w in weights]
        ptrs = (VP * len(src))(*[VP(t.data_ptr()) if t.numel() else VP() for t in src])
        check(L.tx_model_set_weights(self.handle, ptrs, len(src), VP(_stream(stream))))
        (stream or torch.cuda.current_stream()).synchronize()  # sources may go now
        self.model_id = model_id

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.tx_model_destroy(self.handle)
            self.handle = None


class KVCache:
    """Paged per-request cache in a torch-owned device pool, plus a growable
    torch workspace reused across calls."""

    def __init__(self, model: Model, n_pages: int, max_requests: int, max_tokens: int, device: str = "cuda",
                 fill_byte: Optional[int] = None):
        import torch
        self.model = model
        L = lib()
        nbytes = L.tx_kv_pool_bytes(ctypes.byref(model.cfg), n_pages, max_requests, max_tokens)
        if nbytes == 0:
            raise TxError(TX_E_INVALID, "bad pool geometry")
        self.pool = torch.empty(nbytes, dtype=torch.uint8, device=device)
        if fill_byte is not None:
            self.pool.fill_(fill_byte)
        h = VP()
        check(L.tx_kv_cache_create(model.handle, VP(self.pool.data_ptr()), nbytes, n_pages, max_requests,
                                   max_tokens, ctypes.byref(h)))
        self.handle = h
        self.ws = None
        self.device = device

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.tx_kv_cache_destroy(self.handle)
            self.handle = None

    # ---------------------------------------------------------------- helpers
    def workspace(self, nbytes: int):
        import torch
        if self.ws is None or self.ws.numel() < nbytes:
            self.ws = None
            self.ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        return self.ws

    def workspace_bytes(self, op: int, n: int, a, b=None) -> int:
        a = _i64(a)
        bp = _p(_i64(b), I64P) if b is not None else None
        return int(lib().tx_workspace_bytes(self.handle, op, n, _p(a, I64P), bp))

    def workspace_min_bytes(self, op: int, n: int, a, b=None) -> int:
        a = _i64(a)
        bp = _p(_i64(b), I64P) if b is not None else None
        return int(lib().tx_workspace_min_bytes(self.handle, op, n, _p(a, I64P), bp))

    def _ws_for(self, op, n, a, b, ws_limit):
        need = self.workspace_bytes(op, n, a, b)
        if ws_limit is not None:
            need = min(need, max(int(ws_limit), self.workspace_min_bytes(op, n, a, b)))
        ws = self.workspace(need)
        return ws, need

    # ---------------------------------------------------------------- the path
    def build(self, req_ids, behavior, offsets, stream=None, ws_limit: Optional[int] = None):
        ids, off = _i32(req_ids), _i64(offsets)
        ws, n = self._ws_for(TX_OP_BUILD, len(ids), off, None, ws_limit)
        check(lib().kv_cache_build(self.handle, len(ids), _p(ids, I32P), VP(behavior.data_ptr()), _p(off, I64P),
                                   VP(ws.data_ptr()), n, VP(_stream(stream))))

    def append(self, req_ids, events, offsets, stream=None, ws_limit: Optional[int] = None):
        ids, off = _i32(req_ids), _i64(offsets)
        ws, n = self._ws_for(TX_OP_APPEND, len(ids), off, None, ws_limit)
        check(lib().kv_cache_append(self.handle, len(ids), _p(ids, I32P), VP(events.data_ptr()), _p(off, I64P),
                                    VP(ws.data_ptr()), n, VP(_stream(stream))))

    def score(self, req_ids, serving, serving_offsets, candidates, candidate_offsets, out=None, stream=None,
              ws_limit: Optional[int] = None):
        import torch
        ids, so, co = _i32(req_ids), _i64(serving_offsets), _i64(candidate_offsets)
        if out is None:
            n = int(co[-1]) if len(co) else 0
            k = self.model.mc.n_actions
            out = torch.empty((n, k) if k else n, dtype=torch.float32, device=self.device)
        ws, n = self._ws_for(TX_OP_SCORE, len(ids), so, co, ws_limit)
        check(lib().score_candidates(self.handle, len(ids), _p(ids, I32P), VP(serving.data_ptr()), _p(so, I64P),
                                     VP(candidates.data_ptr()), _p(co, I64P), VP(out.data_ptr()), VP(ws.data_ptr()),
                                     n, VP(_stream(stream))))
        return out

    def score_static(self, req_ids, serving, serving_offsets, candidates, candidate_offsets, out=None, stream=None):
        """score_candidates_static: no workspace argument, nothing allocated by
        the library (its fixed device array serves as the workspace)."""
        import torch
        ids, so, co = _i32(req_ids), _i64(serving_offsets), _i64(candidate_offsets)
        if out is None:
            n = int(co[-1]) if len(co) else 0
            k = self.model.mc.n_actions
            out = torch.empty((n, k) if k else n, dtype=torch.float32, device=self.device)
        check(lib().score_candidates_static(self.handle, len(ids), _p(ids, I32P), VP(serving.data_ptr()),
                                            _p(so, I64P), VP(candidates.data_ptr()), _p(co, I64P),
                                            VP(out.data_ptr()), VP(_stream(stream))))
        return out

    def score_events(self, req_ids, prefix_len, serving, serving_offsets, candidates, candidate_offsets, out=None,
                     stream=None, ws_limit: Optional[int] = None):
        """Event-sliced decoding: event e decodes against the first
        prefix_len[e] cached tokens of request req_ids[e] (ids may repeat)."""
        import torch
        ids, pre, so, co = _i32(req_ids), _i64(prefix_len), _i64(serving_offsets), _i64(candidate_offsets)
        if out is None:
            n = int(co[-1]) if len(co) else 0
            k = self.model.mc.n_actions
            out = torch.empty((n, k) if k else n, dtype=torch.float32, device=self.device)
        ws, n = self._ws_for(TX_OP_SCORE, len(ids), so, co, ws_limit)
        check(lib().score_events(self.handle, len(ids), _p(ids, I32P), _p(pre, I64P), VP(serving.data_ptr()),
                                 _p(so, I64P), VP(candidates.data_ptr()), _p(co, I64P), VP(out.data_ptr()),
                                 VP(ws.data_ptr()), n, VP(_stream(stream))))
        return out

    def release(self, req_ids):
        ids = _i32(req_ids)
        check(lib().tx_kv_cache_release(self.handle, len(ids), _p(ids, I32P)))

    def length(self, req_id: int) -> int:
        v = ctypes.c_int64()
        check(lib().tx_kv_cache_length(self.handle, req_id, ctypes.byref(v)))
        return v.value

    def free_pages(self) -> int:
        return int(lib().tx_kv_cache_free_pages(self.handle))

    def model_id(self) -> int:
        return int(lib().tx_kv_cache_model_id(self.handle))

    def export(self, req_id: int, part: int, layer: int, stream=None):
        """Cached tensor of a request as a dense [len, d] device tensor.
        part: 0 encoder K, 1 encoder V, 2 cross K, 3 cross V; 4 and 5 the
        global token's cross K and V (one row) of a model with global pooling."""
        import torch
        n = 1 if part >= 4 else self.length(req_id)
        out = torch.empty((max(n, 0), self.model.mc.d_model), dtype=_torch_dtype(self.model.mc), device=self.device)
        check(lib().tx_kv_cache_export(self.handle, req_id, part, layer, VP(out.data_ptr()), VP(_stream(stream))))
        return out


def profile_enable(on: bool = True):
    check(lib().tx_profile_enable(1 if on else 0))


def profile_select(classes) -> None:
    """Record only the named kernel classes (until profile_enable)."""
    L = lib()
    names = [L.tx_profile_class_name(i).decode() for i in range(L.tx_profile_classes())]
    mask = 0
    for c in classes:
        mask |= 1 << names.index(c)
    check(L.tx_profile_select(mask))


def profile_read() -> dict:
    """{class name: {"ms": total, "launches": n, "flops": F, "bytes": B}} for
    classes with at least one recorded launch."""
    L = lib()
    k = L.tx_profile_classes()
    ms, fl, by = (np.zeros(k) for _ in range(3))
    n = np.zeros(k, dtype=np.int64)
    D = ctypes.POINTER(ctypes.c_double)
    check(L.tx_profile_read(_p(ms, D), _p(n, I64P), _p(fl, D), _p(by, D)))
    return {L.tx_profile_class_name(i).decode(): {"ms": float(ms[i]), "launches": int(n[i]), "flops": float(fl[i]),
                                                  "bytes": float(by[i])} for i in range(k) if n[i] > 0}


def to_device(x: np.ndarray, mc: ModelConfig, device: str = "cuda"):
    """Host float32 array holding stored values -> device tensor of the model dtype."""
    import torch
    return torch.as_tensor(np.ascontiguousarray(x, dtype=np.float32)).to(_torch_dtype(mc)).to(device)
