"""Helpers shared by the GPU parity tests: run a workload through the HIP path
(via the C-ABI binding) and through the fp64 oracle, and compare."""
from __future__ import annotations

import sys
from typing import Dict, List, Optional, Sequence

import numpy as np

from paper_2607_28940_amd import inputs as I

FP32_TOL = 1e-4  # relative error bar for the fp32 model: every score
BF16_TOL = 2e-2  # relative error bar for bf16 scores: every score


def check_err(err: Dict[str, float], tol: float):
    """Every compared score within tol (the error of each score is
    |g - o| / max(|o|, rms(o)), see score_err). The 99th percentile is logged
    beside the maximum."""
    assert err["max"] <= tol, err


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def score_err(g, o) -> Dict[str, float]:
    """Per-score error |g - o| / max(|o|, rms(o)) (rms over all compared
    scores): the max and the 99th percentile."""
    g = np.asarray(g, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    rms = float(np.sqrt(np.mean(o * o))) if o.size else 1.0
    e = np.abs(g - o) / np.maximum(np.abs(o), rms)
    return {"max": float(e.max()) if e.size else 0.0, "p99": float(np.percentile(e, 99)) if e.size else 0.0,
            "rms": rms}


def tensor_err(g, o) -> float:
    """max |g - o| / rms(o) for cache tensors (elementwise)."""
    g = np.asarray(g, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    rms = float(np.sqrt(np.mean(o * o)))
    return float(np.abs(g - o).max() / rms)


class DeviceCase:
    """A model and cache for one workload on cuda:0."""

    def __init__(self, wl: I.Workload, weights, max_tokens: Optional[int] = None, extra_pages: int = 0,
                 fill_byte: Optional[int] = None, model_id: int = 1, max_requests: Optional[int] = None):
        import torch
        from paper_2607_28940_amd import transx as T
        self.T = T
        self.torch = torch
        self.wl = wl
        self.m = wl.model
        self.model = T.Model(wl.model, weights, model_id=model_id)
        mt = max_tokens or (max(wl.L) + wl.n_append)
        pages = sum((L + wl.n_append + 63) // 64 for L in wl.L) + extra_pages
        self.cache = T.KVCache(self.model, n_pages=pages, max_requests=max_requests or wl.B, max_tokens=mt,
                               fill_byte=fill_byte)

    def dev(self, x):
        return self.T.to_device(x, self.m)

    def build(self, reqs: Sequence[int], L: Optional[Sequence[int]] = None, ws_limit=None, ids=None):
        X = [I.request_tokens(self.wl, r, I.STREAM_BEHAVIOR) for r in reqs]
        if L is not None:
            X = [x[:l] for x, l in zip(X, L)]
        off = I.offsets([len(x) for x in X])
        self.cache.build(list(reqs) if ids is None else ids, self.dev(np.concatenate(X)), off, ws_limit=ws_limit)

    def append(self, reqs: Sequence[int], lo: int = 0, hi: Optional[int] = None, ws_limit=None):
        E = [I.request_tokens(self.wl, r, I.STREAM_EVENTS)[lo:hi] for r in reqs]
        off = I.offsets([len(e) for e in E])
        self.cache.append(list(reqs), self.dev(np.concatenate(E)), off, ws_limit=ws_limit)

    def score(self, reqs: Sequence[int], cand: Optional[List[np.ndarray]] = None, ws_limit=None, ids=None):
        Xs = [I.request_tokens(self.wl, r, I.STREAM_SERVING) for r in reqs]
        Xc = cand if cand is not None else [I.request_tokens(self.wl, r, I.STREAM_CANDIDATES) for r in reqs]
        so = I.offsets([len(x) for x in Xs])
        co = I.offsets([len(x) for x in Xc])
        d = self.m.d_model
        xs = self.dev(np.concatenate(Xs) if sum(map(len, Xs)) else np.zeros((1, d), np.float32))
        xc = self.dev(np.concatenate(Xc) if sum(map(len, Xc)) else np.zeros((1, d), np.float32))
        out = self.cache.score(list(reqs) if ids is None else ids, xs, so, xc, co, ws_limit=ws_limit)
        self.torch.cuda.synchronize()
        s = out.cpu().numpy().astype(np.float64)
        return [s[co[i]:co[i + 1]] for i in range(len(reqs))]


def oracle_background(orc, wl: I.Workload, reqs: Sequence[int], append: bool = False):
    """Start the oracle on the given requests in a worker thread (the oracle's
    C code runs outside the GIL) while the GPU side proceeds; returns a future
    of the list of their score arrays."""
    from concurrent.futures import ThreadPoolExecutor
    ex = ThreadPoolExecutor(1)
    fut = ex.submit(lambda: [oracle_request(orc, wl, r, append=append)[0] for r in reqs])
    ex.shutdown(wait=False)
    return fut


def oracle_request(orc, wl: I.Workload, r: int, append: bool = False, L: Optional[int] = None, cand=None):
    Xb = I.request_tokens(wl, r, I.STREAM_BEHAVIOR)
    if L is not None:
        Xb = Xb[:L]
    Xs = I.request_tokens(wl, r, I.STREAM_SERVING)
    Xc = cand if cand is not None else I.request_tokens(wl, r, I.STREAM_CANDIDATES)
    Xev = I.request_tokens(wl, r, I.STREAM_EVENTS) if append else None
    return orc.run_request(Xb, Xs, Xc, Xev)
