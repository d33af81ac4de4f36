"""ctypes front end of the fp64 CPU oracle (oracle/transx_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by tests/, by the package smoke check and by
the benchmark's CPU-baseline leg, never by the product path.

`build()` compiles the C source with gcc; `Oracle` holds one model's weights
as float64 and exposes the oracle's stages (full encode, incremental append,
cross-attention K/V, decoder + head).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "transx_oracle.c")
_LIB = os.path.join(_HERE, "libtransx_oracle.so")


def build(verbose: bool = False, src: str = _SRC, out: str = _LIB) -> str:
    """Compile the oracle (plain C, fp64, OpenMP). Always recompiles."""
    tmp = out + ".tmp"
    cmd = ["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off",
           "-o", tmp, src, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


class _Cfg(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int), ("H", ctypes.c_int), ("F", ctypes.c_int), ("n_enc", ctypes.c_int),
                ("n_dec", ctypes.c_int), ("R", ctypes.c_int), ("eps", ctypes.c_double)]


_libs = {}


def _load(path: Optional[str] = None):
    path = path or _LIB
    if path not in _libs:
        if path == _LIB and not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(path)
        P = ctypes.POINTER
        dp = P(ctypes.c_double)
        wp = P(dp)
        lib.ox_n_weights.argtypes = [P(_Cfg)]
        lib.ox_n_weights.restype = ctypes.c_int
        lib.ox_encode.argtypes = [P(_Cfg), wp, dp, ctypes.c_int, dp, dp, dp, dp]
        lib.ox_encode_append.argtypes = [P(_Cfg), wp, dp, dp, ctypes.c_int, dp, ctypes.c_int, dp, dp, dp]
        lib.ox_cross_kv.argtypes = [P(_Cfg), wp, dp, ctypes.c_int, dp, dp]
        lib.ox_score.argtypes = [P(_Cfg), wp, dp, dp, ctypes.c_int, dp, ctypes.c_int, dp, ctypes.c_int, dp, dp, dp]
        lib.ox_pool.argtypes = [ctypes.c_int, dp, ctypes.c_int, dp, dp]
        lib.ox_actions.argtypes = [ctypes.c_int, ctypes.c_int, dp, ctypes.c_int, dp, dp, dp]
        for f in ("ox_encode", "ox_encode_append", "ox_cross_kv", "ox_score", "ox_pool", "ox_actions"):
            getattr(lib, f).restype = None
        _libs[path] = lib
    return _libs[path]


def _dp(a: Optional[np.ndarray]):
    if a is None:
        return ctypes.POINTER(ctypes.c_double)()
    assert a.dtype == np.float64 and a.flags.c_contiguous
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


class Oracle:
    """One model (config + weights in canonical order) evaluated in fp64.

    A model with local-global sparse cross-attention (model.l_local > 0) has
    one more tensor at the end of the list when model.global_pool is set: the
    pooling vector w_pool [d]."""

    def __init__(self, model, weights: Sequence[np.ndarray], lib_path: Optional[str] = None):
        self.model = model
        self.lib = _load(lib_path)
        self.cfg = _Cfg(model.d_model, model.n_heads, model.d_ffn, model.n_enc_layers, model.n_dec_layers,
                        model.rel_pos_buckets, float(model.ln_eps))
        n = self.lib.ox_n_weights(ctypes.byref(self.cfg))
        self.l_local = int(getattr(model, "l_local", 0))
        has_pool = bool(getattr(model, "global_pool", False))
        if n + has_pool != len(weights):
            raise ValueError(f"oracle expects {n + has_pool} tensors, got {len(weights)}")
        self.w_pool = _f64(weights[n]).reshape(-1) if has_pool else None
        self._w = [_f64(w).reshape(-1) if np.asarray(w).size else np.zeros(1) for w in weights[:n]]
        self._wp = (ctypes.POINTER(ctypes.c_double) * n)(*[_dp(w) for w in self._w])

    @property
    def d(self) -> int:
        return self.model.d_model

    def encode(self, X) -> Tuple[np.ndarray, np.ndarray, np.ndarray, float]:
        """Full causal encoding of [L, d] tokens -> (H_enc [L,d], K_enc, V_enc
        [n_enc, L, d], max |softmax row sum - 1|)."""
        X = _f64(X)
        L = X.shape[0]
        H = np.empty((L, self.d))
        K = np.empty((self.model.n_enc_layers, L, self.d))
        V = np.empty_like(K)
        err = np.zeros(1)
        self.lib.ox_encode(ctypes.byref(self.cfg), self._wp, _dp(X), L, _dp(H), _dp(K), _dp(V), _dp(err))
        return H, K, V, float(err[0])

    def encode_append(self, Kpre, Vpre, Xnew) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
        """Encode n new tokens after a cached prefix given its per-layer K/V
        [n_enc, len, d] -> (H_new [n,d], K_new, V_new [n_enc, n, d])."""
        Kpre, Vpre, Xnew = _f64(Kpre), _f64(Vpre), _f64(Xnew)
        ln, n = Kpre.shape[1], Xnew.shape[0]
        H = np.empty((n, self.d))
        K = np.empty((self.model.n_enc_layers, n, self.d))
        V = np.empty_like(K)
        self.lib.ox_encode_append(ctypes.byref(self.cfg), self._wp, _dp(Kpre), _dp(Vpre), ln, _dp(Xnew), n, _dp(H),
                                  _dp(K), _dp(V))
        return H, K, V

    def cross_kv(self, Henc) -> Tuple[np.ndarray, np.ndarray]:
        """Cross-attention K/V of every decoder layer: [n_dec, L, d] each."""
        Henc = _f64(Henc)
        L = Henc.shape[0]
        K = np.empty((self.model.n_dec_layers, L, self.d))
        V = np.empty_like(K)
        self.lib.ox_cross_kv(ctypes.byref(self.cfg), self._wp, _dp(Henc), L, _dp(K), _dp(V))
        return K, V

    @property
    def n_actions(self) -> int:
        return int(getattr(self.model, "n_actions", 0))

    def actions(self, Z) -> np.ndarray:
        """Query-key softmax over the model's k action tokens for decoder
        outputs Z [C, d] -> probabilities [C, k]."""
        Z = _f64(Z)
        k = self.n_actions
        n = len(self._w)
        W, b = self._w[n - 2], self._w[n - 1]
        P = np.empty((Z.shape[0], k))
        self.lib.ox_actions(self.d, k, _dp(Z), Z.shape[0], _dp(W), _dp(b), _dp(P))
        return P

    def score(self, Kx, Vx, Xs, Xc, trace: bool = False):
        """Decoder + head. Returns scores [C] (the candidate logit) or, for a
        model with k action tokens, probabilities [C, k]; with trace=True also
        the per-layer sublayer outputs [n_dec, 3, S+C, d] and the max softmax
        row-sum deviation."""
        Kx, Vx, Xs, Xc = _f64(Kx), _f64(Vx), _f64(Xs), _f64(Xc)
        L = Kx.shape[1]
        S, C = Xs.shape[0], Xc.shape[0]
        out = np.empty(C)
        want_z = self.n_actions > 0
        tr = np.empty((self.model.n_dec_layers, 3, S + C, self.d)) if (trace or want_z) else None
        err = np.zeros(1)
        self.lib.ox_score(ctypes.byref(self.cfg), self._wp, _dp(Kx), _dp(Vx), L, _dp(Xs), S, _dp(Xc), C, _dp(out),
                          _dp(tr), _dp(err))
        if want_z:  # the scalar head output is meaningless here: apply the action decoder
            out = self.actions(tr[-1, 2, S:])
        if trace:
            return out, tr, float(err[0])
        return out

    def pool(self, Henc, w=None) -> np.ndarray:
        """Attention-pooled global token of the encoded rows [L, d] -> [d]
        (the model's pooling vector unless w is given)."""
        Henc = _f64(Henc)
        w = self.w_pool if w is None else _f64(w).reshape(-1)
        g = np.empty(self.d)
        self.lib.ox_pool(self.d, _dp(Henc), Henc.shape[0], _dp(w), _dp(g))
        return g

    def key_rows(self, Henc) -> np.ndarray:
        """Encoded rows the decoder's cross-attention sees (Sec. 4.1.2): all of
        them for dense cross-attention; for the local-global sparse form the
        last l_local rows, followed by the pooled global token when the model
        has one."""
        Henc = _f64(Henc)
        if self.l_local <= 0:
            return Henc
        rows = Henc[max(0, Henc.shape[0] - self.l_local):]
        if self.w_pool is not None:
            rows = np.concatenate([rows, self.pool(Henc)[None, :]], 0)
        return rows

    def run_events(self, Xb, events):
        """Event-sliced forward of one user (Sec. 4.2, single-pass seq-to-seq
        training; causal attention and prefix reuse): the behavior stream is
        encoded once, and serving event t = (p_t, Xs_t, Xc_t) is decoded
        against the cross K/V of the first p_t encoded rows only (its prefix
        H_<t). Returns the list of per-event scores."""
        H, _, _, _ = self.encode(Xb)
        out = []
        for p, Xs, Xc in events:
            Kx, Vx = self.cross_kv(self.key_rows(H[:p]))
            out.append(self.score(Kx, Vx, Xs, Xc))
        return out

    def run_request(self, Xb, Xs, Xc, Xev=None):
        """Whole path for one request: encode behavior (then append events if
        given), project cross K/V of the rows the cross-attention sees, decode,
        score. Returns (scores, state dict)."""
        H, K, V, _ = self.encode(Xb)
        if Xev is not None and len(Xev):
            Hn, Kn, Vn = self.encode_append(K, V, Xev)
            H = np.concatenate([H, Hn], 0)
            K = np.concatenate([K, Kn], 1)
            V = np.concatenate([V, Vn], 1)
        Kx, Vx = self.cross_kv(self.key_rows(H))
        s = self.score(Kx, Vx, Xs, Xc)
        return s, {"H": H, "K": K, "V": V, "Kx": Kx, "Vx": Vx}
