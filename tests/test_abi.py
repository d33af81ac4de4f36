"""C-ABI library checks that need no GPU: it loads, exports every function the
header declares, and its host-side validation and page bookkeeping return the
documented status codes before anything is launched."""
import ctypes
import subprocess

import numpy as np
import pytest

from paper_2607_28940_amd import inputs as I
from paper_2607_28940_amd import transx as T

# Host-only fake device addresses: the calls below validate and book-keep on
# the host and never dereference them.
FAKE_REPACK = 0x7F0000000000
FAKE_POOL = 0x7E0000000000


@pytest.fixture(scope="module")
def L():
    return T.lib()


def test_exports_every_declared_function(L):
    names = T.header_functions()
    assert {"kv_cache_build", "kv_cache_append", "score_candidates"} <= set(names)
    out = subprocess.run(["nm", "-D", "--defined-only", T.LIB_PATH], capture_output=True, text=True, check=True).stdout
    exported = {ln.split()[-1] for ln in out.splitlines() if ln.strip()}
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    for n in names:
        getattr(L, n)
    # nothing but the ABI leaks out of the library
    extra = sorted(e for e in exported if not e.startswith("_") and e not in names)
    assert not extra, extra


def _cfg(**kw):
    m = I.workload("headline").model
    return T.Config.of(m) if not kw else T.Config.of(I.ModelConfig(**{**m.__dict__, **kw}))


def test_counts_and_sizes(L):
    for name in ("tiny", "uniform", "headline"):
        m = I.workload(name).model
        c = T.Config.of(m)
        assert L.tx_num_weights(ctypes.byref(c)) == I.n_weights(m)
        es = 2 if m.dtype == "bf16" else 4
        assert L.tx_kv_page_bytes(ctypes.byref(c)) == (m.n_enc_layers + m.n_dec_layers) * 2 * 64 * m.d_model * es
        assert L.tx_model_repack_bytes(ctypes.byref(c)) > 0
    c = _cfg()
    assert L.tx_kv_pool_bytes(ctypes.byref(c), 10, 4, 1000) >= 10 * L.tx_kv_page_bytes(ctypes.byref(c)) + 4 * 16 * 4


def test_sparse_config_counts_and_errors(L):
    """Local-global sparse cross-attention: one more weight tensor (the pooling
    vector) and per-request global-token records in the pool; invalid or
    unsupported windows are rejected."""
    base = _cfg()
    for kw in (dict(l_local=10, global_pool=True), dict(l_local=10, global_pool=False)):
        m = I.ModelConfig(**{**I.workload("headline").model.__dict__, **kw})
        c = T.Config.of(m)
        assert L.tx_num_weights(ctypes.byref(c)) == I.n_weights(m)
    c = _cfg(l_local=10, global_pool=True)
    d, n_dec, req = 1024, 2, 4
    extra = L.tx_kv_pool_bytes(ctypes.byref(c), 10, req, 1000) - L.tx_kv_pool_bytes(ctypes.byref(base), 10, req, 1000)
    assert extra >= req * (2 * 4 + d * 4 + 2 * n_dec * d * 2)
    assert L.tx_kv_pool_bytes(ctypes.byref(_cfg(l_local=10)), 10, req, 1000) == \
        L.tx_kv_pool_bytes(ctypes.byref(base), 10, req, 1000)
    h = T.VP()
    for kw, code in ((dict(l_local=-1), T.TX_E_INVALID), (dict(l_local=65), T.TX_E_UNSUPPORTED),
                     (dict(l_local=0, global_pool=True), T.TX_E_INVALID)):
        bad = _cfg(**kw)
        assert L.tx_model_create(ctypes.byref(bad), T.VP(FAKE_REPACK), 1 << 30, 1, ctypes.byref(h)) == code, kw
    bad = _cfg(l_local=4)
    bad.global_pool = 2
    assert L.tx_model_create(ctypes.byref(bad), T.VP(FAKE_REPACK), 1 << 30, 1, ctypes.byref(h)) == T.TX_E_INVALID
    m = _model(L, _cfg(l_local=64, global_pool=True))
    L.tx_model_destroy(m)


def test_action_head_config(L):
    for k in (2, 3, 16):
        m = I.ModelConfig(**{**I.workload("headline").model.__dict__, "n_actions": k})
        c = T.Config.of(m)
        assert L.tx_num_weights(ctypes.byref(c)) == I.n_weights(m)
        assert L.tx_model_repack_bytes(ctypes.byref(c)) > L.tx_model_repack_bytes(ctypes.byref(_cfg()))
    h = T.VP()
    for k, code in ((1, T.TX_E_INVALID), (-2, T.TX_E_INVALID), (17, T.TX_E_UNSUPPORTED)):
        bad = _cfg(n_actions=k)
        assert L.tx_model_create(ctypes.byref(bad), T.VP(FAKE_REPACK), 1 << 30, 1, ctypes.byref(h)) == code, k


def _model(L, cfg):
    h = T.VP()
    rc = L.tx_model_create(ctypes.byref(cfg), T.VP(FAKE_REPACK), L.tx_model_repack_bytes(ctypes.byref(cfg)), 7,
                           ctypes.byref(h))
    assert rc == T.TX_OK, L.tx_last_error()
    return h


def test_model_create_errors(L):
    h = T.VP()
    bad = _cfg(n_heads=16, d_model=768)  # d_head 48
    assert L.tx_model_create(ctypes.byref(bad), T.VP(FAKE_REPACK), 1 << 30, 1, ctypes.byref(h)) == T.TX_E_UNSUPPORTED
    assert b"d_head" in L.tx_last_error()
    bad = _cfg(d_model=1000, n_heads=3)  # not a multiple
    assert L.tx_model_create(ctypes.byref(bad), T.VP(FAKE_REPACK), 1 << 30, 1, ctypes.byref(h)) == T.TX_E_INVALID
    c = _cfg()
    need = L.tx_model_repack_bytes(ctypes.byref(c))
    assert L.tx_model_create(ctypes.byref(c), T.VP(FAKE_REPACK + 8), need, 1, ctypes.byref(h)) == T.TX_E_INVALID
    assert L.tx_model_create(ctypes.byref(c), T.VP(FAKE_REPACK), need - 1, 1, ctypes.byref(h)) == T.TX_E_NOMEM
    m = _model(L, c)
    ptrs = (T.VP * 3)()
    assert L.tx_model_set_weights(m, ptrs, 3, None) == T.TX_E_INVALID
    L.tx_model_destroy(m)


class Host:
    """A model and cache whose device buffers are never touched."""

    def __init__(self, L, n_pages=40, max_req=6, max_tokens=1000):
        self.L = L
        self.cfg = _cfg()
        self.m = _model(L, self.cfg)
        self.pool_bytes = L.tx_kv_pool_bytes(ctypes.byref(self.cfg), n_pages, max_req, max_tokens)
        h = T.VP()
        rc = L.tx_kv_cache_create(self.m, T.VP(FAKE_POOL), self.pool_bytes, n_pages, max_req, max_tokens,
                                  ctypes.byref(h))
        assert rc == T.TX_OK, L.tx_last_error()
        self.c = h

    def close(self):
        self.L.tx_kv_cache_destroy(self.c)
        self.L.tx_model_destroy(self.m)

    def build(self, ids, off, ws_bytes=1 << 40):
        ids, off = T._i32(ids), T._i64(off)
        return self.L.kv_cache_build(self.c, len(ids), T._p(ids, T.I32P), T.VP(0x7D0000000000), T._p(off, T.I64P),
                                     T.VP(0x7C0000000000), ws_bytes, None)

    def append(self, ids, off):
        ids, off = T._i32(ids), T._i64(off)
        return self.L.kv_cache_append(self.c, len(ids), T._p(ids, T.I32P), T.VP(0x7D0000000000), T._p(off, T.I64P),
                                      T.VP(0x7C0000000000), 1 << 40, None)

    def score(self, ids, so, co, ws_bytes=1 << 40):
        ids, so, co = T._i32(ids), T._i64(so), T._i64(co)
        return self.L.score_candidates(self.c, len(ids), T._p(ids, T.I32P), T.VP(0x7D0000000000), T._p(so, T.I64P),
                                       T.VP(0x7B0000000000), T._p(co, T.I64P), T.VP(0x7A0000000000),
                                       T.VP(0x7C0000000000), ws_bytes, None)

    def length(self, i):
        v = ctypes.c_int64()
        assert self.L.tx_kv_cache_length(self.c, i, ctypes.byref(v)) == T.TX_OK
        return v.value


def test_cache_bookkeeping_and_errors(L):
    h = Host(L)
    try:
        assert L.tx_kv_cache_free_pages(h.c) == 40
        assert L.tx_kv_cache_model_id(h.c) == 7
        assert h.length(3) == -1
        # invalid ids / offsets
        assert h.build([0, 0], [0, 10, 20]) == T.TX_E_INVALID and b"repeated" in L.tx_last_error()
        assert h.build([6], [0, 10]) == T.TX_E_INVALID
        assert h.build([-1], [0, 10]) == T.TX_E_INVALID
        assert h.build([1, 2], [0, 10, 5]) == T.TX_E_INVALID
        assert h.build([1], [0, 0]) == T.TX_E_INVALID           # L < 1
        assert h.build([1], [0, 1001]) == T.TX_E_INVALID        # L > max_tokens
        # pool exhaustion is reported before anything changes
        assert h.build([1, 2, 3], [0, 1000, 2000, 3000]) == T.TX_E_NOMEM and b"exhausted" in L.tx_last_error()
        assert L.tx_kv_cache_free_pages(h.c) == 40 and h.length(1) == -1
        # cold start: no cache
        assert h.score([2], [0, 3], [0, 5]) == T.TX_E_NOCACHE
        assert h.append([2], [0, 4]) == T.TX_E_NOCACHE
        # workspace too small for one request
        assert h.build([1], [0, 500], ws_bytes=1024) == T.TX_E_NOMEM
        # with valid arguments the call gets as far as the weights check
        assert h.build([1], [0, 500]) == T.TX_E_INVALID and b"weights" in L.tx_last_error()
        assert L.tx_kv_cache_free_pages(h.c) == 40
        # release of unknown / out of range ids
        ids = T._i32([0, 5])
        assert L.tx_kv_cache_release(h.c, 2, T._p(ids, T.I32P)) == T.TX_OK
        ids = T._i32([9])
        assert L.tx_kv_cache_release(h.c, 1, T._p(ids, T.I32P)) == T.TX_E_INVALID
        # C = 0 everywhere and n_req = 0 are no-ops
        assert h.build([], [0]) == T.TX_OK
        assert h.score([], [0], [0]) == T.TX_OK
    finally:
        h.close()


def test_workspace_sizes(L):
    h = Host(L)
    try:
        so, co = T._i64([0, 64, 128]), T._i64([0, 512, 1024])
        full = L.tx_workspace_bytes(h.c, T.TX_OP_SCORE, 2, T._p(so, T.I64P), T._p(co, T.I64P))
        one = L.tx_workspace_min_bytes(h.c, T.TX_OP_SCORE, 2, T._p(so, T.I64P), T._p(co, T.I64P))
        assert 0 < one < full
        # rows x (7 d + F) activations in bf16 dominate
        assert full >= 2 * 576 * (7 * 1024 + 4096) * 2
    finally:
        h.close()
