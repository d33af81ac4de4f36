"""Pins of the oracle's local-global sparse cross-attention (CPU only).

Sec. 4.1.2 restricts each decoder query's cross-attention to the last L_local
cached tokens plus one globally pooled anchor token; the experiments use
attention pooling for that token (Sec. 5 setup). The oracle evaluates the
pooling (ox_pool) and the decoder over the restricted key set. Pinned here by:
  * closed forms of attention pooling: zero pooling vector -> mean of the rows,
    one row -> that row, two rows -> the logistic weight of their logit
    difference (scipy's expit), a common shift of the rows shifts the pooled
    token by the same vector (softmax is shift invariant), a very sharp pooling
    vector selects the best-aligned row, row order does not matter,
  * the reduction to the dense path when L_local covers the whole history and
    there is no pooled token (bitwise),
  * PyTorch's TransformerDecoderLayer given the sparse memory rows (last
    L_local encoded rows + the pooled token) as its cross-attention memory,
  * planted mistakes in a copy of the pooling code fail the closed forms.
"""
import dataclasses
import os

import numpy as np
import pytest
from scipy.special import expit

from paper_2607_28940_amd import inputs as I
from paper_2607_28940_amd.inputs import ModelConfig

SMALL = ModelConfig(d_model=32, n_heads=4, d_ffn=64, n_enc_layers=2, n_dec_layers=2, rel_pos_buckets=8,
                    dtype="f32")
SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "transx_oracle.c")


def _rel(a, b):
    a, b = np.asarray(a), np.asarray(b)
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-300))


def _rows(L, d, seed):
    return np.random.default_rng(seed).standard_normal((L, d))


def _pool_pins(O, lib_path=None):
    """True when every closed form holds for the oracle built at lib_path."""
    orc = O.Oracle(SMALL, I.make_weights(SMALL), lib_path=lib_path)
    d = SMALL.d_model
    H = _rows(9, d, 1)
    w = np.random.default_rng(2).standard_normal(d)
    ok = True
    # zero pooling vector: uniform weights
    ok &= _rel(orc.pool(H, np.zeros(d)), H.mean(0)) < 1e-14
    # a single row pools to itself
    ok &= np.array_equal(orc.pool(H[3:4], w), H[3])
    # two rows: weight of row 0 is the logistic function of the logit difference
    z = H[:2] @ w / np.sqrt(d)
    a0 = expit(z[0] - z[1])
    ok &= _rel(orc.pool(H[:2], w), a0 * H[0] + (1 - a0) * H[1]) < 1e-13
    # a common shift u of all rows moves every logit by u.w/sqrt(d): same weights
    u = np.random.default_rng(3).standard_normal(d)
    ok &= _rel(orc.pool(H + u, w) - u, orc.pool(H, w)) < 1e-12
    # row order is irrelevant
    perm = np.random.default_rng(4).permutation(len(H))
    ok &= _rel(orc.pool(H[perm], w), orc.pool(H, w)) < 1e-14
    # a very sharp pooling vector along row k selects row k
    k = 5
    wk = 1e4 * H[k] / np.linalg.norm(H[k])
    if np.argmax(H @ wk) == k:
        ok &= _rel(orc.pool(H, wk), H[k]) < 1e-9
    return bool(ok)


def test_pool_closed_forms(oracle_mod):
    assert _pool_pins(oracle_mod)


def test_sparse_without_pool_covering_history_is_dense(oracle_mod):
    """L_local >= L and no pooled token: the key set is the whole cache."""
    w = I.make_weights(SMALL, ("sharp", "affine"))
    wl = I.custom_workload(SMALL, [30], [4], [6], cfg_id=31)
    Xb, Xs, Xc = (I.request_tokens(wl, 0, k) for k in (I.STREAM_BEHAVIOR, I.STREAM_SERVING, I.STREAM_CANDIDATES))
    dense, _ = oracle_mod.Oracle(SMALL, w).run_request(Xb, Xs, Xc)
    m2 = dataclasses.replace(SMALL, l_local=64, global_pool=False)
    sparse, _ = oracle_mod.Oracle(m2, w).run_request(Xb, Xs, Xc)
    assert np.array_equal(dense, sparse)
    # a shorter window changes the scores (the restriction is not a no-op)
    m3 = dataclasses.replace(SMALL, l_local=5, global_pool=False)
    assert _rel(oracle_mod.Oracle(m3, w).run_request(Xb, Xs, Xc)[0], dense) > 1e-3


CASES = [
    ("L5-pool", 5, True, 40, 5, 7, 0),
    ("L10-pool-append", 10, True, 23, 4, 6, 9),
    ("L3-nopool", 3, False, 17, 3, 5, 0),
    ("history-shorter-than-window", 10, True, 6, 2, 4, 0),
    ("S0", 4, True, 20, 0, 5, 0),
    ("L64-pool-append", 64, True, 150, 3, 4, 5),
]


@pytest.mark.parametrize("name,l_local,pool,L,S,C,n_app", CASES, ids=[c[0] for c in CASES])
def test_sparse_matches_torch_decoder(oracle_mod, name, l_local, pool, L, S, C, n_app):
    from tests.torch_ref import TorchTransX
    m = dataclasses.replace(SMALL, l_local=l_local, global_pool=pool)
    w = I.make_weights(m, ("sharp", "affine"))
    wl = I.custom_workload(m, [L], [S], [C], n_append=n_app, cfg_id=32)
    Xb, Xs, Xc = (I.request_tokens(wl, 0, k) for k in (I.STREAM_BEHAVIOR, I.STREAM_SERVING, I.STREAM_CANDIDATES))
    Xev = I.request_tokens(wl, 0, I.STREAM_EVENTS) if n_app else None
    s, st = oracle_mod.Oracle(m, w).run_request(Xb, Xs, Xc, Xev)
    r = TorchTransX(m, w).run_request(Xb, Xs, Xc, Xev)
    assert _rel(s, r) < 1e-12
    assert np.std(r) > 1e-3
    # the pooled token is far from uniform pooling under the sharp variant
    if pool:
        orc = oracle_mod.Oracle(m, w)
        assert _rel(orc.pool(st["H"]), st["H"].mean(0)) > 1e-2


POOL_MUTATIONS = [
    ("logit scale dropped", "    z[j] = s / sqrt((double)d);\n", "    z[j] = s;\n"),
    ("normaliser misses the first row", "  for (int j = 0; j < L; ++j) den += exp(z[j] - mx);",
     "  for (int j = 1; j < L; ++j) den += exp(z[j] - mx);"),
    ("rows weighted by the next row's weight",
     "    const double a = exp(z[j] - mx) / den;", "    const double a = exp(z[(j + 1) % L] - mx) / den;"),
    ("max not subtracted in the weights", "    const double a = exp(z[j] - mx) / den;",
     "    const double a = exp(z[j]) / den;"),
]


@pytest.mark.parametrize("name,find,repl", POOL_MUTATIONS, ids=[m[0] for m in POOL_MUTATIONS])
def test_planted_pool_mistake_is_caught(oracle_mod, tmp_path, name, find, repl):
    text = open(SRC).read()
    assert text.count(find) == 1, f"mutation anchor not found: {find!r}"
    src = tmp_path / "mut.c"
    src.write_text(text.replace(find, repl, 1))
    lib = oracle_mod.build(src=str(src), out=str(tmp_path / "mut.so"))
    assert not _pool_pins(oracle_mod, lib), f"planted mistake not detected: {name}"
