"""Pins of the oracle's query-key softmax decoder over k action tokens (CPU).

Sec. 4.1.3 (Eq. action-decoding): p(y_c) = softmax(Q_dec k_dec), with k
learned action embeddings and the candidate's key k_dec = f_dec(z_c); the
decoder stack's output row is the key (App. B's Transformer-based head). With
two actions whose embeddings differ by the scalar head w_s, the click
probability is the logistic function of the scalar logit. Pinned by:
  * that reduction (scipy's expit of the dense oracle's scalar scores),
  * rows summing to 1, invariance to a common offset of all actions,
    permutation of the actions permuting the outputs,
  * PyTorch's decoder layers followed by torch.softmax (dense and sparse
    cross-attention),
  * planted mistakes in a copy of ox_actions failing these checks.
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


def _req(wl, r=0):
    return tuple(I.request_tokens(wl, r, k) for k in (I.STREAM_BEHAVIOR, I.STREAM_SERVING, I.STREAM_CANDIDATES))


def _rel(a, b):
    a, b = np.asarray(a), np.asarray(b)
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-300))


def _pins(O, lib_path=None) -> bool:
    wl = I.custom_workload(SMALL, [33], [4], [9], cfg_id=51)
    Xb, Xs, Xc = _req(wl)
    ok = True
    # two actions built from the scalar head: p(click) = expit(logit)
    w1 = I.make_weights(SMALL, ("sharp", "affine"))
    s1, _ = O.Oracle(SMALL, w1, lib_path=lib_path).run_request(Xb, Xs, Xc)
    m2 = dataclasses.replace(SMALL, n_actions=2)
    d = SMALL.d_model
    W2 = np.stack([w1[-2], np.zeros(d, np.float32)], 1)
    w2 = list(w1[:-2]) + [W2, np.array([w1[-1][0], 0.0], np.float32)]
    P2, _ = O.Oracle(m2, w2, lib_path=lib_path).run_request(Xb, Xs, Xc)
    ok &= _rel(P2[:, 0], expit(s1)) < 1e-12 and _rel(P2[:, 1], expit(-s1)) < 1e-12
    # five sharp actions: rows sum to 1; a common offset changes nothing;
    # permuting the actions permutes the probabilities
    m5 = dataclasses.replace(SMALL, n_actions=5)
    w5 = I.make_weights(m5, ("sharp", "affine"))
    orc = O.Oracle(m5, w5, lib_path=lib_path)
    P5, _ = orc.run_request(Xb, Xs, Xc)
    ok &= np.abs(P5.sum(1) - 1).max() < 1e-14
    ok &= float(P5.max()) > 0.5 and float(P5.min()) < 0.05  # far from uniform
    w5b = list(w5[:-1]) + [w5[-1].astype(np.float64) + 3.0]  # exact in fp64
    ok &= _rel(O.Oracle(m5, w5b, lib_path=lib_path).run_request(Xb, Xs, Xc)[0], P5) < 1e-13
    perm = np.array([3, 0, 4, 1, 2])
    w5p = list(w5[:-2]) + [w5[-2][:, perm], w5[-1][perm]]
    ok &= _rel(O.Oracle(m5, w5p, lib_path=lib_path).run_request(Xb, Xs, Xc)[0], P5[:, perm]) < 1e-14
    return bool(ok)


def test_action_decoder_pins(oracle_mod):
    assert _pins(oracle_mod)


CASES = [
    ("dense-k3", dict(n_actions=3)),
    ("dense-k16", dict(n_actions=16)),
    ("sparse-k4", dict(n_actions=4, l_local=6, global_pool=True)),
]


@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_action_decoder_matches_torch(oracle_mod, name, kw):
    from tests.torch_ref import TorchTransX
    m = dataclasses.replace(SMALL, **kw)
    w = I.make_weights(m, ("sharp", "affine"))
    wl = I.custom_workload(m, [27], [5], [7], n_append=4, cfg_id=52)
    Xb, Xs, Xc = _req(wl)
    Xev = I.request_tokens(wl, 0, I.STREAM_EVENTS)
    P, _ = oracle_mod.Oracle(m, w).run_request(Xb, Xs, Xc, Xev)
    R = TorchTransX(m, w).run_request(Xb, Xs, Xc, Xev)
    assert P.shape == (7, m.n_actions)
    assert _rel(P, R) < 1e-12


MUTATIONS = [
    ("embedding matrix read transposed", "s += Z[(size_t)c * d + i] * W[(size_t)i * k + a];",
     "s += Z[(size_t)c * d + i] * W[(size_t)a * d + i];"),
    ("action offset dropped", "    double s = b[a];\n", "    double s = 0.0;\n"),
    ("normaliser misses the last action", "  for (int a = 0; a < k; ++a) den += exp(logit[a] - mx);",
     "  for (int a = 0; a + 1 < k; ++a) den += exp(logit[a] - mx);"),
    ("candidate rows mixed up", "s += Z[(size_t)c * d + i] * W[(size_t)i * k + a];",
     "s += Z[(size_t)((c + 1) % C) * d + i] * W[(size_t)i * k + a];"),
]


@pytest.mark.parametrize("name,find,repl", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_action_mistake_is_caught(oracle_mod, tmp_path, name, find, repl):
    text = open(SRC).read()
    assert text.count(find) == 1, f"mutation anchor not found: {find!r}"
    src = tmp_path / "mut.c"
    src.write_text(text.replace(find, repl, 1))
    lib = oracle_mod.build(src=str(src), out=str(tmp_path / "mut.so"))
    assert not _pins(oracle_mod, lib), f"planted mistake not detected: {name}"
