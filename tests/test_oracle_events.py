"""Pins of the oracle's event-sliced forward (CPU only).

Sec. 4.2 (single-pass seq-to-seq training): the behavior stream is encoded
once, and every serving event decodes against its own prefix of the encoded
stream, sliced rather than re-encoded, which the causal encoder makes exact.
Pinned by: equality (bitwise) with encoding each event's prefix on its own,
PyTorch's encoder/decoder layers run per event on the prefix, and the
staircase being real (an event's scores depend on its prefix length).
"""
import dataclasses

import numpy as np
import pytest

from paper_2607_28940_amd import inputs as I
from paper_2607_28940_amd.inputs import ModelConfig

SMALL = ModelConfig(d_model=32, n_heads=4, d_ffn=64, n_enc_layers=2, n_dec_layers=2, rel_pos_buckets=8,
                    dtype="f32")


def _events(m, L, prefixes, S, C, cfg_id):
    wl = I.custom_workload(m, [L] + [1] * len(prefixes), [0] + S, [1] + C, cfg_id=cfg_id)
    Xb = I.request_tokens(wl, 0, I.STREAM_BEHAVIOR)
    ev = [(p, I.request_tokens(wl, 1 + t, I.STREAM_SERVING), I.request_tokens(wl, 1 + t, I.STREAM_CANDIDATES))
          for t, p in enumerate(prefixes)]
    return Xb, ev


CASES = [("dense", {}), ("sparse-local", dict(l_local=5)), ("actions", dict(n_actions=3))]


@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_event_slices_equal_prefix_encodings(oracle_mod, name, kw):
    from tests.torch_ref import TorchTransX
    m = dataclasses.replace(SMALL, **kw)
    w = I.make_weights(m, ("sharp", "affine"))
    Xb, ev = _events(m, 40, [1, 7, 23, 40], [3, 0, 5, 2], [4, 2, 6, 3], cfg_id=71)
    orc = oracle_mod.Oracle(m, w)
    got = orc.run_events(Xb, ev)
    ref = TorchTransX(m, w)
    for (p, Xs, Xc), g in zip(ev, got):
        alone, _ = orc.run_request(Xb[:p], Xs, Xc)
        assert np.array_equal(g, alone), p
        r = ref.run_request(Xb[:p], Xs, Xc)
        assert np.abs(g - r).max() <= 1e-12 * max(np.abs(r).max(), 1e-300), p


def test_staircase_is_not_a_noop(oracle_mod):
    w = I.make_weights(SMALL, ("sharp", "affine"))
    Xb, ev = _events(SMALL, 40, [10, 40], [3, 3], [4, 4], cfg_id=72)
    _, Xs, Xc = ev[0]
    a, b = oracle_mod.Oracle(SMALL, w).run_events(Xb, [(10, Xs, Xc), (40, Xs, Xc)])
    assert np.abs(a - b).max() > 1e-3
