"""Seeded synthetic inputs and model weights for the TransX serving path.

This module only draws random numbers and rounds them; it holds none of the
method's arithmetic. Both the HIP path (through the binding) and the fp64 CPU
oracle consume exactly the values produced here.

Shapes follow the paper's problem statement: a behavior stream H of L tokens
(Sec. 3, Eq. behavior-stream), a serving event with S serving-event tokens and
C candidate tokens (Sec. 3, Eq. serving-stream), d-dimensional tokens after
tokenization (Sec. 4.1.1 assumes tokenization is given). The paper's own data
(LinkedIn production traffic, Sec. 5.1) is not public; these seeded draws stand
in for it with the configured shapes.

Randomness:
  * tensor i of the canonical weight list is drawn from
    Generator(PCG64(SeedSequence([seed_w, i]))),
  * request r's stream k (0 behavior, 1 serving, 2 candidates, 3 appended
    events) from Generator(PCG64(SeedSequence([seed_x, cfg_id, k, r]))),
  * the ragged shapes from SeedSequence([seed_x, cfg_id, 99]).
so any single request can be regenerated on its own.
"""
from __future__ import annotations

import dataclasses
import math
from concurrent.futures import ThreadPoolExecutor
from typing import List, Optional, Sequence

import numpy as np

SEED_W = 1234
SEED_X = 5678

STREAM_BEHAVIOR = 0
STREAM_SERVING = 1
STREAM_CANDIDATES = 2
STREAM_EVENTS = 3


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    d_model: int
    n_heads: int
    d_ffn: int
    n_enc_layers: int
    n_dec_layers: int
    rel_pos_buckets: int = 128
    ln_eps: float = 1e-5
    dtype: str = "bf16"  # "bf16" or "f32": storage type of inputs, weights, cache, activations
    # local-global sparse cross-attention (Sec. 4.1.2): 0 = every cached token;
    # L > 0 = the last L cached tokens, plus the attention-pooled global token
    # when global_pool is set
    l_local: int = 0
    global_pool: bool = False
    # decoder head (Sec. 4.1.3): 0 = one logit per candidate (the two-action
    # case, linear head w_s, b_s); k >= 2 = softmax over k learned action
    # embeddings (W_dec [d, k], b_dec [k]), k probabilities per candidate
    n_actions: int = 0

    @property
    def d_head(self) -> int:
        return self.d_model // self.n_heads


@dataclasses.dataclass
class Workload:
    name: str
    cfg_id: int
    model: ModelConfig
    L: List[int]
    S: List[int]
    C: List[int]
    n_append: int = 0  # events appended per request after the initial build

    @property
    def B(self) -> int:
        return len(self.L)


# ---------------------------------------------------------------------------
# canonical parameter list
# ---------------------------------------------------------------------------

ENC_NAMES = ["Wq", "bq", "Wk", "bk", "Wv", "bv", "Wo", "bo", "ln1_g", "ln1_b",
             "W1", "b1", "W2", "b2", "ln2_g", "ln2_b", "rel"]
DEC_NAMES = ["sWq", "sbq", "sWk", "sbk", "sWv", "sbv", "sWo", "sbo", "ln1_g", "ln1_b",
             "xWq", "xbq", "xWk", "xbk", "xWv", "xbv", "xWo", "xbo", "ln2_g", "ln2_b",
             "W1", "b1", "W2", "b2", "ln3_g", "ln3_b"]
HEAD_NAMES = ["w_s", "b_s"]


def weight_specs(m: ModelConfig) -> List[tuple]:
    """(layer kind, layer index, name, shape) for every tensor, in canonical order.

    Matrices are stored [d_in, d_out] (a layer computes y = x W + b).
    """
    d, F, H, R = m.d_model, m.d_ffn, m.n_heads, m.rel_pos_buckets
    shapes_enc = {"Wq": (d, d), "Wk": (d, d), "Wv": (d, d), "Wo": (d, d),
                  "W1": (d, F), "W2": (F, d), "b1": (F,), "rel": (H, R)}
    shapes_dec = {"W1": (d, F), "W2": (F, d), "b1": (F,)}
    out = []
    for e in range(m.n_enc_layers):
        for n in ENC_NAMES:
            out.append(("enc", e, n, shapes_enc.get(n, (d,))))
    for l in range(m.n_dec_layers):
        for n in DEC_NAMES:
            shp = shapes_dec.get(n)
            if shp is None:
                shp = (d, d) if n.endswith(("Wq", "Wk", "Wv", "Wo")) else (d,)
            out.append(("dec", l, n, shp))
    if m.n_actions:
        out.append(("head", 0, "W_dec", (d, m.n_actions)))
        out.append(("head", 0, "b_dec", (m.n_actions,)))
    else:
        out.append(("head", 0, "w_s", (d,)))
        out.append(("head", 0, "b_s", (1,)))
    if m.global_pool:
        out.append(("pool", 0, "w_pool", (d,)))
    return out


def n_weights(m: ModelConfig) -> int:
    return 17 * m.n_enc_layers + 26 * m.n_dec_layers + 2 + int(bool(m.global_pool))


def _round_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round fp32 draws to the storage type (bf16: round-to-nearest-even) and
    return the exact stored values as float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "f32":
        return x
    if dtype != "bf16":
        raise ValueError(dtype)
    u = x.view(np.uint32)
    # RNE on the upper 16 bits (inputs are finite normals, no NaN handling needed)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) & 0xFFFF0000).astype(np.uint32)
    return r.view(np.float32)


def make_weights(m: ModelConfig, variant: Sequence[str] = (), seed_w: int = SEED_W) -> List[np.ndarray]:
    """All parameters in canonical order, as float32 arrays holding exactly the
    stored (bf16 or fp32) values.

    Base draws: matrices, biases, the head and the relative-position table are
    N(0, 0.02); LayerNorm gain 1 and offset 0.
    variant "sharp": attention Wq and Wk ~ N(0, (2/sqrt(d))^2) and the
      relative-position table ~ N(0, 1), so attention logits have std of a few
      units and softmax is far from uniform.
    variant "sharp-cross": only the decoder cross-attention's Wq and Wk ~
      N(0, (2/sqrt(d))^2): cross-attention logits of a few units over the
      cached tokens, every other tensor at its base draw.
    variant "affine": LayerNorm gain 1 + N(0, 0.1), offset N(0, 0.1).
    The pooling vector of the global token is N(0, 0.02) (nearly uniform
    pooling), N(0, 16) under "sharp" (pooling logits of a few units); the
    action embeddings W_dec are N(0, (4/sqrt d)^2) under "sharp" or
    "sharp-head" (action logits of a few units; "sharp-head" leaves every
    other tensor at its base draw).
    """
    variant = set(variant)
    d = m.d_model
    out = []
    for i, (kind, layer, name, shape) in enumerate(weight_specs(m)):
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed_w, i])))
        z = rng.standard_normal(shape, dtype=np.float32)
        if name.startswith("ln") and name.endswith("_g"):
            w = 1.0 + (0.1 * z if "affine" in variant else 0.0 * z)
        elif name.startswith("ln") and name.endswith("_b"):
            w = 0.1 * z if "affine" in variant else 0.0 * z
        elif name == "rel":
            w = (1.0 if "sharp" in variant else 0.02) * z
        elif name == "w_pool":
            w = (4.0 if "sharp" in variant else 0.02) * z
        elif name == "W_dec" and ("sharp" in variant or "sharp-head" in variant):
            w = (4.0 / math.sqrt(d)) * z
        elif "sharp" in variant and name in ("Wq", "Wk", "sWq", "sWk", "xWq", "xWk"):
            w = (2.0 / math.sqrt(d)) * z
        elif "sharp-cross" in variant and name in ("xWq", "xWk"):
            w = (2.0 / math.sqrt(d)) * z
        else:
            w = 0.02 * z
        out.append(_round_storage(np.asarray(w, dtype=np.float32), m.dtype))
    return out


def _draw(cfg_id: int, stream: int, r: int, rows: int, d: int, dtype: str, seed_x: int) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed_x, cfg_id, stream, r])))
    return _round_storage(rng.standard_normal((rows, d), dtype=np.float32), dtype)


def request_tokens(wl: Workload, r: int, stream: int, seed_x: int = SEED_X) -> np.ndarray:
    """Tokens of request r for one stream, [rows, d] float32 holding stored values."""
    rows = {STREAM_BEHAVIOR: wl.L[r], STREAM_SERVING: wl.S[r],
            STREAM_CANDIDATES: wl.C[r], STREAM_EVENTS: wl.n_append}[stream]
    return _draw(wl.cfg_id, stream, r, rows, wl.model.d_model, wl.model.dtype, seed_x)


def packed_tokens(wl: Workload, stream: int, requests: Optional[Sequence[int]] = None,
                  seed_x: int = SEED_X, threads: int = 8) -> np.ndarray:
    """Concatenation over requests of request_tokens (the packed layout that the
    offset arrays index)."""
    reqs = list(range(wl.B)) if requests is None else list(requests)
    with ThreadPoolExecutor(max(1, threads)) as ex:
        parts = list(ex.map(lambda r: request_tokens(wl, r, stream, seed_x), reqs))
    if not parts:
        return np.zeros((0, wl.model.d_model), np.float32)
    return np.concatenate(parts, axis=0)


def offsets(counts: Sequence[int]) -> np.ndarray:
    o = np.zeros(len(counts) + 1, dtype=np.int64)
    o[1:] = np.cumsum(np.asarray(counts, dtype=np.int64))
    return o


# ---------------------------------------------------------------------------
# named workloads (cfg ids 1..5)
# ---------------------------------------------------------------------------

def _ragged_shapes(B: int, cfg_id: int, seed_x: int):
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed_x, cfg_id, 99])))
    z = rng.standard_normal(B)
    L = np.clip(np.rint(np.exp(math.log(2048.0) + 1.0 * z)), 128, 16384).astype(int)
    S = rng.integers(1, 64, size=B, endpoint=True)
    C = rng.integers(32, 1024, size=B, endpoint=True)
    return [int(v) for v in L], [int(v) for v in S], [int(v) for v in C]


def workload(name: str, seed_x: int = SEED_X, **override) -> Workload:
    """Named workloads. `override` may replace B (number of requests) or any
    ModelConfig field for test variants; shapes stay those of the named case."""
    B = override.pop("B", None)
    if name == "tiny":
        m = ModelConfig(d_model=64, n_heads=2, d_ffn=256, n_enc_layers=1, n_dec_layers=1, dtype="f32")
        B = B or 1
        wl = Workload(name, 1, m, [256] * B, [8] * B, [16] * B)
    elif name == "uniform":
        m = ModelConfig(d_model=512, n_heads=8, d_ffn=2048, n_enc_layers=2, n_dec_layers=2)
        B = B or 64
        wl = Workload(name, 2, m, [1024] * B, [32] * B, [128] * B)
    elif name == "headline":
        m = ModelConfig(d_model=1024, n_heads=8, d_ffn=4096, n_enc_layers=2, n_dec_layers=2)
        B = B or 256
        wl = Workload(name, 3, m, [4096] * B, [64] * B, [512] * B)
    elif name == "ragged":
        m = ModelConfig(d_model=1024, n_heads=8, d_ffn=4096, n_enc_layers=2, n_dec_layers=2)
        Bfull = 512
        L, S, C = _ragged_shapes(Bfull, 4, seed_x)
        B = B or Bfull
        wl = Workload(name, 4, m, L[:B], S[:B], C[:B])
    elif name == "append":
        m = ModelConfig(d_model=1024, n_heads=8, d_ffn=4096, n_enc_layers=2, n_dec_layers=2)
        B = B or 1024
        wl = Workload(name, 5, m, [8192] * B, [32] * B, [256] * B, n_append=16)
    else:
        raise KeyError(name)
    if override:
        wl.model = dataclasses.replace(wl.model, **override)
    return wl


def custom_workload(model: ModelConfig, L, S, C, n_append: int = 0, cfg_id: int = 100,
                    name: str = "custom") -> Workload:
    """A workload with explicit per-request shapes (test cases)."""
    return Workload(name, cfg_id, model, list(map(int, L)), list(map(int, S)), list(map(int, C)),
                    n_append=int(n_append))
