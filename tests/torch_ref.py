"""An independent reference of the TransX model assembled from PyTorch's own
Transformer layers (fp64, CPU), used to pin the oracle.

torch.nn.TransformerEncoderLayer / TransformerDecoderLayer with norm_first=False,
dropout 0 and activation "gelu" are the textbook post-LN blocks
(self-attention -> [cross-attention ->] FFN, each followed by residual + LN).
The relative-position bias enters through a per-head additive float mask; the
candidate-isolating decoder mask (App. B) through a boolean mask. None of this
code is shared with the oracle: the projections, softmax, LayerNorm and GELU
are PyTorch's. For the local-global sparse cross-attention the decoder's
memory is the last l_local encoded rows plus the pooled global token
(torch.softmax over h_j . w / sqrt(d), then a weighted sum of the rows).
"""
from __future__ import annotations

import numpy as np
import torch

from paper_2607_28940_amd.inputs import ENC_NAMES, DEC_NAMES, ModelConfig


def _t(a) -> torch.Tensor:
    return torch.as_tensor(np.asarray(a, dtype=np.float64))


def _split(m: ModelConfig, weights):
    enc, dec = [], []
    i = 0
    for _ in range(m.n_enc_layers):
        enc.append(dict(zip(ENC_NAMES, weights[i:i + len(ENC_NAMES)])))
        i += len(ENC_NAMES)
    for _ in range(m.n_dec_layers):
        dec.append(dict(zip(DEC_NAMES, weights[i:i + len(DEC_NAMES)])))
        i += len(DEC_NAMES)
    head = (weights[i], weights[i + 1])
    pool = weights[i + 2] if m.global_pool else None
    return enc, dec, head, pool


def _set_mha(mha: torch.nn.MultiheadAttention, Wq, bq, Wk, bk, Wv, bv, Wo, bo):
    # torch computes x A^T + b; our matrices are [d_in, d_out] with y = x W + b
    mha.in_proj_weight.copy_(torch.cat([_t(Wq).T, _t(Wk).T, _t(Wv).T], 0))
    mha.in_proj_bias.copy_(torch.cat([_t(bq), _t(bk), _t(bv)], 0))
    mha.out_proj.weight.copy_(_t(Wo).T)
    mha.out_proj.bias.copy_(_t(bo))


class TorchTransX:
    def __init__(self, m: ModelConfig, weights):
        self.m = m
        enc, dec, head, pool = _split(m, weights)
        self.w_pool = None if pool is None else _t(pool).reshape(-1)
        d, H, F = m.d_model, m.n_heads, m.d_ffn
        kw = dict(dropout=0.0, activation="gelu", batch_first=True, norm_first=False, dtype=torch.float64)
        self.enc_layers = []
        self.rel = []
        with torch.no_grad():
            for p in enc:
                layer = torch.nn.TransformerEncoderLayer(d, H, F, layer_norm_eps=m.ln_eps, **kw).eval()
                _set_mha(layer.self_attn, p["Wq"], p["bq"], p["Wk"], p["bk"], p["Wv"], p["bv"], p["Wo"], p["bo"])
                layer.linear1.weight.copy_(_t(p["W1"]).T)
                layer.linear1.bias.copy_(_t(p["b1"]))
                layer.linear2.weight.copy_(_t(p["W2"]).T)
                layer.linear2.bias.copy_(_t(p["b2"]))
                layer.norm1.weight.copy_(_t(p["ln1_g"]))
                layer.norm1.bias.copy_(_t(p["ln1_b"]))
                layer.norm2.weight.copy_(_t(p["ln2_g"]))
                layer.norm2.bias.copy_(_t(p["ln2_b"]))
                self.enc_layers.append(layer)
                self.rel.append(_t(p["rel"]).reshape(H, m.rel_pos_buckets))
            self.dec_layers = []
            for p in dec:
                layer = torch.nn.TransformerDecoderLayer(d, H, F, layer_norm_eps=m.ln_eps, **kw).eval()
                _set_mha(layer.self_attn, p["sWq"], p["sbq"], p["sWk"], p["sbk"], p["sWv"], p["sbv"], p["sWo"],
                         p["sbo"])
                _set_mha(layer.multihead_attn, p["xWq"], p["xbq"], p["xWk"], p["xbk"], p["xWv"], p["xbv"],
                         p["xWo"], p["xbo"])
                layer.linear1.weight.copy_(_t(p["W1"]).T)
                layer.linear1.bias.copy_(_t(p["b1"]))
                layer.linear2.weight.copy_(_t(p["W2"]).T)
                layer.linear2.bias.copy_(_t(p["b2"]))
                for k, ln in ((1, layer.norm1), (2, layer.norm2), (3, layer.norm3)):
                    ln.weight.copy_(_t(p[f"ln{k}_g"]))
                    ln.bias.copy_(_t(p[f"ln{k}_b"]))
                self.dec_layers.append(layer)
        if m.n_actions:
            self.W_dec = _t(head[0]).reshape(d, m.n_actions)
            self.b_dec = _t(head[1]).reshape(-1)
        else:
            self.w_s = _t(head[0]).reshape(-1)
            self.b_s = float(np.asarray(head[1]).reshape(-1)[0])

    def _enc_mask(self, e: int, L: int) -> torch.Tensor:
        H, R = self.m.n_heads, self.m.rel_pos_buckets
        i = torch.arange(L)[:, None]
        j = torch.arange(L)[None, :]
        mask = torch.full((H, L, L), float("-inf"), dtype=torch.float64)
        allowed = j <= i
        if R > 0:
            dist = torch.clamp(i - j, min=0, max=R - 1)
            bias = self.rel[e][:, dist]  # [H, L, L]
            mask = torch.where(allowed[None], bias, mask)
        else:
            mask = torch.where(allowed[None], torch.zeros_like(mask), mask)
        return mask

    def encode(self, X) -> torch.Tensor:
        # grad mode keeps PyTorch on its plain (non-fused) layer path; its fused
        # inference path does not accept a per-head additive mask
        x = _t(X)[None]
        with torch.enable_grad():
            for e, layer in enumerate(self.enc_layers):
                x = layer(x, src_mask=self._enc_mask(e, x.shape[1]))
        return x[0].detach()

    @staticmethod
    def dec_mask(S: int, C: int) -> torch.Tensor:
        """True = blocked. Serving rows: causal among serving; candidate rows:
        all serving tokens and themselves."""
        N = S + C
        i = torch.arange(N)[:, None]
        j = torch.arange(N)[None, :]
        allowed = torch.where(i < S, j <= i, (j < S) | (j == i))
        return ~allowed

    def score(self, Henc, Xs, Xc) -> np.ndarray:
        S, C = len(Xs), len(Xc)
        d = self.m.d_model
        t = torch.cat([_t(Xs).reshape(S, d), _t(Xc).reshape(C, d)], 0)[None]
        mem = _t(Henc)[None]
        mask = self.dec_mask(S, C)
        with torch.enable_grad():
            for layer in self.dec_layers:
                t = layer(t, mem, tgt_mask=mask)
        z = t[0, S:].detach()
        if self.m.n_actions:
            return torch.softmax(z @ self.W_dec + self.b_dec, dim=-1).numpy()
        return (z @ self.w_s + self.b_s).numpy()

    def memory(self, Henc) -> torch.Tensor:
        """Rows the cross-attention attends to: all encoded rows, or the
        local-global sparse set."""
        Henc = _t(Henc)
        if self.m.l_local <= 0:
            return Henc
        rows = Henc[max(0, Henc.shape[0] - self.m.l_local):]
        if self.w_pool is not None:
            a = torch.softmax(Henc @ self.w_pool / float(np.sqrt(self.m.d_model)), 0)
            rows = torch.cat([rows, (a @ Henc)[None]], 0)
        return rows

    def run_request(self, Xb, Xs, Xc, Xev=None) -> np.ndarray:
        X = Xb if Xev is None else np.concatenate([Xb, Xev], 0)
        return self.score(self.memory(self.encode(X)), Xs, Xc)
