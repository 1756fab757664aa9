"""Float64 reference of the encoder forward (test infrastructure; see package docstring).

Readings taken where the paper is silent (it names the model in Section VIII-B
and the masked-attention / MaskKind primitive in Section III-A, but gives no
layer formulas):

* layer structure: post-LN BERT.  X1 = LN(X + Attn(X)), X' = LN(X1 + FFN(X1)),
  no dropout (inference).
* attention scale 1/sqrt(head_dim).
* MaskKind.Custom is a key mask [B,S] (1 = visible); masked keys are excluded
  (their weight is exactly 0).  A query that sees no key outputs 0.
  Causal: key j visible to query i iff j <= i.  SlidingWindow(w): iff
  i - w < j <= i.  An optional key mask further restricts any kind.
* positions 0..S-1 on every row, token type 0, padded ids 0.
* LayerNorm: biased variance, (x - mean) / sqrt(var + eps) * gamma + beta.
* GELU: 0.5 x (1 + erf(x / sqrt(2))), no tanh approximation.
* pooling: mean over valid tokens (denominator clamped at 1e-9), then
  x / max(||x||_2, 1e-12).
* linear weights use the nn.Linear convention: W is [out, in], y = x W^T + b.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf

from .quant import dequant_int4, dequant_int8

MASK_NONE, MASK_CAUSAL, MASK_SLIDING_WINDOW, MASK_CUSTOM = 0, 1, 2, 3


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def layer_norm(x, gamma, beta, eps):
    """LayerNorm over the last axis, two passes in float64."""
    x = _f64(x)
    mu = x.mean(axis=-1, keepdims=True)
    xc = x - mu
    var = (xc * xc).mean(axis=-1, keepdims=True)
    return xc / np.sqrt(var + eps) * _f64(gamma) + _f64(beta)


def gelu(x):
    """Exact (erf) GELU."""
    x = _f64(x)
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def linear(x, w, b=None):
    """y = x W^T + b with W stored [out, in]."""
    y = _f64(x) @ _f64(w).T
    if b is not None:
        y = y + _f64(b)
    return y


def visible_keys(S, kind, key_mask_row=None, window=0):
    """Boolean [S_q, S_k] matrix: entry (i, j) says whether query i may attend key j."""
    i = np.arange(S)[:, None]
    j = np.arange(S)[None, :]
    if kind == MASK_NONE or kind == MASK_CUSTOM:
        vis = np.ones((S, S), dtype=bool)
    elif kind == MASK_CAUSAL:
        vis = j <= i
    elif kind == MASK_SLIDING_WINDOW:
        vis = (j <= i) & (j > i - window)
    else:
        raise ValueError(f"unknown mask kind {kind}")
    if kind == MASK_CUSTOM and key_mask_row is None:
        raise ValueError("custom mask kind needs a key mask")
    if key_mask_row is not None:
        vis = vis & (np.asarray(key_mask_row)[None, :] != 0)
    return vis


def attention_probs(q, k, vis, scale):
    """Softmax over visible keys of scale * q k^T for one (sequence, head).

    q, k: [S, d]; vis: [S, S] bool.  Rows without a visible key are all zero.
    """
    s = scale * (_f64(q) @ _f64(k).T)
    p = np.zeros_like(s)
    for i in range(s.shape[0]):
        cols = np.nonzero(vis[i])[0]
        if cols.size == 0:
            continue
        row = s[i, cols]
        e = np.exp(row - row.max())
        p[i, cols] = e / e.sum()
    return p


def masked_attention(q, k, v, kind=MASK_CUSTOM, key_mask=None, window=0, scale=None):
    """Multi-head masked attention.

    q, k, v: [B, S, nh, d] (heads already split); key_mask: [B, S] or None.
    Returns [B, S, nh, d].  Loops over (sequence, head) and applies the mask
    by excluding keys.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, S, nh, d = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = np.zeros_like(q)
    for b in range(B):
        vis = visible_keys(S, kind, None if key_mask is None else key_mask[b], window)
        for h in range(nh):
            p = attention_probs(q[b, :, h], k[b, :, h], vis, scale)
            out[b, :, h] = p @ v[b, :, h]
    return out


def embed(ids, word, pos, typ, gamma, beta, eps):
    """x0[b,s] = LN(word[ids[b,s]] + pos[s] + type[0])."""
    ids = np.asarray(ids)
    B, S = ids.shape
    x = _f64(word)[ids] + _f64(pos)[np.arange(S)][None, :, :] + _f64(typ)[0][None, None, :]
    return layer_norm(x, gamma, beta, eps)


def encoder_layer(x, mask, lw, heads, eps):
    """One post-LN encoder layer on [B, S, H] hidden states."""
    x = _f64(x)
    B, S, H = x.shape
    d = H // heads
    qkv = linear(x, lw["wqkv"], lw["bqkv"])
    q = qkv[..., 0:H].reshape(B, S, heads, d)
    k = qkv[..., H:2 * H].reshape(B, S, heads, d)
    v = qkv[..., 2 * H:3 * H].reshape(B, S, heads, d)
    ctx = masked_attention(q, k, v, MASK_CUSTOM, mask, 0, 1.0 / math.sqrt(d)).reshape(B, S, H)
    x1 = layer_norm(linear(ctx, lw["wo"], lw["bo"]) + x, lw["ln1_g"], lw["ln1_b"], eps)
    g = gelu(linear(x1, lw["w1"], lw["b1"]))
    return layer_norm(linear(g, lw["w2"], lw["b2"]) + x1, lw["ln2_g"], lw["ln2_b"], eps)


def mean_pool_l2(x, mask):
    """Masked mean over tokens, then L2 normalisation; [B, S, H] -> [B, H]."""
    x = _f64(x)
    m = _f64(mask)[:, :, None]
    e = (x * m).sum(axis=1) / np.maximum(m.sum(axis=1), 1e-9)
    n = np.sqrt((e * e).sum(axis=1, keepdims=True))
    return e / np.maximum(n, 1e-12)


def layer_weights(wl, layer):
    """The float64-ready weights of one layer; on quantised workloads the linear
    weights are the oracle's own dequantisation of the stored codes."""
    lw = dict(wl.layers[layer])
    if wl.quant:
        for nm, qd in wl.quant[layer].items():
            if "zeros" in qd:
                lw[nm] = dequant_int4(qd["q"], qd["scales"], qd["zeros"], wl.spec.group)
            else:
                lw[nm] = dequant_int8(qd["q"], qd["scales"])
    return lw


def encoder_forward(wl, hidden_out=False):
    """Whole forward on a ``workloads.Workload``.

    Returns the pooled, L2-normalised embeddings [B, H] (output kind
    "pooled") or the final hidden states [B, S, H] (output kind "hidden";
    only valid-token rows are meaningful).
    """
    sp = wl.spec
    if sp.input_kind == "ids":
        x = embed(wl.ids, wl.emb["word"], wl.emb["pos"], wl.emb["type"], wl.emb["gamma"], wl.emb["beta"], sp.eps)
    else:
        x = _f64(wl.hidden_in)
    for layer in range(sp.layers):
        x = encoder_layer(x, wl.mask, layer_weights(wl, layer), sp.heads, sp.eps)
    if hidden_out or sp.output_kind == "hidden":
        return x
    return mean_pool_l2(x, wl.mask)
