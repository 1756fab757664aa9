"""A model of the bf16 forward's roundings, for deriving test tolerances.

Not an oracle: the reference is the float64 oracle. This is the dense bf16
encoder forward (post-LN BERT layers, masked mean pooling) in float32, with
every activation rounded to bf16 (round to nearest even) where the GPU path
stores bf16:
  - the embedding output;
  - Q, K and V;
  - the attention probabilities P before P V (their row sum stays fp32);
  - the attention context;
  - the output projection's sum (the LN1 input);
  - the GELU output;
  - FFN-down's sum (the LN2 input).
Each LayerNorm is applied as the deferred form computes it: the consumer
multiplies by bf16(gamma_k W_nk) and applies rstd (acc - mean u_n) + v_n,
with u_n = sum_k bf16(gamma_k W_nk) and v_n = b_n + sum_k beta_k W_nk, and
the statistics are those of the stored bf16 rows. A residual is normalised
in fp32.  The distance between this model and the oracle is the size of the
rounding error the GPU path is built to make; a kernel defect shows up as
a GPU result much farther from the model than that.
"""
import numpy as np


def bf16(x):
    """Round float32 values to the nearest bf16 (ties to even), returned as float32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + r) & np.uint32(0xFFFF0000)).view(np.float32)


def _stats(x, eps):
    x = x.astype(np.float64)
    mean = x.mean(axis=-1, keepdims=True)
    var = ((x - mean) ** 2).mean(axis=-1, keepdims=True)
    return mean.astype(np.float32), (1.0 / np.sqrt(var + eps)).astype(np.float32)


def _fold(w, gamma, beta, bias):
    wf = bf16(w * gamma[None, :].astype(np.float32))
    u = wf.astype(np.float64).sum(axis=1).astype(np.float32)
    v = (bias.astype(np.float64) + w.astype(np.float64) @ beta.astype(np.float64)).astype(np.float32)
    return wf, u, v


def _gelu(x):
    from scipy.special import erf
    return (0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))).astype(np.float32)


def _attention(q, k, v, scale):
    """One sequence and head: q, k, v [L, d] bf16 values."""
    s = (q @ k.T) * np.float32(scale)
    m = s.max(axis=1, keepdims=True)
    p = np.exp(s - m).astype(np.float32)
    l_sum = p.sum(axis=1, keepdims=True)
    return (bf16(p) @ v) / l_sum


def encoder_forward(wl):
    """Pooled, L2-normalised embeddings [B, H] of a dense bf16 id-input workload."""
    sp = wl.spec
    assert sp.input_kind == "ids" and sp.dtype == "bf16" and sp.quant == "none"
    H, heads, eps = sp.hidden, sp.heads, sp.eps
    d = H // heads
    out = np.zeros((sp.batch, H), np.float32)
    E = {k: np.asarray(v, np.float32) for k, v in wl.emb.items()}
    layers = [{k: np.asarray(v, np.float32) for k, v in lw.items()} for lw in wl.layers]
    folds = []
    for li, lw in enumerate(layers):
        f = {}
        if li > 0:
            prev = layers[li - 1]
            f["wqkv"], f["uq"], f["vq"] = _fold(lw["wqkv"], prev["ln2_g"], prev["ln2_b"], lw["bqkv"])
        f["w1"], f["u1"], f["v1"] = _fold(lw["w1"], lw["ln1_g"], lw["ln1_b"], lw["b1"])
        folds.append(f)
    for b in range(sp.batch):
        pos = np.nonzero(wl.mask[b])[0]
        if len(pos) == 0:
            continue
        e = E["word"][wl.ids[b, pos]] + E["pos"][pos] + E["type"][0][None, :]
        mean, rstd = _stats(e, eps)
        x = bf16((e - mean) * rstd * E["gamma"] + E["beta"])  # layer 0 input (normalised)
        x_stats = None  # (mean, rstd, gamma, beta) of x when it is an LN2 input
        for li, lw in enumerate(layers):
            f = folds[li]
            if x_stats is None:
                qkv = x @ lw["wqkv"].T + lw["bqkv"]
                resid = x
            else:
                m2, r2, g2, b2 = x_stats
                qkv = r2 * (x @ f["wqkv"].T - m2 * f["uq"]) + f["vq"]
                resid = (x - m2) * r2 * g2 + b2
            qkv = bf16(qkv)
            ctx = np.zeros((len(pos), H), np.float32)
            for h in range(heads):
                q = qkv[:, h * d:(h + 1) * d]
                k = qkv[:, H + h * d:H + (h + 1) * d]
                v = qkv[:, 2 * H + h * d:2 * H + (h + 1) * d]
                ctx[:, h * d:(h + 1) * d] = _attention(q, k, v, 1.0 / np.sqrt(d))
            a = bf16(bf16(ctx) @ lw["wo"].T + lw["bo"] + resid)
            m1, r1 = _stats(a, eps)
            g = bf16(_gelu(r1 * (a @ f["w1"].T - m1 * f["u1"]) + f["v1"]))
            ln1 = (a - m1) * r1 * lw["ln1_g"] + lw["ln1_b"]
            x = bf16(g @ lw["w2"].T + lw["b2"] + ln1)
            m2, r2 = _stats(x, eps)
            x_stats = (m2, r2, lw["ln2_g"], lw["ln2_b"])
        m2, r2, g2, b2 = x_stats
        pooled = ((x - m2) * r2).astype(np.float64).mean(axis=0) * g2.astype(np.float64) + b2
        out[b] = (pooled / max(np.sqrt((pooled * pooled).sum()), 1e-12)).astype(np.float32)
    return out
