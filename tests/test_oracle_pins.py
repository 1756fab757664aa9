"""Pins for the CPU oracle: each oracle function is checked against something
other than itself -- pure-Python brute force on tiny inputs, closed forms,
invariants, and special cases computed by independent library routines
(torch SDPA, torch TransformerEncoderLayer, transformers BertModel, all in
float64).  No GPU is used.
"""
import math

import numpy as np
import pytest

import oracle
import workloads
from oracle import MASK_CAUSAL, MASK_CUSTOM, MASK_NONE, MASK_SLIDING_WINDOW


# ---------------------------------------------------------------------------
# pure-Python brute force (tiny shapes only)
# ---------------------------------------------------------------------------

def bf_linear(x, w, b):
    m, k = len(x), len(x[0])
    n = len(w)
    return [[sum(x[i][kk] * w[j][kk] for kk in range(k)) + b[j] for j in range(n)] for i in range(m)]


def bf_layer_norm_row(row, g, be, eps):
    n = len(row)
    mu = sum(row) / n
    var = sum((r - mu) ** 2 for r in row) / n
    return [(row[i] - mu) / math.sqrt(var + eps) * g[i] + be[i] for i in range(n)]


def bf_gelu(x):
    return 0.5 * x * (1.0 + math.erf(x / math.sqrt(2.0)))


def bf_attention_head(q, k, v, visible, scale):
    S, d = len(q), len(q[0])
    out = []
    for i in range(S):
        cols = [j for j in range(S) if visible(i, j)]
        if not cols:
            out.append([0.0] * d)
            continue
        sc = [scale * sum(q[i][t] * k[j][t] for t in range(d)) for j in cols]
        mx = max(sc)
        e = [math.exp(s - mx) for s in sc]
        tot = sum(e)
        out.append([sum(e[c] / tot * v[j][t] for c, j in enumerate(cols)) for t in range(d)])
    return out


def bf_encoder_layer(x, mask, lw, heads, eps):
    """Post-LN layer on nested lists: x[b][s][h]."""
    B, S, H = len(x), len(x[0]), len(x[0][0])
    d = H // heads
    out = []
    for b in range(B):
        qkv = bf_linear(x[b], lw["wqkv"].tolist(), lw["bqkv"].tolist())
        ctx = [[0.0] * H for _ in range(S)]
        for h in range(heads):
            q = [row[h * d:(h + 1) * d] for row in qkv]
            k = [row[H + h * d:H + (h + 1) * d] for row in qkv]
            v = [row[2 * H + h * d:2 * H + (h + 1) * d] for row in qkv]
            o = bf_attention_head(q, k, v, lambda i, j: mask[b][j] != 0, 1.0 / math.sqrt(d))
            for s in range(S):
                ctx[s][h * d:(h + 1) * d] = o[s]
        a = bf_linear(ctx, lw["wo"].tolist(), lw["bo"].tolist())
        x1 = [bf_layer_norm_row([a[s][i] + x[b][s][i] for i in range(H)], lw["ln1_g"], lw["ln1_b"], eps)
              for s in range(S)]
        f = bf_linear(x1, lw["w1"].tolist(), lw["b1"].tolist())
        g = [[bf_gelu(t) for t in row] for row in f]
        y = bf_linear(g, lw["w2"].tolist(), lw["b2"].tolist())
        out.append([bf_layer_norm_row([y[s][i] + x1[s][i] for i in range(H)], lw["ln2_g"], lw["ln2_b"], eps)
                    for s in range(S)])
    return out


def tiny_layer(rng, H=8, F=12, affine=True):
    def w(*s):
        return rng.normal(0, 0.3, size=s)
    return dict(wqkv=w(3 * H, H), bqkv=w(3 * H) if affine else np.zeros(3 * H), wo=w(H, H), bo=w(H),
                ln1_g=1 + w(H), ln1_b=w(H), w1=w(F, H), b1=w(F), w2=w(H, F), b2=w(H),
                ln2_g=1 + w(H), ln2_b=w(H))


# ---------------------------------------------------------------------------
# linear
# ---------------------------------------------------------------------------

def test_linear_matches_brute_force_nonsquare():
    rng = np.random.default_rng(10)
    x, w, b = rng.normal(size=(3, 5)), rng.normal(size=(7, 5)), rng.normal(size=7)
    got = oracle.linear(x, w, b)
    ref = np.array(bf_linear(x.tolist(), w.tolist(), b.tolist()))
    assert got.shape == (3, 7)
    assert np.max(np.abs(got - ref)) < 1e-12


def test_linear_identity_weight_closed_form():
    x = np.arange(12.0).reshape(3, 4)
    b = np.array([1.0, -2.0, 0.5, 0.0])
    assert np.array_equal(oracle.linear(x, np.eye(4), b), x + b)


# ---------------------------------------------------------------------------
# GELU
# ---------------------------------------------------------------------------

def test_gelu_closed_forms():
    # GELU(x) = x * Phi(x); Phi(1), Phi(2) from the standard normal CDF.
    assert oracle.gelu(np.array([0.0]))[0] == 0.0
    assert abs(oracle.gelu(np.array([1.0]))[0] - 0.8413447460685429) < 1e-15
    assert abs(oracle.gelu(np.array([2.0]))[0] - 2 * 0.9772498680518208) < 1e-15
    assert abs(oracle.gelu(np.array([-1.0]))[0] - (-(1 - 0.8413447460685429))) < 1e-15
    x = np.linspace(-6, 6, 97)
    # odd part: GELU(x) - GELU(-x) = x
    assert np.max(np.abs(oracle.gelu(x) - oracle.gelu(-x) - x)) < 1e-14
    assert np.max(np.abs(oracle.gelu(x) - np.array([bf_gelu(t) for t in x]))) < 1e-14


# ---------------------------------------------------------------------------
# LayerNorm
# ---------------------------------------------------------------------------

def test_layer_norm_moments_and_constant_rows():
    rng = np.random.default_rng(11)
    x = rng.normal(2.0, 3.0, size=(64, 384))
    y = oracle.layer_norm(x, np.ones(384), np.zeros(384), 1e-12)
    assert np.max(np.abs(y.mean(axis=1))) < 1e-12
    var = x.var(axis=1)
    assert np.max(np.abs(y.var(axis=1) - var / (var + 1e-12))) < 1e-9
    c = np.full((3, 384), 5.0)
    beta = rng.normal(size=384)
    assert np.array_equal(oracle.layer_norm(c, rng.normal(size=384), beta, 1e-12), np.tile(beta, (3, 1)))
    g, be = rng.normal(size=8), rng.normal(size=8)
    row = rng.normal(size=8)
    ref = bf_layer_norm_row(row.tolist(), g, be, 1e-5)
    assert np.max(np.abs(oracle.layer_norm(row[None], g, be, 1e-5)[0] - ref)) < 1e-13


# ---------------------------------------------------------------------------
# masked attention
# ---------------------------------------------------------------------------

def _qkv(rng, B, S, nh, d):
    return (rng.normal(size=(B, S, nh, d)), rng.normal(size=(B, S, nh, d)), rng.normal(size=(B, S, nh, d)))


@pytest.mark.parametrize("kind,window", [(MASK_NONE, 0), (MASK_CUSTOM, 0), (MASK_CAUSAL, 0),
                                         (MASK_SLIDING_WINDOW, 3), (MASK_SLIDING_WINDOW, 1)])
def test_attention_matches_brute_force(kind, window):
    rng = np.random.default_rng(12 + kind + window)
    B, S, nh, d = 2, 6, 2, 4
    q, k, v = _qkv(rng, B, S, nh, d)
    km = np.array([[1, 1, 1, 1, 0, 0], [1, 0, 1, 1, 1, 0]], np.uint8)
    use_mask = km if kind == MASK_CUSTOM else None
    got = oracle.masked_attention(q, k, v, kind, use_mask, window, 0.37)
    for b in range(B):
        def vis(i, j, b=b):
            ok = True
            if kind == MASK_CAUSAL:
                ok = j <= i
            elif kind == MASK_SLIDING_WINDOW:
                ok = (j <= i) and (i - j < window)
            if kind == MASK_CUSTOM:
                ok = ok and km[b][j] == 1
            return ok
        for h in range(nh):
            ref = bf_attention_head(q[b, :, h].tolist(), k[b, :, h].tolist(), v[b, :, h].tolist(), vis, 0.37)
            assert np.max(np.abs(got[b, :, h] - np.array(ref))) < 1e-13


def test_attention_probs_rows_sum_to_one_and_masked_keys_zero():
    rng = np.random.default_rng(13)
    S, d = 40, 32
    q, k = rng.normal(size=(S, d)), rng.normal(size=(S, d))
    km = (rng.random(S) < 0.6).astype(np.uint8)
    km[0] = 1
    vis = oracle.visible_keys(S, MASK_CUSTOM, km)
    p = oracle.attention_probs(q, k, vis, 1 / math.sqrt(d))
    assert np.max(np.abs(p.sum(axis=1) - 1)) < 1e-14
    assert np.all(p[:, km == 0] == 0.0)


def test_attention_padding_extension_invariance():
    rng = np.random.default_rng(14)
    B, S, nh, d, extra = 3, 20, 3, 8, 13
    q, k, v = _qkv(rng, B, S, nh, d)
    lens = np.array([20, 7, 1])
    km = (np.arange(S)[None] < lens[:, None]).astype(np.uint8)
    a = oracle.masked_attention(q, k, v, MASK_CUSTOM, km)
    pad = lambda t: np.concatenate([t, 1e3 * rng.normal(size=(B, extra, nh, d))], axis=1)
    km2 = np.concatenate([km, np.zeros((B, extra), np.uint8)], axis=1)
    b2 = oracle.masked_attention(pad(q), pad(k), pad(v), MASK_CUSTOM, km2)
    for b in range(B):
        assert np.max(np.abs(a[b, :lens[b]] - b2[b, :lens[b]])) < 1e-13


def test_attention_identical_keys_gives_mean_of_values():
    rng = np.random.default_rng(15)
    S, d = 12, 16
    q = rng.normal(size=(1, S, 1, d))
    k = np.tile(rng.normal(size=(1, 1, 1, d)), (1, S, 1, 1))
    v = rng.normal(size=(1, S, 1, d))
    km = np.zeros((1, S), np.uint8)
    km[0, [0, 3, 4, 9]] = 1
    out = oracle.masked_attention(q, k, v, MASK_CUSTOM, km)
    mean_v = v[0, [0, 3, 4, 9], 0].mean(axis=0)
    assert np.max(np.abs(out[0, :, 0] - mean_v)) < 1e-14


def test_attention_single_valid_key_and_empty_rows():
    rng = np.random.default_rng(16)
    S, d = 9, 8
    q, k, v = _qkv(rng, 1, S, 2, d)
    km = np.zeros((1, S), np.uint8)
    km[0, 5] = 1
    out = oracle.masked_attention(q, k, v, MASK_CUSTOM, km)
    assert np.array_equal(out[0, :, 0], np.tile(v[0, 5, 0], (S, 1)))
    km[:] = 0
    assert np.all(oracle.masked_attention(q, k, v, MASK_CUSTOM, km) == 0.0)


@pytest.mark.parametrize("kind", [MASK_NONE, MASK_CUSTOM, MASK_CAUSAL, MASK_SLIDING_WINDOW])
def test_attention_matches_torch_sdpa_float64(kind):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(17)
    B, S, nh, d, w = 3, 24, 4, 32, 5
    q, k, v = _qkv(rng, B, S, nh, d)
    lens = np.array([24, 11, 3])
    km = (np.arange(S)[None] < lens[:, None]).astype(np.uint8)
    km_use = km if kind == MASK_CUSTOM else None
    got = oracle.masked_attention(q, k, v, kind, km_use, w)
    vis = np.stack([oracle.visible_keys(S, kind, None if km_use is None else km_use[b], w) for b in range(B)])
    t = lambda a: torch.from_numpy(a).permute(0, 2, 1, 3)
    ref = torch.nn.functional.scaled_dot_product_attention(
        t(q), t(k), t(v), attn_mask=torch.from_numpy(vis)[:, None]).permute(0, 2, 1, 3).numpy()
    # SDPA gives NaN for rows without any visible key; those rows are 0 by definition here.
    has = vis.any(axis=2)
    for b in range(B):
        assert np.max(np.abs(got[b][has[b]] - ref[b][has[b]])) < 1e-13
        assert np.all(got[b][~has[b]] == 0)


# ---------------------------------------------------------------------------
# pooling
# ---------------------------------------------------------------------------

def test_pooling_unit_norm_and_special_cases():
    rng = np.random.default_rng(18)
    x = rng.normal(size=(4, 10, 384))
    lens = np.array([10, 1, 4, 0])
    m = (np.arange(10)[None] < lens[:, None]).astype(np.uint8)
    p = oracle.mean_pool_l2(x, m)
    assert np.max(np.abs(np.linalg.norm(p[:3], axis=1) - 1)) < 1e-14
    assert np.max(np.abs(p[1] - x[1, 0] / np.linalg.norm(x[1, 0]))) < 1e-15
    e = x[2, :4].mean(axis=0)
    assert np.max(np.abs(p[2] - e / np.linalg.norm(e))) < 1e-14
    assert np.all(p[3] == 0)


# ---------------------------------------------------------------------------
# embedding
# ---------------------------------------------------------------------------

def test_embed_brute_force():
    rng = np.random.default_rng(19)
    V, P, H, B, S = 50, 12, 8, 2, 5
    word, pos, typ = rng.normal(size=(V, H)), rng.normal(size=(P, H)), rng.normal(size=(2, H))
    g, be = rng.normal(size=H), rng.normal(size=H)
    ids = rng.integers(0, V, size=(B, S))
    got = oracle.embed(ids, word, pos, typ, g, be, 1e-12)
    for b in range(B):
        for s in range(S):
            row = [word[ids[b, s], i] + pos[s, i] + typ[0, i] for i in range(H)]
            assert np.max(np.abs(got[b, s] - bf_layer_norm_row(row, g, be, 1e-12))) < 1e-13


# ---------------------------------------------------------------------------
# whole layer and whole encoder
# ---------------------------------------------------------------------------

def test_encoder_layer_matches_brute_force_tiny():
    rng = np.random.default_rng(20)
    B, S, H, heads = 2, 5, 8, 2
    lw = tiny_layer(rng, H=H, F=12)
    x = rng.normal(size=(B, S, H))
    mask = np.array([[1, 1, 1, 0, 0], [1, 1, 1, 1, 1]], np.uint8)
    got = oracle.encoder_layer(x, mask, lw, heads, 1e-12)
    ref = np.array(bf_encoder_layer(x.tolist(), mask.tolist(), lw, heads, 1e-12))
    for b in range(B):
        L = int(mask[b].sum())
        assert np.max(np.abs(got[b, :L] - ref[b, :L])) < 1e-12


def test_encoder_layer_matches_torch_transformer_layer_float64():
    torch = pytest.importorskip("torch")
    wl = workloads.make(workloads.spec("layer_f32_b2_s16"), affine=True)
    lw = wl.layers[0]
    layer = torch.nn.TransformerEncoderLayer(384, 12, 1536, dropout=0.0, activation="gelu", batch_first=True,
                                             norm_first=False, layer_norm_eps=1e-12, dtype=torch.float64).eval()
    sd = {"self_attn.in_proj_weight": lw["wqkv"], "self_attn.in_proj_bias": lw["bqkv"],
          "self_attn.out_proj.weight": lw["wo"], "self_attn.out_proj.bias": lw["bo"],
          "linear1.weight": lw["w1"], "linear1.bias": lw["b1"], "linear2.weight": lw["w2"], "linear2.bias": lw["b2"],
          "norm1.weight": lw["ln1_g"], "norm1.bias": lw["ln1_b"], "norm2.weight": lw["ln2_g"], "norm2.bias": lw["ln2_b"]}
    layer.load_state_dict({k: torch.from_numpy(np.asarray(v, np.float64)) for k, v in sd.items()})
    x = torch.from_numpy(wl.hidden_in.astype(np.float64))
    with torch.no_grad():
        ref = layer(x, src_key_padding_mask=torch.from_numpy(wl.mask == 0)).numpy()
    got = oracle.encoder_forward(wl)
    for b, L in enumerate(wl.lengths):
        assert np.max(np.abs(got[b, :L] - ref[b, :L])) < 1e-10


@pytest.mark.slow
def test_encoder_forward_matches_transformers_bert_float64():
    torch = pytest.importorskip("torch")
    transformers = pytest.importorskip("transformers")
    sp = workloads.spec("minilm_b32_s128_bf16", batch=3, seq=24, layers=2, len_lo=1, len_hi=24)
    wl = workloads.make(sp, affine=True)
    cfg = transformers.BertConfig(vocab_size=sp.vocab, hidden_size=384, num_hidden_layers=sp.layers,
                                  num_attention_heads=12, intermediate_size=1536, hidden_act="gelu",
                                  max_position_embeddings=512, type_vocab_size=2, layer_norm_eps=1e-12,
                                  hidden_dropout_prob=0.0, attention_probs_dropout_prob=0.0,
                                  attn_implementation="eager")
    m = transformers.BertModel(cfg, add_pooling_layer=False).double().eval()
    sd = {"embeddings.word_embeddings.weight": wl.emb["word"], "embeddings.position_embeddings.weight": wl.emb["pos"],
          "embeddings.token_type_embeddings.weight": wl.emb["type"], "embeddings.LayerNorm.weight": wl.emb["gamma"],
          "embeddings.LayerNorm.bias": wl.emb["beta"]}
    H = 384
    for i, lw in enumerate(wl.layers):
        p = f"encoder.layer.{i}."
        sd.update({p + "attention.self.query.weight": lw["wqkv"][:H], p + "attention.self.query.bias": lw["bqkv"][:H],
                   p + "attention.self.key.weight": lw["wqkv"][H:2 * H], p + "attention.self.key.bias": lw["bqkv"][H:2 * H],
                   p + "attention.self.value.weight": lw["wqkv"][2 * H:], p + "attention.self.value.bias": lw["bqkv"][2 * H:],
                   p + "attention.output.dense.weight": lw["wo"], p + "attention.output.dense.bias": lw["bo"],
                   p + "attention.output.LayerNorm.weight": lw["ln1_g"], p + "attention.output.LayerNorm.bias": lw["ln1_b"],
                   p + "intermediate.dense.weight": lw["w1"], p + "intermediate.dense.bias": lw["b1"],
                   p + "output.dense.weight": lw["w2"], p + "output.dense.bias": lw["b2"],
                   p + "output.LayerNorm.weight": lw["ln2_g"], p + "output.LayerNorm.bias": lw["ln2_b"]})
    missing = m.load_state_dict({k: torch.from_numpy(np.asarray(v, np.float64)) for k, v in sd.items()}, strict=False)
    assert not missing.unexpected_keys
    with torch.no_grad():
        hs = m(input_ids=torch.from_numpy(wl.ids.astype(np.int64)),
               attention_mask=torch.from_numpy(wl.mask.astype(np.int64))).last_hidden_state.numpy()
    mk = wl.mask.astype(np.float64)[:, :, None]
    e = (hs * mk).sum(1) / mk.sum(1)
    ref = e / np.linalg.norm(e, axis=1, keepdims=True)
    got = oracle.encoder_forward(wl)
    assert np.max(np.abs(got - ref)) < 1e-10
    hid = oracle.encoder_forward(wl, hidden_out=True)
    for b, L in enumerate(wl.lengths):
        assert np.max(np.abs(hid[b, :L] - hs[b, :L])) < 1e-9


def test_encoder_padding_extension_invariance():
    sp = workloads.spec("minilm_b32_s128_bf16", batch=3, seq=16, layers=2, len_lo=2, len_hi=16)
    wl = workloads.make(sp, affine=True)
    wl2 = workloads.with_padding_extended(wl, 9)
    a = oracle.encoder_forward(wl)
    b = oracle.encoder_forward(wl2)
    assert np.max(np.abs(a - b)) < 1e-12


# ---------------------------------------------------------------------------
# quantisation
# ---------------------------------------------------------------------------

def test_unpack_int4_matches_bit_loop():
    rng = np.random.default_rng(21)
    packed = rng.integers(0, 256, size=(5, 16)).astype(np.uint8)
    got = oracle.unpack_int4(packed)
    for n in range(5):
        for k in range(32):
            byte = int(packed[n, k // 2])
            want = (byte >> (4 * (k % 2))) & 0xF
            assert got[n, k] == want


def test_int4_dequant_bit_loop_and_round_trip():
    rng = np.random.default_rng(22)
    w = rng.normal(0, 0.02, size=(24, 96)).astype(np.float32)
    packed, s, z = workloads.quantize_int4_grouped(w, 32)
    deq = oracle.dequant_int4(packed, s, z, 32)
    # bit loop over one row: (code - zero) * scale, each factor exactly as stored
    for k in range(96):
        code = (int(packed[3, k // 2]) >> (4 * (k & 1))) & 15
        assert deq[3, k] == (code - float(z[3, k // 32])) * float(s[3, k // 32])
    # exactly representable in fp32
    assert np.array_equal(deq.astype(np.float32).astype(np.float64), deq)
    sg = np.repeat(s.astype(np.float64), 32, axis=1)
    codes = oracle.unpack_int4(packed)
    unclamped = (codes > 0) & (codes < 15)
    err = np.abs(w - deq)
    assert np.all(err[unclamped] <= sg[unclamped] / 2 * (1 + 1e-6))
    assert np.all(err <= sg * 1.01)


def test_int8_dequant_round_trip():
    rng = np.random.default_rng(23)
    w = rng.normal(0, 0.02, size=(40, 64)).astype(np.float32)
    q, s = workloads.quantize_int8_per_channel(w)
    deq = oracle.dequant_int8(q, s)
    assert np.array_equal(deq.astype(np.float32).astype(np.float64), deq)
    sn = s.astype(np.float64)[:, None]
    assert np.all(np.abs(w - deq) <= sn / 2 * (1 + 1e-6) + 1e-12)
    assert np.array_equal(deq[7], q[7].astype(np.float64) * float(s[7]))
    assert np.max(np.abs(q)) == 127


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -8 + 2 ** -20, -2.5], np.float32)
    got = workloads.round_to_bf16(x)
    assert got.tolist() == [1.0, 1.0, 1.0 + 2 ** -6, 1.0 + 2 ** -7, -2.5]
