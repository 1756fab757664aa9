"""The oracle's pins are strong enough to catch plausible mistakes.

Each case plants one mistake in the CPU oracle (a dropped term, a wrong sign,
an off-by-one mask, a transposed operand, a swapped nibble ...), runs every pin
of tests/test_oracle_pins.py against the mutated oracle and requires that at
least one pin fails.  Mistakes are planted on the CPU only, by patching the
oracle's module attributes for the duration of one case.
"""
import math

import numpy as np
import pytest

import oracle
import oracle.encoder as enc
import oracle.quant as qnt
import test_oracle_pins as pins

_f64 = enc._f64
# the unmutated functions, for mutants that wrap them
ORIG = {n: getattr(enc, n) for n in ("layer_norm", "gelu", "linear", "visible_keys", "attention_probs",
                                     "masked_attention", "embed", "encoder_layer", "mean_pool_l2")}
ORIG.update({n: getattr(qnt, n) for n in ("unpack_int4", "dequant_int4", "dequant_int8")})


def _pin_calls():
    calls = [
        pins.test_linear_matches_brute_force_nonsquare,
        pins.test_linear_identity_weight_closed_form,
        pins.test_gelu_closed_forms,
        pins.test_layer_norm_moments_and_constant_rows,
        pins.test_attention_probs_rows_sum_to_one_and_masked_keys_zero,
        pins.test_attention_padding_extension_invariance,
        pins.test_attention_identical_keys_gives_mean_of_values,
        pins.test_attention_single_valid_key_and_empty_rows,
        pins.test_pooling_unit_norm_and_special_cases,
        pins.test_embed_brute_force,
        pins.test_encoder_layer_matches_brute_force_tiny,
        pins.test_encoder_padding_extension_invariance,
        pins.test_unpack_int4_matches_bit_loop,
        pins.test_int4_dequant_bit_loop_and_round_trip,
        pins.test_int8_dequant_round_trip,
    ]
    for kind, window in [(oracle.MASK_NONE, 0), (oracle.MASK_CUSTOM, 0), (oracle.MASK_CAUSAL, 0),
                         (oracle.MASK_SLIDING_WINDOW, 1), (oracle.MASK_SLIDING_WINDOW, 3)]:
        calls.append(lambda kind=kind, window=window: pins.test_attention_matches_brute_force(kind, window))
    return calls


# --- planted mistakes (each returns a replacement for one oracle function) ---

def ln_unbiased_variance(x, gamma, beta, eps):
    x = _f64(x)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).sum(axis=-1, keepdims=True) / (x.shape[-1] - 1)
    return (x - mu) / np.sqrt(var + eps) * _f64(gamma) + _f64(beta)


def ln_eps_outside_sqrt(x, gamma, beta, eps):
    x = _f64(x)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / (np.sqrt(var) + eps) * _f64(gamma) + _f64(beta)


def ln_no_beta(x, gamma, beta, eps):
    x = _f64(x)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * _f64(gamma)


def gelu_tanh(x):
    x = _f64(x)
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)))


def gelu_no_sqrt2(x):
    from scipy.special import erf
    x = _f64(x)
    return 0.5 * x * (1.0 + erf(x))


def linear_no_bias(x, w, b=None):
    return _f64(x) @ _f64(w).T


def linear_untransposed(x, w, b=None):
    y = _f64(x) @ _f64(w)
    return y if b is None else y + _f64(b)


def vis_causal_strict(S, kind, key_mask_row=None, window=0):
    i, j = np.arange(S)[:, None], np.arange(S)[None, :]
    vis = ORIG["visible_keys"](S, kind, key_mask_row, window)
    if kind == oracle.MASK_CAUSAL:
        vis = vis & (j < i)
    return vis


def vis_window_inclusive(S, kind, key_mask_row=None, window=0):
    i, j = np.arange(S)[:, None], np.arange(S)[None, :]
    vis = ORIG["visible_keys"](S, kind, key_mask_row, window)
    if kind == oracle.MASK_SLIDING_WINDOW:
        vis = (j <= i) & (j >= i - window)
        if key_mask_row is not None:
            vis = vis & (np.asarray(key_mask_row)[None, :] != 0)
    return vis


def vis_key_mask_ignored(S, kind, key_mask_row=None, window=0):
    return ORIG["visible_keys"](S, oracle.MASK_NONE if kind == oracle.MASK_CUSTOM else kind, None, window)


def probs_no_scale(q, k, vis, scale):
    return ORIG["attention_probs"](q, k, vis, 1.0)


def probs_softmax_over_queries(q, k, vis, scale):
    s = scale * (_f64(q) @ _f64(k).T)
    s = np.where(vis, s, -np.inf)
    with np.errstate(invalid="ignore"):  # columns no query sees
        e = np.exp(s - s.max(axis=0, keepdims=True))
    e = np.where(vis, e, 0.0)
    tot = e.sum(axis=0, keepdims=True)
    return np.divide(e, tot, out=np.zeros_like(e), where=tot > 0)


def attention_heads_mixed(q, k, v, kind=oracle.MASK_CUSTOM, key_mask=None, window=0, scale=None):
    k = np.roll(_f64(k), 1, axis=2)  # head h attends with head h-1's keys
    return ORIG["masked_attention"](q, k, v, kind, key_mask, window, scale)


def pool_l1_norm(x, mask):
    # (dividing the sum by S instead of the token count is no mistake here: the
    # L2 normalisation removes any positive scale)
    x = _f64(x)
    m = _f64(mask)[:, :, None]
    e = (x * m).sum(axis=1) / np.maximum(m.sum(axis=1), 1e-9)
    n = np.abs(e).sum(axis=1, keepdims=True)
    return e / np.maximum(n, 1e-12)


def pool_mask_ignored(x, mask):
    return ORIG["mean_pool_l2"](x, np.ones_like(np.asarray(mask)))


def embed_pos_off_by_one(ids, word, pos, typ, gamma, beta, eps):
    ids = np.asarray(ids)
    B, S = ids.shape
    x = _f64(word)[ids] + _f64(pos)[np.arange(1, S + 1)][None] + _f64(typ)[0][None, None]
    return enc.layer_norm(x, gamma, beta, eps)


def embed_type_one(ids, word, pos, typ, gamma, beta, eps):
    ids = np.asarray(ids)
    B, S = ids.shape
    x = _f64(word)[ids] + _f64(pos)[np.arange(S)][None] + _f64(typ)[1][None, None]
    return enc.layer_norm(x, gamma, beta, eps)


def layer_pre_ln(x, mask, lw, heads, eps):
    x = _f64(x)
    B, S, H = x.shape
    d = H // heads
    h = enc.layer_norm(x, lw["ln1_g"], lw["ln1_b"], eps)
    qkv = enc.linear(h, lw["wqkv"], lw["bqkv"])
    q, k, v = (qkv[..., i * H:(i + 1) * H].reshape(B, S, heads, d) for i in range(3))
    ctx = enc.masked_attention(q, k, v, oracle.MASK_CUSTOM, mask, 0, 1.0 / math.sqrt(d)).reshape(B, S, H)
    x1 = x + enc.linear(ctx, lw["wo"], lw["bo"])
    g = enc.gelu(enc.linear(enc.layer_norm(x1, lw["ln2_g"], lw["ln2_b"], eps), lw["w1"], lw["b1"]))
    return x1 + enc.linear(g, lw["w2"], lw["b2"])


def layer_no_ffn_residual(x, mask, lw, heads, eps):
    x = _f64(x)
    B, S, H = x.shape
    d = H // heads
    qkv = enc.linear(x, lw["wqkv"], lw["bqkv"])
    q, k, v = (qkv[..., i * H:(i + 1) * H].reshape(B, S, heads, d) for i in range(3))
    ctx = enc.masked_attention(q, k, v, oracle.MASK_CUSTOM, mask, 0, 1.0 / math.sqrt(d)).reshape(B, S, H)
    x1 = enc.layer_norm(enc.linear(ctx, lw["wo"], lw["bo"]) + x, lw["ln1_g"], lw["ln1_b"], eps)
    g = enc.gelu(enc.linear(x1, lw["w1"], lw["b1"]))
    return enc.layer_norm(enc.linear(g, lw["w2"], lw["b2"]), lw["ln2_g"], lw["ln2_b"], eps)


def unpack_high_nibble_first(packed):
    p = np.asarray(packed, dtype=np.uint8)
    n, kh = p.shape
    q = np.empty((n, 2 * kh), dtype=np.uint8)
    q[:, 0::2] = p >> 4
    q[:, 1::2] = p & 0x0F
    return q


def int4_zero_ignored(packed, scales, zeros, group):
    return ORIG["dequant_int4"](packed, scales, np.zeros_like(np.asarray(zeros)), group)


def int8_scale_ignored(q, scales):
    return np.asarray(q, dtype=np.int8).astype(np.float64)


MUTANTS = {
    "layer_norm: unbiased variance": ("layer_norm", ln_unbiased_variance),
    "layer_norm: eps outside the square root": ("layer_norm", ln_eps_outside_sqrt),
    "layer_norm: beta dropped": ("layer_norm", ln_no_beta),
    "gelu: tanh approximation": ("gelu", gelu_tanh),
    "gelu: erf(x) instead of erf(x/sqrt 2)": ("gelu", gelu_no_sqrt2),
    "linear: bias dropped": ("linear", linear_no_bias),
    "linear: weight not transposed": ("linear", linear_untransposed),
    "mask: causal excludes the diagonal": ("visible_keys", vis_causal_strict),
    "mask: sliding window one key too wide": ("visible_keys", vis_window_inclusive),
    "mask: key mask ignored": ("visible_keys", vis_key_mask_ignored),
    "attention: scale dropped": ("attention_probs", probs_no_scale),
    "attention: softmax over queries": ("attention_probs", probs_softmax_over_queries),
    "attention: keys of the wrong head": ("masked_attention", attention_heads_mixed),
    "pooling: L1 instead of L2 normalisation": ("mean_pool_l2", pool_l1_norm),
    "pooling: mask ignored": ("mean_pool_l2", pool_mask_ignored),
    "embed: positions shifted by one": ("embed", embed_pos_off_by_one),
    "embed: token type 1": ("embed", embed_type_one),
    "layer: pre-LN instead of post-LN": ("encoder_layer", layer_pre_ln),
    "layer: FFN residual dropped": ("encoder_layer", layer_no_ffn_residual),
    "int4: high nibble first": ("unpack_int4", unpack_high_nibble_first),
    "int4: zero-point ignored": ("dequant_int4", int4_zero_ignored),
    "int8: scale ignored": ("dequant_int8", int8_scale_ignored),
}


@pytest.mark.parametrize("name", list(MUTANTS))
def test_planted_mistake_fails_a_pin(name, monkeypatch):
    attr, fake = MUTANTS[name]
    home = qnt if attr in ("unpack_int4", "dequant_int4", "dequant_int8") else enc
    monkeypatch.setattr(home, attr, fake)
    monkeypatch.setattr(oracle, attr, fake)
    if home is qnt and hasattr(enc, attr):
        monkeypatch.setattr(enc, attr, fake)  # the encoder module holds its own binding
    failed = []
    for call in _pin_calls():
        try:
            call()
        except Exception as e:  # an assertion, or a shape error from the planted mistake
            failed.append(type(e).__name__)
    assert failed, f"no pin caught the planted mistake '{name}'"


# --- planted mistakes in the block-scaled minifloat matmul oracle ---

import oracle.mx as omx  # noqa: E402
import test_oracle_mx as mxpins  # noqa: E402

MX_ORIG = {n: getattr(omx, n) for n in ("decode", "decode_scale", "unpack", "dequant", "MX_FORMATS")}


def _mx_pin_calls():
    calls = [mxpins.test_decode_values_fixed_by_the_format_definitions,
             mxpins.test_float8_decode_matches_torch_for_every_code,
             mxpins.test_block_scale_multiplies_its_block_only]
    for fmt in mxpins.FORMATS:
        calls.append(lambda fmt=fmt: mxpins.test_grid_structure(fmt))
        calls.append(lambda fmt=fmt: mxpins.test_unpack_matches_bit_loop(fmt))
    for fa, fb in [("e4m3", "e4m3"), ("e5m2", "e2m1"), ("e2m3", "e3m2"), ("e2m1", "e2m1")]:
        calls.append(lambda fa=fa, fb=fb: mxpins.test_scaled_matmul_matches_exact_rational_brute_force(fa, fb))
    return calls


def mx_subnormal_as_normal(codes, fmt):
    c = np.asarray(codes, dtype=np.int64)
    ebits, mbits, bias = MX_ORIG["MX_FORMATS"][fmt]
    v = MX_ORIG["decode"](codes, fmt)
    e = (c >> mbits) & ((1 << ebits) - 1)
    m = (c & ((1 << mbits) - 1)).astype(np.float64)
    sign = np.where((c >> (ebits + mbits)) & 1, -1.0, 1.0)
    return np.where(e == 0, sign * np.ldexp(1.0 + m / (1 << mbits), -bias), v)


def mx_e4m3_ieee_specials(codes, fmt):
    v = MX_ORIG["decode"](codes, fmt)
    if fmt != "e4m3":
        return v
    c = np.asarray(codes, dtype=np.int64)
    return np.where((c & 0x78) == 0x78, np.where((c & 7) == 0, np.inf, np.nan), v)


def mx_scale_bias_128(s):
    return MX_ORIG["decode_scale"](s) / 2.0


def mx_fp4_high_nibble_first(packed, fmt, K):
    q = MX_ORIG["unpack"](packed, fmt, K)
    if fmt == "e2m1":
        q = q.reshape(q.shape[0], -1, 2)[:, :, ::-1].reshape(q.shape)
    return q


def mx_fp6_big_endian(packed, fmt, K):
    if fmt not in ("e2m3", "e3m2"):
        return MX_ORIG["unpack"](packed, fmt, K)
    p = np.asarray(packed, dtype=np.uint8)
    w = p.reshape(p.shape[0], K // 4, 3).astype(np.uint32)
    word = (w[:, :, 0] << 16) | (w[:, :, 1] << 8) | w[:, :, 2]
    q = np.stack([(word >> (18 - 6 * i)) & 0x3F for i in range(4)], axis=-1)
    return q.reshape(p.shape[0], K).astype(np.uint8)


def mx_scale_per_element_block_shifted(packed, scales, fmt, K):
    v = omx.decode(omx.unpack(packed, fmt, K), fmt)
    x = omx.decode_scale(scales)
    idx = np.minimum((np.arange(K) + 1) // 32, K // 32 - 1)  # block boundary off by one
    return v * x[:, idx]


MX_MUTANTS = {
    "mx: subnormals decoded as normals": ("decode", mx_subnormal_as_normal),
    "mx: E4M3 with IEEE infinities": ("decode", mx_e4m3_ieee_specials),
    "mx: E8M0 bias 128": ("decode_scale", mx_scale_bias_128),
    "mx: FP4 high nibble first": ("unpack", mx_fp4_high_nibble_first),
    "mx: FP6 big-endian packing": ("unpack", mx_fp6_big_endian),
    "mx: block boundary off by one": ("dequant", mx_scale_per_element_block_shifted),
}


@pytest.mark.parametrize("name", list(MX_MUTANTS))
def test_planted_mx_mistake_fails_a_pin(name, monkeypatch):
    attr, fake = MX_MUTANTS[name]
    monkeypatch.setattr(omx, attr, fake)
    failed = []
    for call in _mx_pin_calls():
        try:
            call()
        except Exception as e:
            failed.append(type(e).__name__)
    assert failed, f"no pin caught the planted mistake '{name}'"


# --- planted mistakes in the GGUF block oracle ---

import oracle.gguf as ogg  # noqa: E402
import test_oracle_gguf as ggpins  # noqa: E402

GG_ORIG = {n: getattr(ogg, n) for n in ("parse", "dequant", "_f16")}


def _gguf_pin_calls():
    calls = [ggpins.test_block_sizes_and_bits_per_weight, ggpins.test_hand_built_blocks,
             ggpins.test_formats_equal_their_internal_layouts]
    for fmt in ggpins.FMTS:
        calls.append(lambda fmt=fmt: ggpins.test_element_order_matches_byte_loop(fmt))
        calls.append(lambda fmt=fmt: ggpins.test_quantise_dequantise_error_bound(fmt))
    return calls


def gg_interleaved_nibbles(blocks, fmt, K):
    codes, d, m = GG_ORIG["parse"](blocks, fmt, K)
    if fmt != "q8_0":  # elements 2j / 2j+1 in byte j instead of j / j+16
        c = codes.reshape(codes.shape[0], -1, 2, 16)
        codes = np.stack([c[:, :, 0, :], c[:, :, 1, :]], axis=3).reshape(codes.shape)
    return codes, d, m


def gg_q8_unsigned(blocks, fmt, K):
    codes, d, m = GG_ORIG["parse"](blocks, fmt, K)
    if fmt == "q8_0":
        codes = codes.view(np.uint8)
    return codes, d, m


def gg_q4_0_no_offset(blocks, fmt, K):
    w = GG_ORIG["dequant"](blocks, fmt, K)
    if fmt == "q4_0":
        _, d, _ = GG_ORIG["parse"](blocks, fmt, K)
        w = w + 8.0 * np.repeat(d, 32, axis=1)
    return w


def gg_q4_1_min_subtracted(blocks, fmt, K):
    w = GG_ORIG["dequant"](blocks, fmt, K)
    if fmt == "q4_1":
        _, _, m = GG_ORIG["parse"](blocks, fmt, K)
        w = w - 2.0 * np.repeat(m, 32, axis=1)
    return w


def gg_f16_big_endian(lo, hi):
    return GG_ORIG["_f16"](hi, lo)


GG_MUTANTS = {
    "gguf: 4-bit elements interleaved": ("parse", gg_interleaved_nibbles),
    "gguf: Q8_0 codes unsigned": ("parse", gg_q8_unsigned),
    "gguf: Q4_0 without the -8": ("dequant", gg_q4_0_no_offset),
    "gguf: Q4_1 min subtracted": ("dequant", gg_q4_1_min_subtracted),
    "gguf: f16 big-endian": ("_f16", gg_f16_big_endian),
}


@pytest.mark.parametrize("name", list(GG_MUTANTS))
def test_planted_gguf_mistake_fails_a_pin(name, monkeypatch):
    attr, fake = GG_MUTANTS[name]
    monkeypatch.setattr(ogg, attr, fake)
    failed = []
    for call in _gguf_pin_calls():
        try:
            call()
        except Exception as e:
            failed.append(type(e).__name__)
    assert failed, f"no pin caught the planted mistake '{name}'"


# --- planted mistakes in the K-quant part of the GGUF oracle ---

KQ_ORIG = {n: getattr(ogg, n) for n in ("parse_q4_k", "parse_q6_k", "dequant_k")}


def _kquant_pin_calls():
    calls = [ggpins.test_kquant_block_sizes_and_bits_per_weight, ggpins.test_hand_built_q4_k_super_block,
             ggpins.test_hand_built_q6_k_super_block]
    for fmt in ggpins.KFMTS:
        calls.append(lambda fmt=fmt: ggpins.test_kquant_element_order_matches_bit_addresses(fmt))
        calls.append(lambda fmt=fmt: ggpins.test_kquant_internal_layouts(fmt))
    return calls


def kq_scale_min_swapped_high(blocks, K):
    codes, d, dmin, sc, mn = KQ_ORIG["parse_q4_k"](blocks, K)
    s, m = sc.reshape(sc.shape[0], -1, 8).copy(), mn.reshape(mn.shape[0], -1, 8).copy()
    s[:, :, 4:], m[:, :, 4:] = m[:, :, 4:].copy(), s[:, :, 4:].copy()  # sub-blocks 4-7: scale and min exchanged
    return codes, d, dmin, s.reshape(sc.shape), m.reshape(mn.shape)


def kq_q4_k_runs_interleaved(blocks, K):
    codes, d, dmin, sc, mn = KQ_ORIG["parse_q4_k"](blocks, K)
    r = codes.reshape(codes.shape[0], -1, 2, 32)  # low / high nibbles as weights 2l / 2l+1
    return np.stack([r[:, :, 0], r[:, :, 1]], axis=3).reshape(codes.shape), d, dmin, sc, mn


def kq_q6_k_no_offset(blocks, K):
    codes, d, sc = KQ_ORIG["parse_q6_k"](blocks, K)
    return codes + 32, d, sc


def kq_q6_k_high_bits_reversed(blocks, K):
    codes, d, sc = KQ_ORIG["parse_q6_k"](blocks, K)
    u = (codes + 32).reshape(codes.shape[0], -1, 2, 4, 32)
    lo, hi = u & 15, u >> 4
    u = lo | (hi[:, :, :, ::-1, :] << 4)  # quarter k takes the bit pair of quarter 3 - k
    return u.reshape(codes.shape) - 32, d, sc


def kq_q4_k_min_added(blocks, fmt, K):
    w = KQ_ORIG["dequant_k"](blocks, fmt, K)
    if fmt == "q4_k":
        _, _, dmin, _, mn = ogg.parse_q4_k(blocks, K)
        w = w + 2.0 * dmin[:, np.arange(K) // 256] * mn[:, np.arange(K) // 32]
    return w


KQ_MUTANTS = {
    "q4_k: scale and min of sub-blocks 4-7 exchanged": ("parse_q4_k", kq_scale_min_swapped_high),
    "q4_k: nibbles of a run interleaved": ("parse_q4_k", kq_q4_k_runs_interleaved),
    "q6_k: codes without the -32": ("parse_q6_k", kq_q6_k_no_offset),
    "q6_k: high bit pairs in reverse order": ("parse_q6_k", kq_q6_k_high_bits_reversed),
    "q4_k: min added instead of subtracted": ("dequant_k", kq_q4_k_min_added),
}


@pytest.mark.parametrize("name", list(KQ_MUTANTS))
def test_planted_kquant_mistake_fails_a_pin(name, monkeypatch):
    attr, fake = KQ_MUTANTS[name]
    monkeypatch.setattr(ogg, attr, fake)
    failed = []
    for call in _kquant_pin_calls():
        try:
            call()
        except Exception as e:
            failed.append(type(e).__name__)
    assert failed, f"no pin caught the planted mistake '{name}'"


# --- token compaction ------------------------------------------------------------

import oracle.compaction as ocp  # noqa: E402
import test_oracle_compaction as cpins  # noqa: E402

_ORIG_MAPS = ocp.token_maps


def cp_order_ties_reversed(mask):
    cu, src, dst, _ = _ORIG_MAPS(mask)
    lengths = np.diff(cu)
    return cu, src, dst, np.lexsort((-np.arange(len(lengths)), -lengths))


def cp_order_shortest_first(mask):
    cu, src, dst, _ = _ORIG_MAPS(mask)
    lengths = np.diff(cu)
    return cu, src, dst, np.lexsort((np.arange(len(lengths)), lengths))


def cp_cu_inclusive(mask):
    cu, src, dst, order = _ORIG_MAPS(mask)
    return np.concatenate([cu[1:], cu[-1:]]), src, dst, order


def cp_src_column_major(mask):
    m = np.asarray(mask) != 0
    cu, _, _, order = _ORIG_MAPS(mask)
    B, S = m.shape
    flat = np.flatnonzero(m.T.reshape(-1))
    src = (flat % B) * S + flat // B  # the same tokens, position-major
    dst = np.full(B * S, -1)
    dst[src] = np.arange(src.size)
    return cu, src, dst, order


def cp_dst_masked_zero(mask):
    cu, src, dst, order = _ORIG_MAPS(mask)
    return cu, src, np.maximum(dst, 0), order


CP_MUTANTS = {
    "order: equal counts by descending index": cp_order_ties_reversed,
    "order: shortest first": cp_order_shortest_first,
    "cu: inclusive prefix": cp_cu_inclusive,
    "tok_src: positions before sequences": cp_src_column_major,
    "tok_dst: masked tokens map to 0": cp_dst_masked_zero,
}


@pytest.mark.parametrize("name", list(CP_MUTANTS))
def test_planted_compaction_mistake_fails_a_pin(name, monkeypatch):
    monkeypatch.setattr(ocp, "token_maps", CP_MUTANTS[name])
    failed = []
    for call in (cpins.test_hand_worked_mask, cpins.test_against_position_loops):
        try:
            call()
        except Exception as e:
            failed.append(type(e).__name__)
    assert failed, f"no pin caught the planted mistake '{name}'"
