"""Seeded synthetic inputs for the MiniLM-L6-shaped encoder forward.

This module is shared by the CPU oracle (``oracle/``) and by the HIP path
(tests and ``bench.py``).  It draws random numbers and lays them out; it holds
none of the encoder's arithmetic.  Two input-preparation steps live here
because they produce *inputs*, not results:

* rounding fp32 draws to bfloat16-representable values (round to nearest,
  ties to even on the top 16 bits of the IEEE-754 single) for the bf16 path;
* offline weight-only quantisation (int8 symmetric per output channel; int4
  with group-wise fp16 scale and zero-point, packed two per byte).  The
  dequantisation that the forward pass performs lives separately in the
  oracle and in the HIP kernels.

The model is the one the paper benchmarks in its inference evaluation
(Section VIII-B): all-MiniLM-L6-v2, hidden 384, 6 layers, sequence length
128, synthetic inputs.  Trained weights are not used; N(0, 0.02) weights of
the same shapes stand in for them.  Draw order and seeds are fixed so that a
workload is reproduced bit for bit from its name.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

# MiniLM-L6 (BERT-style) dimensions.
HIDDEN = 384
HEADS = 12
HEAD_DIM = 32
FFN = 1536
LAYERS = 6
VOCAB = 30522
MAX_POS = 512
TYPE_VOCAB = 2
LN_EPS = 1e-12
INT4_GROUP = 32

LINEAR_NAMES = ("wqkv", "wo", "w1", "w2")


@dataclass(frozen=True)
class Spec:
    """Shape and distribution recipe of one workload."""

    name: str
    batch: int
    seq: int
    layers: int
    dtype: str            # "f32" | "bf16"  (activation / unquantised weight type)
    input_kind: str       # "ids" | "hidden"
    output_kind: str      # "pooled" | "hidden"
    len_lo: int
    len_hi: int
    seed: int
    quant: str = "none"   # "none" | "int8" | "int4"
    full_rows: int = 0    # trailing rows whose length is exactly ``seq``
    hidden: int = HIDDEN
    heads: int = HEADS
    ffn: int = FFN
    vocab: int = VOCAB
    max_pos: int = MAX_POS
    type_vocab: int = TYPE_VOCAB
    eps: float = LN_EPS
    group: int = INT4_GROUP

    @property
    def head_dim(self) -> int:
        return self.hidden // self.heads

    @property
    def tokens(self) -> int:
        return self.batch * self.seq


SWEEP_BATCHES = (1, 4, 16, 64, 256)


def _registry() -> Dict[str, Spec]:
    r: Dict[str, Spec] = {}
    # One post-LN layer in fp32 on N(0,1) hidden input; outputs hidden states.
    r["layer_f32_b2_s16"] = Spec("layer_f32_b2_s16", 2, 16, 1, "f32", "hidden", "hidden", 4, 16, seed=1)
    # The headline workload: batch 32, sequence 128, bf16, pooled + L2-normalised.
    r["minilm_b32_s128_bf16"] = Spec("minilm_b32_s128_bf16", 32, 128, LAYERS, "bf16", "ids", "pooled", 16, 128, seed=2)
    # Batch sweep at sequence 128 in fp32 and bf16 (both dtypes share the seed).
    for b in SWEEP_BATCHES:
        for dt in ("f32", "bf16"):
            n = f"minilm_b{b}_s128_{dt}"
            r[n] = Spec(n, b, 128, LAYERS, dt, "ids", "pooled", 8, 128, seed=3000 + b)
    # Long sequences: half the rows U[64,512], half exactly 512.
    r["minilm_b8_s512_bf16"] = Spec("minilm_b8_s512_bf16", 8, 512, LAYERS, "bf16", "ids", "pooled", 64, 512,
                                    seed=4, full_rows=4)
    # Weight-only quantised linears, bf16 activations.
    for q in ("int8", "int4"):
        n = f"minilm_b32_s128_{q}"
        r[n] = Spec(n, 32, 128, LAYERS, "bf16", "ids", "pooled", 16, 128, seed=5, quant=q)
        # the small-batch regime of the quantised encoder (lengths as the batch sweep)
        for b in (1, 4):
            n = f"minilm_b{b}_s128_{q}"
            r[n] = Spec(n, b, 128, LAYERS, "bf16", "ids", "pooled", 8, 128, seed=3000 + b, quant=q)
    return r


REGISTRY: Dict[str, Spec] = _registry()

# The five workload families, in the order they are usually quoted.
PARITY_CONFIGS = (
    "layer_f32_b2_s16",
    "minilm_b32_s128_bf16",
    *(f"minilm_b{b}_s128_{dt}" for b in SWEEP_BATCHES for dt in ("f32", "bf16")),
    "minilm_b8_s512_bf16",
    "minilm_b32_s128_int8",
    "minilm_b32_s128_int4",
)


def spec(name: str, **overrides) -> Spec:
    """Look up a named workload; keyword overrides make a derived (e.g. smaller) one."""
    base = REGISTRY[name]
    if not overrides:
        return base
    d = dict(base.__dict__)
    d.update(overrides)
    if "name" not in overrides:
        d["name"] = base.name + "+" + ",".join(f"{k}={v}" for k, v in sorted(overrides.items()))
    return Spec(**d)


# ---------------------------------------------------------------------------
# input preparation helpers (no encoder arithmetic)
# ---------------------------------------------------------------------------

def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 -> nearest bfloat16 value (ties to even), returned as fp32.

    bfloat16 is the upper half of an IEEE-754 binary32; rounding adds
    0x7FFF plus the lowest kept bit before truncating the low 16 bits.
    Inputs here are finite draws, so NaN/Inf handling is not needed.
    """
    a = np.ascontiguousarray(x, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).reshape(a.shape)


def _rne(x: np.ndarray) -> np.ndarray:
    return np.rint(x)  # numpy rounds half to even


def quantize_int8_per_channel(w: np.ndarray):
    """Symmetric per-output-channel int8: s_n = fp16(max_k |W_nk| / 127),
    q = clamp(rne(W / s_n), -127, 127) using the fp16-rounded scale."""
    w = np.asarray(w, dtype=np.float32)
    amax = np.abs(w).max(axis=1)
    s16 = (amax / 127.0).astype(np.float16)
    s16 = np.where(s16 == 0, np.float16(1.0), s16)
    s = s16.astype(np.float64)[:, None]
    q = np.clip(_rne(w.astype(np.float64) / s), -127, 127).astype(np.int8)
    return q, s16


def quantize_int4_grouped(w: np.ndarray, group: int = INT4_GROUP):
    """Asymmetric int4 with a fp16 scale and fp16 (integer-valued) zero-point per
    group of ``group`` consecutive k.  Codes are unsigned 0..15, packed two per
    byte: byte j of a row holds k = 2j in its low nibble and k = 2j+1 in its
    high nibble."""
    w = np.asarray(w, dtype=np.float32)
    n, k = w.shape
    assert k % group == 0 and group % 2 == 0
    g = w.reshape(n, k // group, group).astype(np.float64)
    mn = g.min(axis=2)
    mx = g.max(axis=2)
    s16 = ((mx - mn) / 15.0).astype(np.float16)
    flat = (mx == mn) | (s16 == 0)
    s16 = np.where(flat, np.float16(1.0), s16)
    s = s16.astype(np.float64)
    z16 = np.clip(_rne(-mn / s), 0, 15).astype(np.float16)
    z16 = np.where(flat, np.float16(0.0), z16)
    z = z16.astype(np.float64)
    q = np.clip(_rne(g / s[:, :, None]) + z[:, :, None], 0, 15).astype(np.uint8).reshape(n, k)
    packed = (q[:, 0::2] | (q[:, 1::2] << 4)).astype(np.uint8)
    return packed, s16, z16


# ---------------------------------------------------------------------------
# workload generation
# ---------------------------------------------------------------------------

@dataclass
class Workload:
    spec: Spec
    lengths: np.ndarray                   # int64 [B]
    mask: np.ndarray                      # uint8 [B,S], 1 = valid token (right-padded)
    ids: Optional[np.ndarray]             # int32 [B,S] (input_kind == "ids"); padded ids are 0
    hidden_in: Optional[np.ndarray]       # float32 [B,S,H] (input_kind == "hidden")
    emb: Dict[str, np.ndarray]            # word, pos, type (float32, bf16-exact on the bf16 path), gamma, beta
    layers: List[Dict[str, np.ndarray]]   # per-layer float32 arrays (dequantised values on quantised paths)
    quant: List[Dict[str, np.ndarray]] = field(default_factory=list)  # per-layer codes/scales/zeros


def _lengths(rng, sp: Spec) -> np.ndarray:
    n_rand = sp.batch - sp.full_rows
    lens = rng.integers(sp.len_lo, sp.len_hi + 1, size=n_rand)
    return np.concatenate([lens, np.full(sp.full_rows, sp.seq)]).astype(np.int64)


def make(name_or_spec, affine: bool = False) -> Workload:
    """Build a workload from its name (or a Spec).

    Draw order (numpy default_rng(seed)): lengths, ids (or hidden input), word,
    position, type embeddings, embedding-LN affine noise, then per layer
    Wq, bq, Wk, bk, Wv, bv, Wo, bo, LN1 (gamma, beta), W1, b1, W2, b2,
    LN2 (gamma, beta).  Biases and LN affine noise are always drawn; unless
    ``affine`` they are replaced by 0 (biases, beta) and 1 (gamma), so both
    variants share every weight matrix.
    """
    sp = name_or_spec if isinstance(name_or_spec, Spec) else spec(name_or_spec)
    rng = np.random.default_rng(sp.seed)
    H, F, B, S = sp.hidden, sp.ffn, sp.batch, sp.seq
    bf16 = sp.dtype == "bf16"

    def wdraw(*shape, std=0.02):
        return rng.normal(0.0, std, size=shape).astype(np.float32)

    def act_store(a):  # storage rounding of an unquantised weight / table
        return round_to_bf16(a) if bf16 else a

    def bias(n):
        b = wdraw(n)
        return b if affine else np.zeros(n, np.float32)

    def ln_params():
        g = rng.normal(0.0, 0.1, size=H).astype(np.float32)
        be = rng.normal(0.0, 0.1, size=H).astype(np.float32)
        if affine:
            return (1.0 + g).astype(np.float32), be
        return np.ones(H, np.float32), np.zeros(H, np.float32)

    lengths = _lengths(rng, sp)
    mask = (np.arange(S)[None, :] < lengths[:, None]).astype(np.uint8)
    ids = hidden_in = None
    if sp.input_kind == "ids":
        ids = rng.integers(1000, sp.vocab, size=(B, S)).astype(np.int32)
        ids[mask == 0] = 0
        word = act_store(wdraw(sp.vocab, H))
        pos = act_store(wdraw(sp.max_pos, H))
        typ = act_store(wdraw(sp.type_vocab, H))
        eg, eb = ln_params()
        emb = dict(word=word, pos=pos, type=typ, gamma=eg, beta=eb)
    else:
        hidden_in = rng.normal(0.0, 1.0, size=(B, S, H)).astype(np.float32)
        hidden_in = act_store(hidden_in)
        emb = {}

    layers, quant = [], []
    for _ in range(sp.layers):
        wq, bq = wdraw(H, H), bias(H)
        wk, bk = wdraw(H, H), bias(H)
        wv, bv = wdraw(H, H), bias(H)
        wo, bo = wdraw(H, H), bias(H)
        g1, be1 = ln_params()
        w1, b1 = wdraw(F, H), bias(F)
        w2, b2 = wdraw(H, F), bias(H)
        g2, be2 = ln_params()
        lw = dict(wqkv=np.concatenate([wq, wk, wv], axis=0), bqkv=np.concatenate([bq, bk, bv]),
                  wo=wo, bo=bo, ln1_g=g1, ln1_b=be1, w1=w1, b1=b1, w2=w2, b2=b2, ln2_g=g2, ln2_b=be2)
        if sp.quant == "none":
            for nm in LINEAR_NAMES:
                lw[nm] = act_store(lw[nm])
        else:
            qd = {}
            for nm in LINEAR_NAMES:
                if sp.quant == "int8":
                    q, s = quantize_int8_per_channel(lw[nm])
                    qd[nm] = dict(q=q, scales=s)
                else:
                    q, s, z = quantize_int4_grouped(lw[nm], sp.group)
                    qd[nm] = dict(q=q, scales=s, zeros=z)
                lw[nm] = None  # filled with dequantised values by the consumer's own dequant
            quant.append(qd)
        layers.append(lw)
    return Workload(sp, lengths, mask, ids, hidden_in, emb, layers, quant)


def with_padding_extended(wl: Workload, extra: int) -> Workload:
    """Same valid tokens, ``extra`` more padded positions per row (ids 0, mask 0)."""
    sp = spec(wl.spec.name) if wl.spec.name in REGISTRY else wl.spec
    sp = Spec(**{**wl.spec.__dict__, "seq": wl.spec.seq + extra, "name": wl.spec.name + f"+pad{extra}"})
    B, S = wl.mask.shape
    mask = np.zeros((B, S + extra), np.uint8)
    mask[:, :S] = wl.mask
    ids = hidden_in = None
    if wl.ids is not None:
        ids = np.zeros((B, S + extra), np.int32)
        ids[:, :S] = wl.ids
    if wl.hidden_in is not None:
        hidden_in = np.zeros((B, S + extra, wl.hidden_in.shape[2]), np.float32)
        hidden_in[:, :S] = wl.hidden_in
    return Workload(sp, wl.lengths.copy(), mask, ids, hidden_in, wl.emb, wl.layers, wl.quant)


def select_rows(wl: Workload, rows) -> Workload:
    """The sub-workload of the given sequences (same weights).  Sequences are
    independent in the encoder, so this is how a large batch is checked on a
    sample of its rows."""
    rows = np.asarray(rows)
    sp = Spec(**{**wl.spec.__dict__, "batch": len(rows), "full_rows": 0, "name": wl.spec.name + f"[{len(rows)} rows]"})
    return Workload(sp, wl.lengths[rows].copy(), wl.mask[rows].copy(),
                    None if wl.ids is None else wl.ids[rows].copy(),
                    None if wl.hidden_in is None else wl.hidden_in[rows].copy(), wl.emb, wl.layers, wl.quant)
