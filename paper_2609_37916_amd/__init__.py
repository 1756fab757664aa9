"""Python binding of librlx.so, the gfx950 MiniLM-L6-shaped encoder forward.

Argument marshalling only: every step of the computation runs in the HIP
kernels behind the C ABI declared in ``include/rlx.h``.  PyTorch supplies
device memory and the current stream.  If the library is not built, or a
tensor is not on the GPU, calls raise instead of computing anything
elsewhere.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Dict, List, Optional

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "librlx.so")

# enums (mirror include/rlx.h)
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_HIP, ERR_OOM = range(5)
F32, BF16, F16, I8, U4X2, I32, U8 = range(7)
MASK_NONE, MASK_CAUSAL, MASK_SLIDING_WINDOW, MASK_CUSTOM = range(4)
Q_NONE, Q_INT8_PER_CHANNEL, Q_INT4_GROUP_ZP, Q_INT8_GROUP, Q_INT4_GROUP_MIN, Q_INT8_GROUP16 = range(6)
GGUF_Q4_0, GGUF_Q4_1, GGUF_Q8_0, GGUF_Q4_K, GGUF_Q6_K = 2, 3, 8, 12, 14
GGUF_TYPES = {"q4_0": GGUF_Q4_0, "q4_1": GGUF_Q4_1, "q8_0": GGUF_Q8_0, "q4_k": GGUF_Q4_K, "q6_k": GGUF_Q6_K}
# bytes per block and weights per block
GGUF_BLOCK_BYTES = {GGUF_Q4_0: 18, GGUF_Q4_1: 20, GGUF_Q8_0: 34, GGUF_Q4_K: 144, GGUF_Q6_K: 210}
GGUF_BLOCK_WEIGHTS = {GGUF_Q4_0: 32, GGUF_Q4_1: 32, GGUF_Q8_0: 32, GGUF_Q4_K: 256, GGUF_Q6_K: 256}
EPI_NONE, EPI_BIAS, EPI_BIAS_GELU, EPI_BIAS_RESIDUAL = range(4)
MX_E4M3, MX_E5M2, MX_E2M3, MX_E3M2, MX_E2M1 = range(5)
MX_FORMAT_CODES = {"e4m3": MX_E4M3, "e5m2": MX_E5M2, "e2m3": MX_E2M3, "e3m2": MX_E3M2, "e2m1": MX_E2M1}
INPUT_IDS, INPUT_HIDDEN = range(2)
OUTPUT_POOLED, OUTPUT_HIDDEN = range(2)

STATUS_NAMES = {0: "RLX_OK", 1: "RLX_ERR_INVALID_ARG", 2: "RLX_ERR_UNSUPPORTED", 3: "RLX_ERR_HIP", 4: "RLX_ERR_OOM"}

# every symbol include/rlx.h declares
EXPORTS = ("rlx_masked_attention", "rlx_dequant_matmul", "rlx_dequant_unpack", "rlx_gguf_repack", "rlx_scaled_matmul",
           "rlx_encoder_create",
           "rlx_encoder_forward", "rlx_encoder_forward_noalloc", "rlx_encoder_destroy", "rlx_encoder_set_profiling",
           "rlx_encoder_profile_read", "rlx_encoder_check", "rlx_encoder_uses_persistent_forward",
           "rlx_mask_compaction", "rlx_encoder_token_maps", "rlx_last_error", "rlx_version")


class RlxError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status
        self.message = message


class EncoderConfig(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int), ("heads", ctypes.c_int), ("head_dim", ctypes.c_int), ("ffn", ctypes.c_int),
                ("layers", ctypes.c_int), ("vocab", ctypes.c_int), ("max_pos", ctypes.c_int),
                ("type_vocab", ctypes.c_int), ("ln_eps", ctypes.c_float), ("dtype", ctypes.c_int),
                ("quant", ctypes.c_int), ("group_size", ctypes.c_int), ("input_kind", ctypes.c_int),
                ("output_kind", ctypes.c_int), ("max_batch", ctypes.c_int), ("max_seq", ctypes.c_int),
                ("use_graph", ctypes.c_int)]


_vp = ctypes.c_void_p
_LAYER_FIELDS = []
for _nm in ("wqkv", "wo"):
    _LAYER_FIELDS += [(_nm, _vp), (_nm + "_scales", _vp), (_nm + "_zeros", _vp), ("b" + _nm[1:], _vp)]
_LAYER_FIELDS += [("ln1_gamma", _vp), ("ln1_beta", _vp)]
for _nm in ("w1", "w2"):
    _LAYER_FIELDS += [(_nm, _vp), (_nm + "_scales", _vp), (_nm + "_zeros", _vp), ("b" + _nm[1:], _vp)]
_LAYER_FIELDS += [("ln2_gamma", _vp), ("ln2_beta", _vp)]


class LayerWeights(ctypes.Structure):
    _fields_ = _LAYER_FIELDS


class EncoderWeights(ctypes.Structure):
    _fields_ = [("word_emb", _vp), ("pos_emb", _vp), ("type_emb", _vp), ("emb_ln_gamma", _vp),
                ("emb_ln_beta", _vp), ("layers", ctypes.POINTER(LayerWeights))]


_LIB = None


def lib() -> ctypes.CDLL:
    """Load librlx.so (raises if it has not been built)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() (or python "
                           f"paper_2609_37916_amd/_build.py) first")
    L = ctypes.CDLL(LIB_PATH)
    i64, i32, f32 = ctypes.c_int64, ctypes.c_int, ctypes.c_float
    L.rlx_masked_attention.argtypes = [_vp, _vp, _vp, i64, _vp, i64, i32, i32, i32, i32, i32, i32, _vp, i32, f32, _vp]
    L.rlx_dequant_matmul.argtypes = [_vp, i32, i32, i32, _vp, i32, _vp, _vp, i32, i32, _vp, _vp, i32, _vp, i32, _vp]
    L.rlx_dequant_unpack.argtypes = [_vp, i32, _vp, _vp, i32, i32, i32, _vp, _vp]
    L.rlx_scaled_matmul.argtypes = [_vp, _vp, i32, _vp, _vp, i32, i32, i32, i32, _vp, _vp]
    L.rlx_gguf_repack.argtypes = [_vp, i32, i32, i32, _vp, _vp, _vp, ctypes.POINTER(i32), _vp]
    L.rlx_encoder_create.argtypes = [ctypes.POINTER(EncoderConfig), ctypes.POINTER(EncoderWeights),
                                     ctypes.POINTER(_vp)]
    L.rlx_encoder_forward.argtypes = [_vp, _vp, _vp, i32, i32, _vp, _vp]
    L.rlx_encoder_forward_noalloc.argtypes = [ctypes.POINTER(EncoderConfig), ctypes.POINTER(EncoderWeights), _vp, _vp,
                                              i32, i32, _vp, _vp]
    L.rlx_mask_compaction.argtypes = [_vp, i32, i32, _vp, _vp, _vp, _vp, _vp]
    L.rlx_encoder_token_maps.argtypes = [_vp, i32, i32, _vp, _vp, _vp, _vp, _vp]
    L.rlx_encoder_check.argtypes = [_vp]
    L.rlx_encoder_uses_persistent_forward.argtypes = [_vp]
    L.rlx_encoder_uses_persistent_forward.restype = ctypes.c_int
    L.rlx_encoder_destroy.argtypes = [_vp]
    L.rlx_encoder_destroy.restype = None
    L.rlx_encoder_set_profiling.argtypes = [_vp, i32]
    L.rlx_encoder_profile_read.argtypes = [_vp, i32, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(i32),
                                           ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i32)]
    for nm in ("rlx_masked_attention", "rlx_dequant_matmul", "rlx_dequant_unpack", "rlx_gguf_repack", "rlx_scaled_matmul",
               "rlx_encoder_create", "rlx_encoder_forward", "rlx_encoder_forward_noalloc", "rlx_encoder_set_profiling",
               "rlx_encoder_profile_read", "rlx_encoder_check"):
        getattr(L, nm).restype = ctypes.c_int
    L.rlx_last_error.restype = ctypes.c_char_p
    L.rlx_last_error.argtypes = []
    L.rlx_version.restype = ctypes.c_char_p
    L.rlx_version.argtypes = []
    _LIB = L
    return L


def check(status: int) -> None:
    if status != OK:
        raise RlxError(status, lib().rlx_last_error().decode())


def version() -> str:
    return lib().rlx_version().decode()


# ---------------------------------------------------------------------------
# torch marshalling helpers
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("librlx works on GPU tensors only; got a tensor on " + str(t.device))
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _dt(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise ValueError(f"unsupported activation dtype {t.dtype} (bfloat16 or float32)")


# ---------------------------------------------------------------------------
# entry points
# ---------------------------------------------------------------------------

def masked_attention(q, k, v, *, B: int, S: int, heads: int, head_dim: int = 32, kind: int = MASK_CUSTOM,
                     key_mask=None, window: int = 0, scale: Optional[float] = None, row_stride: Optional[int] = None,
                     out=None, out_row_stride: Optional[int] = None, stream=None):
    """Masked multi-head attention over [B*S, row_stride] views (see rlx_masked_attention)."""
    torch = _torch()
    H = heads * head_dim
    row_stride = row_stride if row_stride is not None else q.stride(0) if q.dim() == 2 else H
    if out is None:
        out = torch.empty((B * S, H), dtype=q.dtype, device=q.device)
    out_row_stride = out_row_stride if out_row_stride is not None else out.stride(0)
    if scale is None:
        scale = 1.0 / math.sqrt(head_dim)
    check(lib().rlx_masked_attention(_ptr(q), _ptr(k), _ptr(v), row_stride, _ptr(out), out_row_stride, B, S, heads,
                                     head_dim, _dt(q), kind, _ptr(key_mask), window, float(scale), _stream(stream)))
    return out


def dequant_matmul(x, w, *, scheme: int = Q_NONE, scales=None, zeros=None, group_size: int = 32, N: Optional[int] = None,
                   bias=None, residual=None, epi: int = EPI_NONE, out=None, out_dtype=None, stream=None):
    """y = epi(x @ dequant(w)^T) (see rlx_dequant_matmul); y has x's dtype
    unless ``out_dtype`` (or ``out``) says float32."""
    torch = _torch()
    M, K = x.shape
    if N is None:
        N = w.shape[0]
    if out is None:
        out = torch.empty((M, N), dtype=out_dtype if out_dtype is not None else x.dtype, device=x.device)
    check(lib().rlx_dequant_matmul(_ptr(x), _dt(x), M, K, _ptr(w), scheme, _ptr(scales), _ptr(zeros), group_size, N,
                                   _ptr(bias), _ptr(residual), epi, _ptr(out), _dt(out), _stream(stream)))
    return out


def scaled_matmul(x, x_scales, fx, w, w_scales, fw, *, K: int, out=None, stream=None):
    """y = X W^T for block-scaled minifloat operands (see rlx_scaled_matmul).

    x, w: uint8 device tensors of packed rows ([M, K*bits/8], [N, K*bits/8]);
    x_scales, w_scales: uint8 [M, K/32], [N, K/32]; fx, fw: format names
    ("e4m3", "e5m2", "e2m3", "e3m2", "e2m1") or codes.  Returns float32 [M, N]."""
    torch = _torch()
    fx = MX_FORMAT_CODES.get(fx, fx)
    fw = MX_FORMAT_CODES.get(fw, fw)
    M, N = x.shape[0], w.shape[0]
    bits = {MX_E4M3: 8, MX_E5M2: 8, MX_E2M3: 6, MX_E3M2: 6, MX_E2M1: 4}
    if fx not in bits or fw not in bits:
        raise ValueError(f"unknown element format {fx!r} / {fw!r}")
    # the C ABI cannot see buffer sizes: check them here so no kernel reads past a tensor
    for t, rows, nbytes, what in ((x, M, K * bits[fx] // 8, "x"), (w, N, K * bits[fw] // 8, "w"),
                                  (x_scales, M, K // 32, "x_scales"), (w_scales, N, K // 32, "w_scales")):
        if t.dtype != torch.uint8 or not t.is_contiguous() or t.numel() != rows * nbytes:
            raise ValueError(f"{what}: expected a contiguous uint8 tensor of {rows} x {nbytes} bytes, "
                             f"got {t.dtype} {tuple(t.shape)}")
    if out is None:
        out = torch.empty((M, N), dtype=torch.float32, device=x.device)
    check(lib().rlx_scaled_matmul(_ptr(x), _ptr(x_scales), fx, _ptr(w), _ptr(w_scales), fw, M, N, K, _ptr(out),
                                  _stream(stream)))
    return out


def dequant_unpack(w, *, scheme: int, scales, zeros=None, group_size: int = 32, N: int, K: int, stream=None):
    """Dequantised weights as float32 [N, K] (see rlx_dequant_unpack)."""
    torch = _torch()
    out = torch.empty((N, K), dtype=torch.float32, device=w.device)
    check(lib().rlx_dequant_unpack(_ptr(w), scheme, _ptr(scales), _ptr(zeros), group_size, N, K, _ptr(out),
                                   _stream(stream)))
    return out


def _token_map_tensors(B: int, S: int, device, with_order: bool):
    torch = _torch()
    cu = torch.empty(B + 1, dtype=torch.int32, device=device)
    src = torch.full((B * S,), -2, dtype=torch.int32, device=device)
    dst = torch.empty(B * S, dtype=torch.int32, device=device)
    order = torch.empty(B, dtype=torch.int32, device=device) if with_order else None
    return cu, src, dst, order


def mask_compaction(mask, *, with_order: bool = True, stream=None):
    """Token compaction maps of a u8 mask [B, S] (see rlx_mask_compaction):
    (cu [B+1], tok_src [cu[B]], tok_dst [B*S], order [B] or None), int32."""
    torch = _torch()
    if mask.dtype != torch.uint8 or mask.dim() != 2 or not mask.is_contiguous():
        raise ValueError("mask: expected a contiguous uint8 [B, S] tensor")
    B, S = mask.shape
    cu, src, dst, order = _token_map_tensors(B, S, mask.device, with_order)
    check(lib().rlx_mask_compaction(_ptr(mask), B, S, _ptr(cu), _ptr(src), _ptr(dst), _ptr(order), _stream(stream)))
    (stream or torch.cuda.current_stream()).synchronize()  # the slice below reads cu[B]
    return cu, src[:int(cu[-1].item())], dst, order


def gguf_repack(blocks, gguf_type, *, N: int, K: int, stream=None):
    """GGUF blocks (uint8 device tensor of N * K/32 blocks, or N * K/256 for the
    K-quants) -> (scheme, codes, scales, zeros) for dequant_matmul (see
    rlx_gguf_repack); zeros is None for Q8_0 and Q6_K, whose group size is 32
    and 16."""
    torch = _torch()
    t = GGUF_TYPES.get(gguf_type, gguf_type)
    if t not in GGUF_BLOCK_BYTES:
        raise ValueError(f"unknown GGUF type {gguf_type!r}")
    # the C ABI cannot see buffer sizes: check the block tensor here so no kernel reads past it
    bw = GGUF_BLOCK_WEIGHTS[t]
    want = N * (K // bw) * GGUF_BLOCK_BYTES[t]
    if blocks.dtype != torch.uint8 or not blocks.is_contiguous() or blocks.numel() != want or K % bw:
        raise ValueError(f"blocks: expected a contiguous uint8 tensor of {want} bytes, got {blocks.dtype} "
                         f"{tuple(blocks.shape)}")
    dev = blocks.device
    int8_codes = t in (GGUF_Q8_0, GGUF_Q6_K)
    codes = torch.empty((N, K if int8_codes else K // 2), dtype=torch.int8 if int8_codes else torch.uint8, device=dev)
    scales = torch.empty((N, K // (16 if t == GGUF_Q6_K else 32)), dtype=torch.float16, device=dev)
    zeros = None if int8_codes else torch.empty((N, K // 32), dtype=torch.float16, device=dev)
    scheme = ctypes.c_int(-1)
    check(lib().rlx_gguf_repack(_ptr(blocks), t, N, K, _ptr(codes), _ptr(scales), _ptr(zeros), ctypes.byref(scheme),
                                _stream(stream)))
    return scheme.value, codes, scales, zeros


def _encoder_structs(keep: List, weights: Dict, *, hidden=384, heads=12, head_dim=32, ffn=1536, layers=6, vocab=30522,
                     max_pos=512, type_vocab=2, ln_eps=1e-12, dtype="bf16", quant="none", group_size=32,
                     input_kind="ids", output_kind="pooled", max_batch=32, max_seq=128, use_graph=False):
    """EncoderConfig, EncoderWeights and the per-layer array they point to,
    from keyword settings and a dict of device tensors (see Encoder); every
    tensor passed is appended to ``keep``."""
    cfg = EncoderConfig(hidden, heads, head_dim, ffn, layers, vocab, max_pos, type_vocab, ln_eps,
                        {"f32": F32, "bf16": BF16}[dtype],
                        {"none": Q_NONE, "int8": Q_INT8_PER_CHANNEL, "int4": Q_INT4_GROUP_ZP}[quant], group_size,
                        {"ids": INPUT_IDS, "hidden": INPUT_HIDDEN}[input_kind],
                        {"pooled": OUTPUT_POOLED, "hidden": OUTPUT_HIDDEN}[output_kind], max_batch, max_seq,
                        1 if use_graph else 0)

    def p(t):
        if t is None:
            return None
        keep.append(t)
        return _ptr(t)

    lw_arr = (LayerWeights * layers)()
    for i, lw in enumerate(weights["layers"]):
        L = lw_arr[i]
        for nm in ("wqkv", "wo", "w1", "w2"):
            setattr(L, nm, p(lw[nm]))
            setattr(L, nm + "_scales", p(lw.get(nm + "_scales")))
            setattr(L, nm + "_zeros", p(lw.get(nm + "_zeros")))
        L.bqkv, L.bo, L.b1, L.b2 = p(lw["bqkv"]), p(lw["bo"]), p(lw["b1"]), p(lw["b2"])
        L.ln1_gamma, L.ln1_beta = p(lw["ln1_g"]), p(lw["ln1_b"])
        L.ln2_gamma, L.ln2_beta = p(lw["ln2_g"]), p(lw["ln2_b"])
    w = EncoderWeights(p(weights.get("word")), p(weights.get("pos")), p(weights.get("type")),
                       p(weights.get("emb_gamma")), p(weights.get("emb_beta")),
                       ctypes.cast(lw_arr, ctypes.POINTER(LayerWeights)))
    keep.append(lw_arr)
    return cfg, w


def encoder_forward_noalloc(inp, mask, *, weights: Dict, out=None, stream=None, **settings):
    """One encoder forward without a handle and without any device allocation
    by the library (see rlx_encoder_forward_noalloc); ``settings`` are the
    Encoder keyword settings."""
    torch = _torch()
    keep: List = []
    cfg, w = _encoder_structs(keep, weights, **settings)
    B, S = mask.shape
    hidden = settings.get("hidden", 384)
    if out is None:
        shape = (B, hidden) if settings.get("output_kind", "pooled") == "pooled" else (B, S, hidden)
        out = torch.empty(shape, dtype=torch.float32, device=mask.device)
    check(lib().rlx_encoder_forward_noalloc(ctypes.byref(cfg), ctypes.byref(w), _ptr(inp), _ptr(mask), B, S, _ptr(out),
                                            _stream(stream)))
    return out


class Encoder:
    """A compiled encoder: weights bound once, forward run many times.

    ``weights`` maps names to device tensors: word, pos, type, emb_gamma,
    emb_beta (id input), and ``layers``: a list of dicts with wqkv, bqkv, wo,
    bo, ln1_g, ln1_b, w1, b1, w2, b2, ln2_g, ln2_b and, for quantised weights,
    ``<name>_scales`` / ``<name>_zeros``.  The tensors are kept alive by the
    object.
    """

    def __init__(self, *, hidden=384, heads=12, head_dim=32, ffn=1536, layers=6, vocab=30522, max_pos=512,
                 type_vocab=2, ln_eps=1e-12, dtype="bf16", quant="none", group_size=32, input_kind="ids",
                 output_kind="pooled", max_batch=32, max_seq=128, use_graph=False, weights: Dict = None):
        self._keep: List = []
        cfg, w = _encoder_structs(self._keep, weights, hidden=hidden, heads=heads, head_dim=head_dim, ffn=ffn,
                                  layers=layers, vocab=vocab, max_pos=max_pos, type_vocab=type_vocab, ln_eps=ln_eps,
                                  dtype=dtype, quant=quant, group_size=group_size, input_kind=input_kind,
                                  output_kind=output_kind, max_batch=max_batch, max_seq=max_seq, use_graph=use_graph)
        self.cfg = cfg
        self.hidden = hidden
        self.output_kind = output_kind
        h = _vp()
        check(lib().rlx_encoder_create(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(h)))
        self._h = h

    def forward(self, inp, mask, out=None, stream=None):
        torch = _torch()
        B, S = mask.shape
        if out is None:
            shape = (B, self.hidden) if self.output_kind == "pooled" else (B, S, self.hidden)
            out = torch.empty(shape, dtype=torch.float32, device=mask.device)
        check(lib().rlx_encoder_forward(self._h, _ptr(inp), _ptr(mask), B, S, _ptr(out), _stream(stream)))
        return out

    __call__ = forward

    @property
    def persistent(self) -> bool:
        """True when supported forwards run as one persistent launch."""
        return bool(lib().rlx_encoder_uses_persistent_forward(self._h))

    def token_maps(self, B: int, S: int, *, with_order: bool = True, stream=None):
        """The token compaction maps of this handle's most recent forward of
        B x S (see rlx_encoder_token_maps), as for mask_compaction."""
        torch = _torch()
        cu, src, dst, order = _token_map_tensors(B, S, torch.device("cuda", torch.cuda.current_device()), with_order)
        check(lib().rlx_encoder_token_maps(self._h, B, S, _ptr(cu), _ptr(src), _ptr(dst), _ptr(order),
                                           _stream(stream)))
        (stream or torch.cuda.current_stream()).synchronize()  # the slice below reads cu[B]
        return cu, src[:int(cu[-1].item())], dst, order

    def check(self) -> None:
        """Waits for the last forward; raises if a wait of the persistent launch gave up."""
        check(lib().rlx_encoder_check(self._h))

    def set_profiling(self, enable: bool) -> None:
        check(lib().rlx_encoder_set_profiling(self._h, 1 if enable else 0))

    def profile_read(self) -> Dict[str, tuple]:
        n = ctypes.c_int(0)
        cap = 32
        names = (ctypes.c_char_p * cap)()
        launches = (ctypes.c_int * cap)()
        ms = (ctypes.c_double * cap)()
        check(lib().rlx_encoder_profile_read(self._h, cap, names, launches, ms, ctypes.byref(n)))
        return {names[i].decode(): (launches[i], ms[i]) for i in range(min(n.value, cap))}

    def close(self) -> None:
        if getattr(self, "_h", None):
            lib().rlx_encoder_destroy(self._h)
            self._h = None
            self._keep.clear()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
