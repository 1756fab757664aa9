"""Host-only checks of the C ABI: the library loads, exports every function
that include/rlx.h declares, and rejects bad arguments before touching the
GPU (no compute call is made here)."""
import ctypes
import os
import re

import pytest

import paper_2609_37916_amd as rlx

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(rlx.LIB_PATH):
        from paper_2609_37916_amd import _build
        _build.build_library()
    return rlx.lib()


def header_functions():
    text = open(os.path.join(ROOT, "include", "rlx.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rlx_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_function_is_exported(L):
    declared = header_functions()
    assert set(declared) == set(rlx.EXPORTS), declared
    for name in declared:
        assert getattr(L, name) is not None


def test_token_compaction_argument_errors(L):
    P = 4096  # an aligned stand-in address: validation rejects before any use
    f = L.rlx_mask_compaction
    assert f(None, 2, 8, P, P, P, None, None) == rlx.ERR_INVALID_ARG
    assert f(P, 2, 8, P, None, P, None, None) == rlx.ERR_INVALID_ARG
    assert f(P, 0, 8, P, P, P, None, None) == rlx.ERR_INVALID_ARG
    assert f(P, 2, 0, P, P, P, None, None) == rlx.ERR_INVALID_ARG
    assert f(P, 2, 513, P, P, P, None, None) == rlx.ERR_UNSUPPORTED
    assert f(P, 8193, 8, P, P, P, None, None) == rlx.ERR_UNSUPPORTED
    assert f(P, 257, 8, P, P, P, P, None) == rlx.ERR_UNSUPPORTED
    assert b"order" in L.rlx_last_error()
    g = L.rlx_encoder_token_maps
    assert g(None, 2, 8, P, P, P, None, None) == rlx.ERR_INVALID_ARG
    assert b"null handle" in L.rlx_last_error()


def test_version_string(L):
    assert "gfx950" in rlx.version()


def test_attention_argument_errors(L):
    f = L.rlx_masked_attention
    P = 4096  # an aligned stand-in address: validation rejects before any use
    assert f(None, P, P, 96, P, 32, 1, 8, 1, 32, rlx.BF16, rlx.MASK_NONE, None, 0, 1.0, None) == rlx.ERR_INVALID_ARG
    assert b"non-null" in L.rlx_last_error()
    assert f(P, P, P, 96, P, 32, 1, 8, 1, 32, rlx.BF16, rlx.MASK_CUSTOM, None, 0, 1.0, None) == rlx.ERR_INVALID_ARG
    assert b"key mask" in L.rlx_last_error()
    assert f(P, P, P, 96, P, 32, 1, 8, 1, 32, rlx.BF16, rlx.MASK_SLIDING_WINDOW, None, 0, 1.0, None) == \
        rlx.ERR_INVALID_ARG
    assert f(P, P, P, 192, P, 64, 1, 8, 1, 64, rlx.BF16, rlx.MASK_NONE, None, 0, 1.0, None) == rlx.ERR_UNSUPPORTED
    assert b"head_dim" in L.rlx_last_error()
    assert f(P, P, P, 96, P, 32, 1, 513, 1, 32, rlx.BF16, rlx.MASK_NONE, None, 0, 1.0, None) == rlx.ERR_UNSUPPORTED
    assert f(P, P, P, 96, P, 32, 1, 8, 1, 32, rlx.F16, rlx.MASK_NONE, None, 0, 1.0, None) == rlx.ERR_UNSUPPORTED
    assert f(P, P, P, 20, P, 32, 1, 8, 1, 32, rlx.BF16, rlx.MASK_NONE, None, 0, 1.0, None) == rlx.ERR_INVALID_ARG
    assert f(P + 2, P, P, 96, P, 32, 1, 8, 1, 32, rlx.BF16, rlx.MASK_NONE, None, 0, 1.0, None) == rlx.ERR_UNSUPPORTED
    assert f(P, P, P, 96, P, 32, -1, 8, 1, 32, rlx.BF16, rlx.MASK_NONE, None, 0, 1.0, None) == rlx.ERR_INVALID_ARG
    assert f(P, P, P, 96, P, 32, 1, 8, 1, 32, rlx.BF16, rlx.MASK_NONE, None, 0, float("nan"), None) == \
        rlx.ERR_INVALID_ARG
    # empty batch / sequence: a no-op that succeeds without touching the device
    assert f(P, P, P, 96, P, 32, 0, 8, 1, 32, rlx.BF16, rlx.MASK_NONE, None, 0, 1.0, None) == rlx.OK
    assert f(P, P, P, 96, P, 32, 3, 0, 1, 32, rlx.BF16, rlx.MASK_NONE, None, 0, 1.0, None) == rlx.OK
    assert L.rlx_last_error() == b""


def test_dequant_matmul_argument_errors(L):
    f = L.rlx_dequant_matmul
    P = 4096
    # (x, x_dt, M, K, w, scheme, scales, zeros, group, N, bias, residual, epi, y, y_dt, stream)
    assert f(P, rlx.BF16, 8, 96, P, rlx.Q_NONE, None, None, 32, 64, None, None, 0, P, rlx.BF16, None) == \
        rlx.ERR_UNSUPPORTED
    assert f(P, rlx.BF16, 8, 64, P, rlx.Q_NONE, None, None, 32, 64, None, None, rlx.EPI_BIAS, P, rlx.BF16, None) == \
        rlx.ERR_INVALID_ARG
    assert f(P, rlx.BF16, 8, 64, P, rlx.Q_NONE, None, None, 32, 64, P,
             None, rlx.EPI_BIAS_RESIDUAL, P, rlx.BF16, None) == \
        rlx.ERR_INVALID_ARG
    assert f(P, rlx.F32, 8, 64, P, rlx.Q_INT8_PER_CHANNEL, P, None, 32, 64, None, None, 0, P, rlx.F32, None) == \
        rlx.ERR_UNSUPPORTED
    assert f(P, rlx.BF16, 8, 64, P, rlx.Q_INT8_PER_CHANNEL, None, None, 32, 64, None, None, 0, P, rlx.BF16, None) == \
        rlx.ERR_INVALID_ARG
    assert f(P, rlx.BF16, 8, 64, P, rlx.Q_INT4_GROUP_ZP, P, P, 64, 64, None, None, 0, P, rlx.BF16, None) == \
        rlx.ERR_UNSUPPORTED
    assert f(P, rlx.BF16, 8, 64, P, rlx.Q_INT4_GROUP_ZP, P, None, 32, 64, None, None, 0, P, rlx.BF16, None) == \
        rlx.ERR_INVALID_ARG
    assert f(P, rlx.F16, 8, 64, P, rlx.Q_NONE, None, None, 32, 64, None, None, 0, P, rlx.BF16, None) == \
        rlx.ERR_UNSUPPORTED
    assert f(None, rlx.BF16, 8, 64, P, rlx.Q_NONE, None, None, 32, 64, None, None, 0, P, rlx.BF16, None) == \
        rlx.ERR_INVALID_ARG
    assert f(P, rlx.BF16, -1, 64, P, rlx.Q_NONE, None, None, 32, 64, None, None, 0, P, rlx.BF16, None) == \
        rlx.ERR_INVALID_ARG
    assert f(P, rlx.BF16, 0, 64, P, rlx.Q_NONE, None, None, 32, 64, None, None, 0, P, rlx.BF16, None) == rlx.OK
    # output dtype: bf16 x gives bf16 or f32, f32 x gives f32
    assert f(P, rlx.BF16, 8, 64, P, rlx.Q_NONE, None, None, 32, 64, None, None, 0, P, rlx.F16, None) == \
        rlx.ERR_UNSUPPORTED
    assert f(P, rlx.F32, 8, 64, P, rlx.Q_NONE, None, None, 32, 64, None, None, 0, P, rlx.BF16, None) == \
        rlx.ERR_UNSUPPORTED
    assert b"output dtype" in L.rlx_last_error()
    assert f(P, rlx.BF16, 0, 64, P, rlx.Q_NONE, None, None, 32, 64, None, None, 0, P, rlx.F32, None) == rlx.OK
    assert f(P, rlx.F32, 0, 64, P, rlx.Q_NONE, None, None, 32, 64, None, None, 0, P, rlx.F32, None) == rlx.OK
    assert L.rlx_dequant_unpack(P, rlx.Q_NONE, P, None, 32, 64, 64, P, None) == rlx.ERR_INVALID_ARG


def _cfg(**kw):
    base = dict(hidden=384, heads=12, head_dim=32, ffn=1536, layers=6, vocab=30522, max_pos=512, type_vocab=2,
                ln_eps=1e-12, dtype=rlx.BF16, quant=rlx.Q_NONE, group_size=32, input_kind=rlx.INPUT_IDS,
                output_kind=rlx.OUTPUT_POOLED, max_batch=32, max_seq=128, use_graph=1)
    base.update(kw)
    return rlx.EncoderConfig(**base)


def _weights(layers=6, **null):
    P = 4096
    arr = (rlx.LayerWeights * layers)()
    for L_ in arr:
        for f, _ in rlx.LayerWeights._fields_:
            if not f.endswith("_scales") and not f.endswith("_zeros"):
                setattr(L_, f, P)
    w = rlx.EncoderWeights(P, P, P, P, P, ctypes.cast(arr, ctypes.POINTER(rlx.LayerWeights)))
    for k, v in null.items():
        setattr(w, k, v)
    return w, arr


@pytest.mark.parametrize("kw,status,needle", [
    (dict(head_dim=64, heads=6), rlx.ERR_UNSUPPORTED, b"head_dim"),
    (dict(hidden=380), rlx.ERR_INVALID_ARG, b"hidden"),
    (dict(max_seq=1024), rlx.ERR_UNSUPPORTED, b"max_seq"),
    (dict(max_pos=64), rlx.ERR_UNSUPPORTED, b"max_pos"),
    (dict(dtype=rlx.F32, quant=rlx.Q_INT8_PER_CHANNEL), rlx.ERR_UNSUPPORTED, b"bf16"),
    (dict(quant=rlx.Q_INT4_GROUP_ZP, group_size=128), rlx.ERR_UNSUPPORTED, b"group"),
    (dict(dtype=rlx.F16), rlx.ERR_UNSUPPORTED, b"dtype"),
    (dict(layers=0), rlx.ERR_INVALID_ARG, b"positive"),
    (dict(max_batch=0), rlx.ERR_INVALID_ARG, b"max_batch"),
    (dict(ffn=1500), rlx.ERR_UNSUPPORTED, b"multiples of 64"),
])
def test_encoder_create_config_errors(L, kw, status, needle):
    w, _arr = _weights()
    h = ctypes.c_void_p()
    st = L.rlx_encoder_create(ctypes.byref(_cfg(**kw)), ctypes.byref(w), ctypes.byref(h))
    assert st == status
    assert needle in L.rlx_last_error()
    assert not h.value


def test_encoder_create_weight_errors(L):
    h = ctypes.c_void_p()
    w, _arr = _weights(word_emb=None)
    assert L.rlx_encoder_create(ctypes.byref(_cfg()), ctypes.byref(w), ctypes.byref(h)) == rlx.ERR_INVALID_ARG
    w, arr = _weights()
    arr[3].b1 = None
    assert L.rlx_encoder_create(ctypes.byref(_cfg()), ctypes.byref(w), ctypes.byref(h)) == rlx.ERR_INVALID_ARG
    assert b"layer 3" in L.rlx_last_error()
    w, arr = _weights()
    assert L.rlx_encoder_create(ctypes.byref(_cfg(quant=rlx.Q_INT8_PER_CHANNEL)), ctypes.byref(w),
                                ctypes.byref(h)) == rlx.ERR_INVALID_ARG
    assert b"scales" in L.rlx_last_error()
    assert L.rlx_encoder_create(None, ctypes.byref(w), ctypes.byref(h)) == rlx.ERR_INVALID_ARG


def test_encoder_forward_null_handle(L):
    assert L.rlx_encoder_forward(None, 4096, 4096, 1, 1, 4096, None) == rlx.ERR_INVALID_ARG
    L.rlx_encoder_destroy(None)


def test_scaled_matmul_argument_errors(L):
    f = L.rlx_scaled_matmul
    P = 4096  # aligned stand-in addresses: validation rejects before any use
    E4M3, E2M1 = rlx.MX_E4M3, rlx.MX_E2M1
    assert f(None, P, E4M3, P, P, E4M3, 8, 128, 128, P, None) == rlx.ERR_INVALID_ARG
    assert b"non-null" in L.rlx_last_error()
    assert f(P, P, 5, P, P, E4M3, 8, 128, 128, P, None) == rlx.ERR_INVALID_ARG
    assert f(P, P, E4M3, P, P, -1, 8, 128, 128, P, None) == rlx.ERR_INVALID_ARG
    assert f(P, P, E4M3, P, P, E2M1, -1, 128, 128, P, None) == rlx.ERR_INVALID_ARG
    assert f(P, P, E4M3, P, P, E2M1, 8, 0, 128, P, None) == rlx.ERR_INVALID_ARG
    assert f(P, P, E4M3, P, P, E2M1, 8, 192, 128, P, None) == rlx.ERR_UNSUPPORTED
    assert b"multiples of 128" in L.rlx_last_error()
    assert f(P, P, E4M3, P, P, E2M1, 8, 128, 96, P, None) == rlx.ERR_UNSUPPORTED
    assert f(P + 8, P, E4M3, P, P, E2M1, 8, 128, 128, P, None) == rlx.ERR_UNSUPPORTED
    assert f(P, P + 2, E4M3, P, P, E2M1, 8, 128, 128, P, None) == rlx.ERR_UNSUPPORTED
    assert b"aligned" in L.rlx_last_error()
    # M == 0: a no-op that succeeds without touching the device
    assert f(P, P, E4M3, P, P, E2M1, 0, 128, 128, P, None) == rlx.OK


def test_gguf_repack_argument_errors(L):
    """Rejected before any launch (fake, never dereferenced device addresses)."""
    p16, p2 = 0x10000, 0x10002
    st = L.rlx_gguf_repack(p16, 6, 64, 64, p16, p16, p16, None, None)  # Q5_0
    assert st == rlx.ERR_UNSUPPORTED and b"Q4_0" in L.rlx_last_error()
    assert L.rlx_gguf_repack(p16, 2, 64, 96, p16, p16, p16, None, None) == rlx.ERR_UNSUPPORTED  # K % 64
    assert L.rlx_gguf_repack(p16, 2, -1, 64, p16, p16, p16, None, None) == rlx.ERR_INVALID_ARG
    assert L.rlx_gguf_repack(p16, 2, 64, 64, p16, p16, None, None, None) == rlx.ERR_INVALID_ARG  # Q4_0 needs zeros
    assert L.rlx_gguf_repack(None, 8, 64, 64, p16, p16, None, None, None) == rlx.ERR_INVALID_ARG
    assert L.rlx_gguf_repack(p16 + 1, 2, 64, 64, p16, p16, p16, None, None) == rlx.ERR_UNSUPPORTED  # odd address
    assert L.rlx_gguf_repack(p16, 8, 64, 64, p2, p16, None, None, None) == rlx.ERR_UNSUPPORTED  # codes not 16-aligned
    assert L.rlx_gguf_repack(None, 2, 0, 64, None, None, None, None, None) == rlx.OK  # N == 0: nothing to do


def test_new_schemes_argument_errors(L):
    p16 = 0x10000
    # int4 min needs mins in `zeros`; the group schemes need group_size 32
    st = L.rlx_dequant_matmul(p16, rlx.BF16, 4, 64, p16, rlx.Q_INT4_GROUP_MIN, p16, None, 32, 64, None, None,
                              rlx.EPI_NONE, p16, rlx.BF16, None)
    assert st == rlx.ERR_INVALID_ARG
    st = L.rlx_dequant_matmul(p16, rlx.BF16, 4, 64, p16, rlx.Q_INT8_GROUP, p16, None, 64, 64, None, None,
                              rlx.EPI_NONE, p16, rlx.BF16, None)
    assert st == rlx.ERR_UNSUPPORTED
    st = L.rlx_dequant_matmul(p16, rlx.BF16, 4, 64, p16, 6, p16, p16, 32, 64, None, None, rlx.EPI_NONE, p16, rlx.BF16,
                              None)
    assert st == rlx.ERR_INVALID_ARG  # unknown scheme
    # int8 with a scale per 16 (GGUF Q6_K's layout): scales required, group size 16 only
    st = L.rlx_dequant_matmul(p16, rlx.BF16, 4, 64, p16, rlx.Q_INT8_GROUP16, None, None, 16, 64, None, None,
                              rlx.EPI_NONE, p16, rlx.BF16, None)
    assert st == rlx.ERR_INVALID_ARG
    st = L.rlx_dequant_matmul(p16, rlx.BF16, 4, 64, p16, rlx.Q_INT8_GROUP16, p16, None, 32, 64, None, None,
                              rlx.EPI_NONE, p16, rlx.BF16, None)
    assert st == rlx.ERR_UNSUPPORTED and b"group size 16" in L.rlx_last_error()
    # K-quant repack: K a multiple of 256; Q4_K needs the mins array
    assert L.rlx_gguf_repack(p16, rlx.GGUF_Q4_K, 64, 128, p16, p16, p16, None, None) == rlx.ERR_UNSUPPORTED
    assert L.rlx_gguf_repack(p16, rlx.GGUF_Q4_K, 64, 256, p16, p16, None, None, None) == rlx.ERR_INVALID_ARG
    assert L.rlx_gguf_repack(p16, rlx.GGUF_Q6_K, 64, 320, p16, p16, None, None, None) == rlx.ERR_UNSUPPORTED
    assert L.rlx_gguf_repack(p16, 13, 64, 256, p16, p16, p16, None, None) == rlx.ERR_UNSUPPORTED  # Q5_K


def test_encoder_forward_noalloc_argument_errors(L):
    """The allocation-free forward validates like create and forward, and
    rejects a batch whose workspace does not fit its static scratch, all
    before any HIP call."""
    f = L.rlx_encoder_forward_noalloc
    P = 4096
    w, _arr = _weights()
    cfg = _cfg()
    assert f(None, ctypes.byref(w), P, P, 4, 128, P, None) == rlx.ERR_INVALID_ARG
    assert f(ctypes.byref(_cfg(head_dim=64, heads=6)), ctypes.byref(w), P, P, 4, 128, P, None) == \
        rlx.ERR_UNSUPPORTED
    assert f(ctypes.byref(cfg), ctypes.byref(w), None, P, 4, 128, P, None) == rlx.ERR_INVALID_ARG
    assert f(ctypes.byref(cfg), ctypes.byref(w), P, P, 0, 128, P, None) == rlx.ERR_INVALID_ARG
    assert f(ctypes.byref(cfg), ctypes.byref(w), P, P, 1, 1024, P, None) == rlx.ERR_UNSUPPORTED
    # 64 x 512 bf16 tokens need far more than the 16 MiB scratch
    assert f(ctypes.byref(cfg), ctypes.byref(w), P, P, 64, 512, P, None) == rlx.ERR_UNSUPPORTED
    assert b"static scratch" in L.rlx_last_error()
    # max_batch / max_seq of the config do not limit it (only the scratch does)
    assert f(ctypes.byref(_cfg(max_batch=1, max_seq=8)), ctypes.byref(w), P, P, 64, 512, P, None) == \
        rlx.ERR_UNSUPPORTED
    assert b"static scratch" in L.rlx_last_error()
