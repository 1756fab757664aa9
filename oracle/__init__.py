"""CPU oracle for the MiniLM-L6-shaped encoder forward -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never calls it and shares no code with it; the two meet
only at the seeded inputs drawn by ``workloads``.

Everything here is a plain, slow, float64 restatement of what the forward pass
computes, step by step, in the order the hot path runs it:

  embedding gather + LayerNorm, then per layer: QKV projection, masked
  multi-head attention, output projection + residual, LayerNorm, FFN up +
  erf-GELU, FFN down + residual, LayerNorm; finally masked mean-pooling and
  L2 normalisation.  Weight-only int8 / int4 dequantisation supplies the
  linear weights on the quantised path.

The paper (RLX, arxiv 2609.37916) names the model and its primitives --
masked attention parameterised by an explicit MaskKind (Section III-A),
Op::DequantMatMul (Sections III-A and VI), F32 accumulation over BF16
(Section III-B, numeric precision), the fused attention block and the strided
Narrow x3 -> Attention pattern (Section III-B) -- and benchmarks the forward
of all-MiniLM-L6-v2 (Section VIII-B), but prints no formula for the encoder.
The layer-level definitions are the standard post-LN BERT encoder; every point
where a reading had to be chosen is listed in the module docstrings below.

``oracle.mx`` is the block-scaled minifloat matmul of the ScaledMatMul path
(FP8 / FP6 / FP4 elements with E8M0 block scales), decoded from the format
definitions and multiplied in float64.

``oracle.gguf`` reads the GGUF Q4_0 / Q4_1 / Q8_0 weight blocks (and the int8
group and int4 min layouts they map onto) into float64 weights.

``oracle.compaction`` lists a padded batch's real tokens (the index maps every
forward computes before its row-local steps).

Pins (tests/test_oracle_*.py) tie each function to something other than
itself: brute force on tiny inputs, closed forms, invariants, library special
cases (torch SDPA, nn.TransformerEncoderLayer, transformers.BertModel in
float64), and bit loops for the nibble unpacking.
"""
from .encoder import (  # noqa: F401
    MASK_NONE, MASK_CAUSAL, MASK_SLIDING_WINDOW, MASK_CUSTOM,
    layer_norm, gelu, linear, visible_keys, attention_probs, masked_attention,
    embed, encoder_layer, mean_pool_l2, encoder_forward, layer_weights,
)
from .quant import unpack_int4, dequant_int8, dequant_int4  # noqa: F401
from . import mx  # noqa: F401
from . import gguf  # noqa: F401
from . import compaction  # noqa: F401
