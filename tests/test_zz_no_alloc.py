"""rlx_encoder_forward_noalloc (the handle-free forward whose workspace is the
library's static scratch) against rlx_encoder_forward on the same weights and
inputs, through the C ABI: two calls in a row per case, the second with a
smaller input, each checked against the handle's forward and against the
oracle with the target tolerances (fp32 1e-4, bf16 2e-2, int8/int4 5e-2 on the
final outputs).  The handle's bf16 forward folds the LayerNorms into derived
weights while the allocation-free one runs them as kernels, so the two agree
up to bf16 rounding, within the same bound."""
import numpy as np
import pytest

import oracle
import workloads
from workloads.device import encoder_kwargs, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TOL = {"f32": 1e-4, "bf16": 2e-2, "int8": 5e-2, "int4": 5e-2}


@pytest.fixture(scope="module")
def rlx():
    import paper_2609_37916_amd as m
    m.lib()
    return m


def _valid(out, wl):
    """Pooled rows, or the valid tokens of hidden-state rows."""
    if wl.spec.output_kind == "hidden":
        return np.concatenate([out[b, :L] for b, L in enumerate(wl.lengths) if L > 0])
    return out


# (first call, second call): the second is smaller in batch and sequence
CASES = {
    "bf16_ids_pooled": (dict(name="minilm_b32_s128_bf16", batch=6, layers=3),
                        dict(name="minilm_b32_s128_bf16", batch=3, seq=48, layers=3, len_lo=5, len_hi=48)),
    "f32_hidden_in_out": (dict(name="layer_f32_b2_s16", batch=4, seq=32, len_lo=3, len_hi=32),
                          dict(name="layer_f32_b2_s16", batch=2, seq=16)),
    "int8_ids_pooled": (dict(name="minilm_b32_s128_int8", batch=5, seq=96, layers=2, len_lo=10, len_hi=96),
                        dict(name="minilm_b32_s128_int8", batch=2, seq=40, layers=2, len_lo=10, len_hi=40)),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_noalloc_forward_matches_handle_forward(rlx, case):
    for i, kw in enumerate(CASES[case]):
        kw = dict(kw)
        sp = workloads.spec(kw.pop("name"), **kw)
        wl = workloads.make(sp, affine=True)
        weights, inputs = to_device(wl)
        settings = encoder_kwargs(sp)
        print(f"case {case} call {i}: B={sp.batch} S={sp.seq} layers={sp.layers} {sp.dtype} {sp.quant}", flush=True)
        got = rlx.encoder_forward_noalloc(inputs["input"], inputs["mask"], weights=weights, **settings)
        torch.cuda.synchronize()
        got = got.cpu().numpy()
        enc = rlx.Encoder(**settings, weights=weights)
        ref_handle = enc.forward(inputs["input"], inputs["mask"])
        torch.cuda.synchronize()
        ref_handle = ref_handle.cpu().numpy()
        enc.close()
        ref = oracle.encoder_forward(wl)
        tol = TOL[sp.quant] if sp.quant != "none" else TOL[sp.dtype]
        assert np.all(np.isfinite(got))
        if sp.output_kind == "hidden":
            for b, L in enumerate(wl.lengths):
                assert np.all(got[b, L:] == 0), "padded rows must be zero"
        e_handle = float(np.abs(_valid(got, wl) - _valid(ref_handle, wl)).max())
        e_oracle = float(np.abs(_valid(got, wl) - _valid(ref, wl)).max())
        print(f"  max-abs vs rlx_encoder_forward {e_handle:.3g}, vs oracle {e_oracle:.3g} (tolerance {tol})",
              flush=True)
        assert e_handle <= tol and e_oracle <= tol
