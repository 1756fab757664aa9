"""GPU parity of the persistent encoder forward (one launch per forward, each
XCD working on its own run of sequences) through the C ABI, against the CPU
oracle and against the kernel-per-step forward of the same weights.

Besides the encoder parity tests (which take this path for every bf16
id-input pooled workload of at most 128 tokens), these cover what is specific
to it: the sync words are cleared by each launch for the next (many forwards
in a row with changing masks, eager and replayed from a HIP graph), batches
with fewer sequences than XCDs, empty and full-length sequences anywhere in
the batch, and the bounded waits never giving up (rlx_encoder_check).
Tolerance: the bf16 target, 2e-2 max-abs on the pooled embeddings.
"""
import os

import numpy as np
import pytest

import oracle
import workloads
from workloads.device import encoder_kwargs, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TOL = 2e-2


@pytest.fixture(scope="module")
def rlx():
    import paper_2609_37916_amd as m
    m.lib()
    return m


def _encoder(rlx, sp, weights, persistent=True, use_graph=False, max_batch=None):
    old = os.environ.get("RLX_PIPELINE")
    os.environ["RLX_PIPELINE"] = "1" if persistent else "0"
    try:
        enc = rlx.Encoder(**encoder_kwargs(sp, max_batch=max_batch, use_graph=use_graph), weights=weights)
    finally:
        if old is None:
            del os.environ["RLX_PIPELINE"]
        else:
            os.environ["RLX_PIPELINE"] = old
    return enc


def _forward(enc, inputs):
    out = enc.forward(inputs["input"], inputs["mask"])
    enc.check()
    return out.cpu().numpy()


def _err(got, ref):
    assert np.all(np.isfinite(got))
    return float(np.abs(got - ref).max())


@pytest.mark.parametrize("batch,seq,layers,lo,hi", [(32, 128, 6, 16, 128), (1, 128, 2, 128, 128), (3, 48, 2, 5, 48),
                                                   (7, 64, 3, 1, 64), (64, 128, 2, 8, 128), (256, 128, 1, 8, 128)])
def test_persistent_matches_oracle_and_kernel_per_step(rlx, batch, seq, layers, lo, hi):
    sp = workloads.spec("minilm_b32_s128_bf16", batch=batch, seq=seq, layers=layers, len_lo=lo, len_hi=hi)
    wl = workloads.make(sp, affine=True)
    weights, inputs = to_device(wl)
    enc = _encoder(rlx, sp, weights)
    assert enc.persistent, "a supported shape must take the persistent launch"
    got = _forward(enc, inputs)
    enc.close()
    ref_enc = _encoder(rlx, sp, weights, persistent=False)
    assert not ref_enc.persistent
    got_steps = _forward(ref_enc, inputs)
    ref_enc.close()
    rows = np.arange(batch) if batch <= 64 else np.random.default_rng(5).choice(batch, 24, replace=False)
    ref = oracle.encoder_forward(workloads.select_rows(wl, np.sort(rows)))
    e_oracle = _err(got[np.sort(rows)], ref)
    e_steps = _err(got, got_steps)
    print(f"B={batch} S={seq} layers={layers}: vs oracle {e_oracle:.3g}, vs kernel-per-step {e_steps:.3g}", flush=True)
    assert e_oracle <= TOL and e_steps <= TOL
    assert np.max(np.abs(np.linalg.norm(got, axis=1) - 1)) < 1e-3


def test_empty_and_full_sequences_anywhere(rlx):
    """Sequences with no token at the start, middle and end of the batch (and
    next to each other), full-length ones, and a mask with holes."""
    sp = workloads.spec("minilm_b32_s128_bf16", batch=20, seq=128, layers=2, len_lo=1, len_hi=128)
    wl = workloads.make(sp, affine=True)
    rng = np.random.default_rng(11)
    wl.mask[:, :] = (np.arange(128)[None] < wl.lengths[:, None]).astype(np.uint8)
    wl.mask[[0, 9, 10, 19]] = 0
    wl.mask[[3, 12]] = 1
    wl.mask[5] &= (rng.random(128) < 0.5).astype(np.uint8)
    wl.lengths = wl.mask.sum(axis=1)
    weights, inputs = to_device(wl)
    enc = _encoder(rlx, sp, weights)
    got = _forward(enc, inputs)
    enc.close()
    for b in (0, 9, 10, 19):
        assert np.all(got[b] == 0), f"sequence {b} has no token: zero vector"
    e = _err(got, oracle.encoder_forward(wl))
    print(f"empty/full/holes: vs oracle {e:.3g}", flush=True)
    assert e <= TOL


@pytest.mark.parametrize("use_graph", [False, True])
def test_many_forwards_with_changing_masks(rlx, use_graph):
    """Every launch clears the sync words it used for the next one: twelve
    forwards in a row, alternating three masks (different token counts, so
    different XCD runs and item counts), each compared to the oracle."""
    sp = workloads.spec("minilm_b32_s128_bf16", batch=24, seq=128, layers=2)
    wls = [workloads.make(workloads.spec("minilm_b32_s128_bf16", batch=24, seq=128, layers=2, len_lo=lo,
                                         len_hi=128))
           for lo in (16, 100, 1)]
    # same weights (same seed and draw order), different lengths: the weights of the first serve all
    weights, _ = to_device(wls[0])
    masks = [torch.from_numpy(w.mask).cuda() for w in wls]
    ids = [torch.from_numpy(w.ids).cuda() for w in wls]
    refs = [oracle.encoder_forward(w) for w in wls]
    enc = _encoder(rlx, sp, weights, use_graph=use_graph)
    assert enc.persistent
    outs = [torch.empty((24, 384), dtype=torch.float32, device="cuda") for _ in wls]
    for i in range(12):
        k = i % 3
        enc.forward(ids[k], masks[k], out=outs[k])
        if i % 3 == 2:
            enc.check()
            for j in range(3):
                e = _err(outs[j].cpu().numpy(), refs[j])
                assert e <= TOL, f"forward {i}, mask {j}: {e}"
    enc.check()
    enc.close()


def test_profiled_forward_takes_one_launch(rlx):
    """The profiling mode reports the persistent forward as one kernel class."""
    sp = workloads.spec("minilm_b32_s128_bf16", batch=8, layers=2)
    wl = workloads.make(sp)
    weights, inputs = to_device(wl)
    enc = _encoder(rlx, sp, weights)
    enc.set_profiling(True)
    out = enc.forward(inputs["input"], inputs["mask"])
    prof = enc.profile_read()
    enc.set_profiling(False)
    enc.check()
    assert list(prof) == ["encoder_pipe"] and prof["encoder_pipe"][0] == 1, prof
    assert _err(out.cpu().numpy(), oracle.encoder_forward(wl)) <= TOL
    enc.close()
