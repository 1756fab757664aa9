"""GPU bit-exactness of token compaction, the index work every forward starts
with, through the C ABI against oracle.compaction:

* rlx_mask_compaction runs the standalone mask-scan kernel (the one a forward
  uses for hidden-state input and for masks of more than 16384 entries) on
  every row-length class it specialises (up to 64, 128, 256 and 512
  positions) and on batches that need more than one pass of its waves;
* rlx_encoder_token_maps returns the maps a forward actually used: the
  embedding kernel's own scan for small id-input masks, the mask-scan kernel
  for large ones and for hidden-state input.

Masks mix right-padded rows, rows with holes, empty and full rows; nonzero
bytes other than 1 count as real tokens.  cu, the tok_src entries that are
defined, every tok_dst entry and the order must equal the oracle's exactly.
"""
import numpy as np
import pytest

import oracle
import workloads
from workloads.device import encoder_kwargs, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def rlx():
    import paper_2609_37916_amd as m
    m.lib()
    return m


def _mask(B, S, seed):
    """Right-padded rows of random length, a third of them with holes, an empty
    row, a full row, and real-token bytes drawn from 1..255."""
    rng = np.random.default_rng(seed)
    lengths = rng.integers(0, S + 1, B)
    m = (np.arange(S)[None, :] < lengths[:, None]).astype(np.uint8)
    holes = rng.random((B, S)) < 0.3
    rows = rng.random(B) < 1 / 3
    m[rows[:, None] & holes] = 0
    m[rng.integers(0, B)] = 0
    m[rng.integers(0, B)] = 1
    return m * rng.integers(1, 256, (B, S)).astype(np.uint8)


def _check(got, mask, what):
    cu, src, dst, order = (None if t is None else t.cpu().numpy() for t in got)
    w_cu, w_src, w_dst, w_order = oracle.compaction.token_maps(mask)
    assert np.array_equal(cu, w_cu), f"{what}: cu"
    assert np.array_equal(src, w_src), f"{what}: tok_src"
    assert np.array_equal(dst, w_dst), f"{what}: tok_dst"
    if order is not None:
        assert np.array_equal(order, w_order), f"{what}: order"


# (B, S): each row-length class, one and several passes of the scan's waves
# (32 / 16 / 8 / 4 sequences per wave, 16 waves), batches past the ordered limit
SCAN_SHAPES = [(1, 1), (3, 7), (1, 64), (520, 64), (32, 128), (256, 128), (300, 66), (130, 256), (70, 260),
               (8, 512), (65, 512), (4096, 3), (8192, 2)]


@pytest.mark.parametrize("B,S", SCAN_SHAPES)
def test_mask_scan_kernel_bit_exact(rlx, B, S):
    mask = _mask(B, S, 100 + B + S)
    got = rlx.mask_compaction(torch.from_numpy(mask).cuda(), with_order=B <= 256)
    _check(got, mask, f"mask scan {B}x{S}")


def test_mask_scan_rejects_order_past_its_batch_limit(rlx):
    mask = torch.ones((257, 4), dtype=torch.uint8, device="cuda")
    with pytest.raises(rlx.RlxError):
        rlx.mask_compaction(mask, with_order=True)


def _tiny_encoder(rlx, B, S, input_kind):
    sp = workloads.spec("minilm_b4_s128_bf16", batch=B, seq=S, layers=1, hidden=64, heads=2, ffn=128,
                        input_kind=input_kind, output_kind="pooled")
    wl = workloads.make(sp)
    weights, _ = to_device(wl)
    return rlx.Encoder(**encoder_kwargs(sp), weights=weights), wl


# id input: the embedding kernel scans masks of up to 16384 entries itself (the
# first four), the mask-scan kernel takes larger ones; hidden input always the latter
@pytest.mark.parametrize("B,S,kind", [(1, 512, "ids"), (4, 128, "ids"), (32, 128, "ids"), (45, 300, "ids"),
                                      (200, 100, "ids"), (64, 384, "ids"), (32, 128, "hidden"), (9, 200, "hidden")])
def test_forward_token_maps_bit_exact(rlx, B, S, kind):
    enc, wl = _tiny_encoder(rlx, B, S, kind)
    try:
        mask = _mask(B, S, 7 * B + S)
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
        inp = dev(wl.ids) if kind == "ids" else dev(wl.hidden_in).to(torch.bfloat16)
        enc.forward(inp, dev(mask))
        got = enc.token_maps(B, S, with_order=B <= 256)
        _check(got, mask, f"forward maps {B}x{S} {kind}")
        with pytest.raises(rlx.RlxError):
            enc.token_maps(B, S + 1)  # not the most recent forward's shape
    finally:
        enc.close()
