"""Upload a workload to GPU tensors in the layout the C ABI expects.

Only moves and casts arrays: fp32 values that are bf16-representable become
torch.bfloat16 exactly; quantised codes, scales and zero-points keep their
integer / fp16 storage.  Used by the tests and the benchmark, never by the
oracle.
"""
from __future__ import annotations

import numpy as np


def to_device(wl, device="cuda"):
    import torch

    sp = wl.spec
    act = torch.bfloat16 if sp.dtype == "bf16" else torch.float32

    def f(a, dtype=act):
        return torch.from_numpy(np.ascontiguousarray(a)).to(device=device, dtype=dtype)

    def f32(a):
        return f(np.asarray(a, np.float32), torch.float32)

    weights = {"layers": []}
    if sp.input_kind == "ids":
        weights.update(word=f(wl.emb["word"]), pos=f(wl.emb["pos"]), type=f(wl.emb["type"]),
                       emb_gamma=f32(wl.emb["gamma"]), emb_beta=f32(wl.emb["beta"]))
    for li, lw in enumerate(wl.layers):
        d = {k: f32(lw[k]) for k in ("bqkv", "bo", "b1", "b2", "ln1_g", "ln1_b", "ln2_g", "ln2_b")}
        for nm in ("wqkv", "wo", "w1", "w2"):
            if sp.quant == "none":
                d[nm] = f(lw[nm])
            else:
                qd = wl.quant[li][nm]
                d[nm] = torch.from_numpy(np.ascontiguousarray(qd["q"])).to(device)
                d[nm + "_scales"] = torch.from_numpy(np.ascontiguousarray(qd["scales"])).to(device)
                if "zeros" in qd:
                    d[nm + "_zeros"] = torch.from_numpy(np.ascontiguousarray(qd["zeros"])).to(device)
        weights["layers"].append(d)
    inputs = {"mask": torch.from_numpy(wl.mask).to(device)}
    if sp.input_kind == "ids":
        inputs["input"] = torch.from_numpy(wl.ids).to(device)
    else:
        inputs["input"] = f(wl.hidden_in)
    return weights, inputs


def encoder_kwargs(sp, max_batch=None, max_seq=None, use_graph=False):
    return dict(hidden=sp.hidden, heads=sp.heads, head_dim=sp.head_dim, ffn=sp.ffn, layers=sp.layers, vocab=sp.vocab,
                max_pos=sp.max_pos, type_vocab=sp.type_vocab, ln_eps=sp.eps, dtype=sp.dtype, quant=sp.quant,
                group_size=sp.group, input_kind=sp.input_kind, output_kind=sp.output_kind,
                max_batch=max_batch or sp.batch, max_seq=max_seq or sp.seq, use_graph=use_graph)
