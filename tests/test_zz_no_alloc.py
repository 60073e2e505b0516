"""quasar_reconstruct_noalloc (the entry point that allocates nothing)
against quasar_reconstruct with a workspace, through the C ABI.

The NVFP4 call without a tensor amax is the one that needs scratch memory
(the tensor absmax pass); the allocation-free entry point takes it from the
library's static per-GPU array.  Two calls in a row, the second on a smaller
matrix whose absmax is smaller than the first's, so that a value left in the
array by the first call would show in the second's tensor scale and codes.
An INT call (no scratch) passes through unchanged."""
import numpy as np
import pytest
import torch

from paper_2608_13966_amd import quasar as Q
from paper_2608_13966_amd import synth

pytestmark = pytest.mark.gpu

KEYS = ("codes", "scales", "zeros", "r", "best_clip", "err", "tensor_scale")


def _bytes(t):
    return t.contiguous().view(torch.uint8)


def _both(W, v, g, **kw):
    """One call through each entry point on copies of v; returns both output dicts."""
    stream = torch.cuda.current_stream().cuda_stream
    d = Q.Descriptor(*W.shape, w_dtype=Q.BF16 if W.dtype == torch.bfloat16 else Q.F32, g_dtype=Q.BF16, **kw)
    res = []
    for noalloc in (False, True):
        o = Q.alloc_outputs(d, W, want_r=True, want_diag=True, has_amax=False)
        for k in KEYS:
            if o.get(k) is not None:
                o[k].view(torch.uint8).fill_(0xA5)
        vv = v.clone()
        if noalloc:
            s = Q.quasar_reconstruct_noalloc(d, W, vv, g, o["codes"], o["scales"], o["zeros"], o["r"],
                                             o["best_clip"], o["err"], o["tensor_scale"], None, stream)
        else:
            s = Q.quasar_reconstruct(d, W, vv, g, o["codes"], o["scales"], o["zeros"], o["r"], o["best_clip"],
                                     o["err"], o["tensor_scale"], None, o["workspace"], o["workspace_bytes"], stream)
        assert s == Q.OK, (noalloc, s, Q.quasar_status_string(s))
        o["v"] = vv
        res.append(o)
    torch.cuda.synchronize()
    return res


def _same(a, b, name):
    for k in KEYS + ("v",):
        x, y = a.get(k), b.get(k)
        if x is None and y is None:
            continue
        bx, by = _bytes(x), _bytes(y)
        if k == "tensor_scale":
            bx, by = bx[:4], by[:4]
        assert torch.equal(bx, by), f"{name}: {k} differs"


def test_noalloc_matches_workspace_call_twice():
    clips = tuple(synth.clip_grid(1.0, 0.7, 8))
    W1, v1, g1 = synth.gen_matrix(256, 512, 71, w_bf16=True, ema=True, device="cuda")
    W2, v2, g2 = synth.gen_matrix(37, 128, 72, w_bf16=True, ema=True, device="cuda")
    W2 = (W2.float() * 0.25).to(torch.bfloat16)  # a smaller tensor absmax than the first call's
    assert float(W2.float().abs().max()) < float(W1.float().abs().max())
    print("[case] noalloc nvfp4 256x512 then 37x128", flush=True)
    a1, b1 = _both(W1, v1, g1, fmt="nvfp4", clips=clips)
    _same(a1, b1, "nvfp4 first call")
    a2, b2 = _both(W2, v2, g2, fmt="nvfp4", clips=clips)
    _same(a2, b2, "nvfp4 second, smaller call")
    st = float(b2["tensor_scale"][0])
    assert st == np.float32(np.float32(W2.float().abs().max().item()) / np.float32(2688.0))
    print("[case] noalloc int3 g128 (no scratch)", flush=True)
    a3, b3 = _both(W2, v2, g2, fmt="int", bits=3, group=128, clips=clips)
    _same(a3, b3, "int3")


def test_noalloc_rejects_what_the_workspace_call_rejects():
    W, v, _ = synth.gen_matrix(8, 256, 73, w_bf16=True, ema=False, device="cuda")
    d = Q.Descriptor(8, 256, fmt="nvfp4", clips=(1.0, 1.5))  # clip factor out of range
    o = Q.alloc_outputs(Q.Descriptor(8, 256, fmt="nvfp4", clips=(1.0,)), W)
    o["codes"].fill_(7)
    s = Q.quasar_reconstruct_noalloc(d, W, v, None, o["codes"], o["scales"], None, o["r"], None, None,
                                     o["tensor_scale"], None, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert s == Q.ERR_ARG and torch.all(o["codes"] == 7)
