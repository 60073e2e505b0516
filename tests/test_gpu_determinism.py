"""Run-to-run determinism on the GPU: the same inputs give the same bytes.

Every output has one owner, and the only atomics (the Rubin kernel's 64-bit
integer additions of fixed-point limbs, the absmax's atomic max on fp32 bit
patterns) are order-independent, so two runs -- single-matrix or batched --
must agree bit for bit."""
import numpy as np
import pytest
import torch

from paper_2608_13966_amd import quasar as Q
from paper_2608_13966_amd import synth
from tests.test_gpu_batch import KEYS, _same

pytestmark = pytest.mark.gpu

CASES = [
    dict(fmt="int", bits=2, group=64, clips=tuple(synth.clip_grid(1.0, 0.5, 12))),
    dict(fmt="int", bits=4, group=128, clips=tuple(synth.clip_grid(1.0, 0.65, 8))),
    dict(fmt="int_sym", bits=4, group=128, clips=tuple(synth.clip_grid(1.0, 0.65, 8))),
    dict(fmt="nvfp4", clips=tuple(synth.clip_grid(1.0, 0.7, 8))),
    dict(fmt="rubin", clips=synth.PAPER_CLIPS),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: c["fmt"] + str(c.get("bits", "")))
def test_repeat_runs_identical(case):
    W, v, g = synth.gen_matrix(512, 1024, 4242, w_bf16=True, ema=True, device="cuda")
    print(f"[case] determinism {case['fmt']} shape={tuple(W.shape)}", flush=True)
    runs = []
    for rep in range(3):
        vv = v.clone()
        out = Q.reconstruct(W, vv, g, **case)
        torch.cuda.synchronize()
        runs.append((out, vv))
    for rep in (1, 2):
        _same(f"{case['fmt']}.rep{rep}", runs[0][0], runs[rep][0], KEYS)
        assert torch.equal(runs[0][1].view(torch.int32), runs[rep][1].view(torch.int32))


def test_repeat_batched_runs_identical():
    mats = [synth.gen_matrix(r, c, 4300 + i, w_bf16=True, ema=True, device="cuda")
            for i, (r, c) in enumerate([(64, 512), (24, 1024), (8, 64)])]
    outs = []
    for rep in range(2):
        outs.append(Q.reconstruct_batch([(W, v.clone(), g) for W, v, g in mats], fmt="rubin",
                                        clips=synth.PAPER_CLIPS))
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(zip(*outs)):
        _same(f"batch.rubin.{i}", a, b, KEYS)


@pytest.mark.parametrize("fmt", ["int", "nvfp4"])
@pytest.mark.parametrize("by_product", [True, False])
def test_repeat_adamw_batched_runs_identical(fmt, by_product):
    """The batched fused AdamW step, from the same optimiser state, twice:
    identical W', m', v', outputs and (NVFP4) max |W'| by-products, with and
    without the by-product."""
    shapes = [(96, 256), (37, 384), (200, 128)]
    state = []
    for i, (r, c) in enumerate(shapes):
        W, v, g = synth.gen_matrix(r, c, 4400 + i, w_bf16=False, ema=True, device="cuda")
        m, v = synth.gen_adamw_state(r, c, 4400 + i, v, device="cuda")
        a = torch.zeros(4, dtype=torch.float32, device="cuda")
        a[0] = W.abs().max()
        state.append((W, m, v, g, a))
    kw = dict(lr=3e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.05, step=4, fmt=fmt, bits=2, group=64,
              clips=tuple(synth.clip_grid(1.0, 0.5, 12)) if fmt == "int" else tuple(synth.clip_grid(1.0, 0.7, 8)),
              want_amax_out=by_product and fmt == "nvfp4")
    print(f"[case] determinism adamw batch {fmt} by_product={by_product}", flush=True)
    runs = []
    for rep in range(2):
        items = [(W.clone(), m.clone(), v.clone(), g, a) if fmt == "nvfp4" else (W.clone(), m.clone(), v.clone(), g)
                 for W, m, v, g, a in state]
        outs = Q.adamw_reconstruct_batch(items, **kw)
        torch.cuda.synchronize()
        runs.append((items, outs))
    for i in range(len(shapes)):
        (ia, oa), (ib, ob) = runs[0], runs[1]
        for t in range(3):
            assert torch.equal(ia[i][t].view(torch.int32), ib[i][t].view(torch.int32)), (i, "Wmv"[t])
        _same(f"adamw.{fmt}.{i}", oa[i], ob[i], KEYS + ("amax_out",))
