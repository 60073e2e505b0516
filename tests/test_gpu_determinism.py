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
