"""Capture in a HIP graph: a step of the path (batched reconstruction, with
the NVFP4 tensor absmax pass) recorded once with torch.cuda.CUDAGraph and
replayed several times, with the program's own eager work and
synchronisations between the replays; every replay must give the bytes of
the eager call on the same inputs.  The library records no memset nodes (its
clears are kernels), which is what makes replays after the first safe."""
import pytest
import torch

from paper_2608_13966_amd import quasar as Q
from paper_2608_13966_amd import synth
from tests.test_gpu_batch import KEYS, _same

pytestmark = pytest.mark.gpu

SHAPES = [(64, 512), (24, 1024), (8, 128)]
CASES = [
    dict(fmt="int", bits=3, group=128, clips=tuple(synth.clip_grid(1.0, 0.65, 8))),
    dict(fmt="nvfp4", clips=tuple(synth.clip_grid(1.0, 0.7, 8))),
    dict(fmt="rubin", clips=synth.PAPER_CLIPS),
]


def _outputs(mats, kw):
    """Output buffers and a launcher for one batched call (plus the batched
    absmax for NVFP4) on fixed buffers, as a captured step needs."""
    W0 = mats[0][0]
    d = Q.Descriptor(*W0.shape, w_dtype=Q.BF16, g_dtype=Q.BF16, **kw)
    outs, arr_items, amax = [], [], []
    for W, v, g in mats:
        dd = Q.Descriptor(*W.shape, w_dtype=Q.BF16, g_dtype=Q.BF16, **kw)
        o = Q.alloc_outputs(dd, W, want_r=True, want_diag=True, has_amax=True)
        a = torch.zeros(4, dtype=torch.float32, device="cuda") if kw["fmt"] == "nvfp4" else None
        outs.append(o)
        amax.append(a)
        arr_items.append(Q.matrix(W, v, g, o, a))

    def launch(stream):
        if kw["fmt"] == "nvfp4":
            s = Q.quasar_absmax_batch(d, arr_items, amax, stream)
            assert s == Q.OK, s
        s = Q.quasar_reconstruct_batch(d, arr_items, stream)
        assert s == Q.OK, s

    return outs, launch


@pytest.mark.parametrize("kw", CASES, ids=lambda c: c["fmt"])
def test_graph_replays_match_eager(kw):
    mats = [synth.gen_matrix(r, c, 5100 + i, w_bf16=True, ema=False, device="cuda")
            for i, (r, c) in enumerate(SHAPES)]
    print(f"[case] graph {kw['fmt']}", flush=True)
    # eager reference on the same inputs (no EMA: v is only read, so every
    # replay sees the same inputs)
    ref_outs, ref_launch = _outputs(mats, kw)
    ref_launch(torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()

    outs, launch = _outputs(mats, kw)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up outside the capture
        launch(side.cuda_stream)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        launch(torch.cuda.current_stream().cuda_stream)
    for rep in range(4):
        for o in outs:  # scribble over the outputs so a replay that writes nothing fails
            for k in KEYS:
                if o.get(k) is not None:
                    o[k].view(torch.uint8).fill_(0xA5)
        junk = torch.randn(1 << 20, device="cuda").sum()  # eager work between replays
        graph.replay()
        torch.cuda.synchronize()
        assert torch.isfinite(junk)
        for i, (a, b) in enumerate(zip(ref_outs, outs)):
            _same(f"graph.{kw['fmt']}.rep{rep}.{i}", a, b, KEYS)
