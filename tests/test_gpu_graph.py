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


ADAMW_CASES = [
    dict(fmt="int", bits=2, group=64, clips=tuple(synth.clip_grid(1.0, 0.5, 12))),
    dict(fmt="nvfp4", clips=tuple(synth.clip_grid(1.0, 0.7, 8))),
]


@pytest.mark.parametrize("kw", ADAMW_CASES, ids=lambda c: c["fmt"])
def test_graph_adamw_batch_replays_match_eager(kw):
    """The batched fused AdamW step (with the NVFP4 max |W'| by-product, whose
    clear is a kernel) captured once and replayed from a restored optimiser
    state: every replay gives the eager call's W', m', v' and outputs."""
    HP = dict(lr=3e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.05, step=2)
    state = []
    for i, (r, c) in enumerate(SHAPES):
        W, v, g = synth.gen_matrix(r, c, 5200 + i, w_bf16=False, ema=True, device="cuda")
        m, v = synth.gen_adamw_state(r, c, 5200 + i, v, device="cuda")
        state.append((W, m, v, g))
    nv = kw["fmt"] == "nvfp4"
    amax_in = [torch.tensor([float(W.abs().max()), 0, 0, 0], dtype=torch.float32, device="cuda") for W, *_ in state]
    d = Q.Descriptor(*state[0][0].shape, w_dtype=Q.F32, g_dtype=Q.BF16, **kw)
    opt = Q.AdamW(HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], HP["weight_decay"], HP["step"])

    def buffers():
        work = [(W.clone(), m.clone(), v.clone(), g) for W, m, v, g in state]
        outs, mats = [], []
        for (W, m, v, g), a in zip(work, amax_in):
            dd = Q.Descriptor(*W.shape, w_dtype=Q.F32, g_dtype=Q.BF16, **kw)
            o = Q.alloc_outputs(dd, W, want_r=False, want_diag=True, has_amax=True)
            o["r"] = torch.empty(W.shape, dtype=torch.bfloat16, device="cuda")
            o["amax_out"] = torch.zeros(4, dtype=torch.float32, device="cuda") if nv else None
            outs.append(o)
            mats.append(Q.AdamWMatrix(W.shape[0], W.shape[1], Q._p(W), Q._p(m), Q._p(v), Q._p(g), Q._p(o["codes"]),
                                      Q._p(o["scales"]), Q._p(o["zeros"]), Q._p(o["r"]), Q._p(o["best_clip"]),
                                      Q._p(o["err"]), Q._p(o["tensor_scale"]), Q._p(a if nv else None),
                                      Q._p(o["amax_out"])))

        def launch(stream):
            s = Q.quasar_adamw_reconstruct_batch(d, opt, mats, Q.BF16, stream)
            assert s == Q.OK, s

        return work, outs, launch

    print(f"[case] graph adamw batch {kw['fmt']}", flush=True)
    ref_work, ref_outs, ref_launch = buffers()
    ref_launch(torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()

    work, outs, launch = buffers()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up outside the capture (it updates the state, restored below)
        launch(side.cuda_stream)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        launch(torch.cuda.current_stream().cuda_stream)
    keys = KEYS + ("amax_out",)
    for rep in range(4):
        for (W, m, v, _), (W0, m0, v0, _) in zip(work, state):  # the step's starting state, eagerly
            W.copy_(W0)
            m.copy_(m0)
            v.copy_(v0)
        for o in outs:  # scribble over the outputs so a replay that writes nothing fails
            for k in keys:
                if o.get(k) is not None:
                    o[k].view(torch.uint8).fill_(0xA5)
        junk = torch.randn(1 << 20, device="cuda").sum()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.isfinite(junk)
        for i, (a, b) in enumerate(zip(ref_outs, outs)):
            _same(f"graph.adamw.{kw['fmt']}.rep{rep}.{i}", a, b, keys)
        for i, (x, y) in enumerate(zip(ref_work, work)):
            for t in range(3):
                assert torch.equal(x[t].view(torch.int32), y[t].view(torch.int32)), (rep, i, "Wmv"[t])
