"""GPU parity of the fused AdamW step + reconstruction
(quasar_adamw_reconstruct) against the oracle, on the same seeded bytes."""
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2608_13966_amd import quasar as Q
from paper_2608_13966_amd import synth
from tests import _parity
from tests.test_gpu_parity import THREADS, host, record

pytestmark = pytest.mark.gpu

HP = dict(lr=3e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.05)


def _bits(a):
    return np.ascontiguousarray(a).view(np.uint16 if a.dtype == np.uint16 else np.uint32)


def _inputs(rows, cols, seed, w_bf16, g_fp32):
    W, v, g = synth.gen_matrix(rows, cols, seed, w_bf16=w_bf16, ema=True, device="cuda")
    m, v = synth.gen_adamw_state(rows, cols, seed, v, device="cuda")
    if g_fp32:
        g = g.float()
    return W, m.contiguous(), v.contiguous(), g


def run_step(name, W, m, v, g, *, step, fmt="int", bits=4, group=128, clips=(1.0, 0.8, 0.6), r_dtype="bf16",
             weighting="h", row_step=1, amax=None):
    """One fused step on the GPU tensors (updated in place) and on host copies
    through the oracle; compares every output.  Returns the oracle dict."""
    Wh, mh, vh, gh = host(W), host(m), host(v), host(g)
    amax_t = None
    if fmt == "nvfp4":
        amax_t = torch.tensor([amax, 0, 0, 0], dtype=torch.float32, device="cuda")
    print(f"[case] {name} shape={tuple(W.shape)} fmt={fmt} bits={bits} step={step} r={r_dtype}", flush=True)
    out = Q.adamw_reconstruct(W, m, v, g, step=step, fmt=fmt, bits=bits, group=group, clips=clips,
                              tensor_amax=amax_t, r_dtype=r_dtype, want_amax_out=fmt == "nvfp4",
                              weighting=weighting, **HP)
    torch.cuda.synchronize()
    R, C = W.shape
    rows = np.arange(0, R, row_step)
    o = oracle.adamw_reconstruct(Wh[rows], mh[rows], vh[rows], gh[rows], step=step, fmt=fmt, bits=bits,
                                 group=group, clips=clips, tensor_amax=amax, want_scores=True, want_diag=True,
                                 n_threads=THREADS, weighting=weighting, **HP)
    # optimiser state: bit-exact
    for k, t in (("W_out", W), ("m_out", m), ("v_out", v)):
        got = host(t)[rows]
        bad = np.count_nonzero(_bits(got) != _bits(o[k]))
        assert bad == 0, f"{name}: {k} differs in {bad} elements"
    G = 16 if fmt == "nvfp4" else group
    nb = 4 if fmt == "nvfp4" else bits
    gpr = C // G
    gidx = (rows[:, None] * gpr + np.arange(gpr)[None, :]).ravel()
    gpu = {"codes": out["codes"].cpu().numpy().reshape(R, C * nb // 8)[rows].ravel(),
           "scales": out["scales"].cpu().numpy()[gidx], "best_clip": out["best_clip"].cpu().numpy()[gidx],
           "err": out["err"].cpu().numpy()[gidx], "r": host(out["r"])[rows]}
    if fmt == "nvfp4":
        gpu["tensor_scale"] = out["tensor_scale"].cpu().numpy()[0]
        assert out["amax_out"].cpu().numpy()[0] == oracle.absmax(host(W)), "amax by-product"
    else:
        gpu["zeros"] = out["zeros"].cpu().numpy()[gidx]
    # the oracle's r is in W's dtype; a bf16 r of an fp32 W is its RNE rounding
    if gpu["r"].dtype == np.uint16 and o["r"].dtype == np.float32:
        o["r"] = synth.to_host(torch.from_numpy(o["r"]).to(torch.bfloat16))
    h = o["v_out"]
    if weighting == "h2":
        h = (h * h).astype(np.float32)
    elif weighting == "none":
        h = np.ones_like(h)
    fails, st = _parity.compare(fmt=fmt, bits=bits, group=group, W=o["W_out"], h=h, o=o, gpu=gpu)
    record(name, st)
    assert not fails, "\n".join(fails)
    assert st["near_tie"] + st["near_e4m3"] <= max(2, 0.001 * st["groups"]), dict(st)
    return o


CASES = [
    # fmt, bits, group, W bf16, g fp32, r dtype, weighting
    ("int", 4, 128, False, False, "bf16", "h"),
    ("int", 2, 64, False, False, "fp32", "h"),
    ("int", 3, 128, True, False, "bf16", "h"),
    ("int", 4, 64, True, True, "bf16", "h2"),
    ("int", 2, 128, False, True, "bf16", "none"),
    ("nvfp4", 4, 16, False, False, "bf16", "h"),
    ("nvfp4", 4, 16, True, True, "bf16", "h"),
    ("nvfp4", 4, 16, False, False, "fp32", "h2"),
]


@pytest.mark.parametrize("fmt,bits,group,wb,gf,rd,wt", CASES)
def test_fused_adamw_three_steps(fmt, bits, group, wb, gf, rd, wt):
    """Three consecutive steps on a ragged shape: the optimiser state stays
    bit-identical to the oracle's and every reconstruction matches."""
    cols = 3 * (group if fmt == "int" else 128)
    W, m, v, g = _inputs(37, cols, 500 + bits + int(wb), wb, gf)
    clips = tuple(synth.clip_grid(1.0, 0.4, 9))
    amax = oracle.absmax(host(W)) if fmt == "nvfp4" else None
    for step in (1, 2, 3):
        o = run_step(f"adamw.{fmt}{bits}g{group}.{'bf16' if wb else 'f32'}W.{rd}r.{wt}.t{step}", W, m, v, g,
                     step=step, fmt=fmt, bits=bits, group=group, clips=clips, r_dtype=rd, weighting=wt, amax=amax)
        if fmt == "nvfp4":
            amax = float(o["amax_out"])  # last step's by-product sets this step's tensor scale
        gen = torch.Generator(device="cuda").manual_seed(step)
        g.copy_((torch.randn(g.shape, generator=gen, device="cuda") * 1e-3).to(g.dtype))


@pytest.mark.parametrize("fmt,bits,group", [("int", 2, 64), ("nvfp4", 4, 16)])
def test_fused_adamw_llama_gate_sampled(fmt, bits, group):
    """A full-size Llama-3.1-8B gate projection with fp32 master weights and a
    bf16 gradient, as the benchmark runs it; every 97th row is checked."""
    W, m, v, g = _inputs(14336, 4096, 4, False, False)
    amax = oracle.absmax(host(W)) if fmt == "nvfp4" else None
    clips = tuple(synth.clip_grid(1.0, 0.5, 12)) if fmt == "int" else tuple(synth.clip_grid(1.0, 0.7, 8))
    run_step(f"adamw.llama-gate.{fmt}", W, m, v, g, step=5, fmt=fmt, bits=bits, group=group, clips=clips,
             row_step=97, amax=amax)
    del W, m, v, g
    torch.cuda.empty_cache()


def test_fused_adamw_error_leaves_state_untouched():
    W, m, v, g = _inputs(8, 256, 9, False, False)
    W0, m0, v0 = W.clone(), m.clone(), v.clone()
    with pytest.raises(Q.QuasarError):
        Q.adamw_reconstruct(W, m, v, g, step=0, bits=4, group=128, **HP)
    with pytest.raises(Q.QuasarError):
        Q.adamw_reconstruct(W, m, v, g, step=1, fmt="nvfp4", **HP)  # no tensor amax
    torch.cuda.synchronize()
    assert torch.equal(W, W0) and torch.equal(m, m0) and torch.equal(v, v0)


@pytest.mark.parametrize("fmt,bits,group,clips,w_bf16", [
    ("int", 2, 64, tuple(synth.clip_grid(1.0, 0.5, 12)), False),   # binned INT kernel
    ("int", 4, 128, tuple(synth.clip_grid(1.0, 0.65, 8)), True),   # direct INT kernel
    ("nvfp4", 4, 16, tuple(synth.clip_grid(1.0, 0.7, 8)), False)])
def test_adamw_batch_equals_single_calls(fmt, bits, group, clips, w_bf16):
    """quasar_adamw_reconstruct_batch over matrices of different shapes gives
    bit-identical W', m, v, codes, scales, zeros, r, chosen clips, scores and
    amax by-products to one quasar_adamw_reconstruct per matrix."""
    shapes = [(96, 256), (32, 512), (200, 128)]
    inputs = [_inputs(r, c, 930 + i, w_bf16, False) for i, (r, c) in enumerate(shapes)]
    amaxes = [torch.tensor([float(oracle.absmax(host(W))), 0, 0, 0], dtype=torch.float32, device="cuda")
              for W, _, _, _ in inputs]
    kw = dict(step=3, fmt=fmt, bits=bits, group=group, clips=clips, want_amax_out=fmt == "nvfp4", **HP)
    single = []
    for (W, m, v, g), a in zip(inputs, amaxes):
        Ws, ms, vs = W.clone(), m.clone(), v.clone()
        o = Q.adamw_reconstruct(Ws, ms, vs, g, tensor_amax=a if fmt == "nvfp4" else None, **kw)
        single.append((Ws, ms, vs, o))
    items = [(W, m, v, g, a) if fmt == "nvfp4" else (W, m, v, g) for (W, m, v, g), a in zip(inputs, amaxes)]
    print(f"[case] adamw.batch.{fmt}{bits}g{group} shapes={shapes}", flush=True)
    outs = Q.adamw_reconstruct_batch(items, **kw)
    torch.cuda.synchronize()
    keys = ["codes", "scales", "zeros", "best_clip", "err", "r", "tensor_scale", "amax_out"]
    for i, ((W, m, v, _), (Ws, ms, vs, o), ob) in enumerate(zip(inputs, single, outs)):
        if fmt == "nvfp4":  # the by-product is exactly max |W'|, also where the last workgroup is partly idle
            want = W.float().abs().max().reshape(1).view(torch.int32).item()
            assert ob["amax_out"][:1].view(torch.int32).item() == want, (i, "amax_out")
        for name, a, b in (("W", W, Ws), ("m", m, ms), ("v", v, vs)):
            assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a.view(torch.int32),
                               b.view(torch.int16) if b.dtype == torch.bfloat16 else b.view(torch.int32)), (i, name)
        for k in keys:
            x, y = o.get(k), ob.get(k)
            assert (x is None) == (y is None), (i, k)
            if x is None:
                continue
            if k in ("tensor_scale", "amax_out"):  # element 0 holds the value
                x, y = x[:1], y[:1]
            assert torch.equal(x.view(torch.uint8), y.view(torch.uint8)), (i, k)


@pytest.mark.parametrize("w_bf16", [False, True])
def test_adamw_amax_by_product_exact_and_repeatable(w_bf16):
    """The by-product max |W'| of the fused NVFP4 step is exactly the largest
    magnitude of the updated weights, on shapes whose last workgroup is
    partly idle (200 x 128: 64 of its 256 lanes hold a block; 37 x 384: 120),
    and two runs from the same state give identical bytes, single-matrix and
    batched.  Lanes past the last block re-run the step on a copy of the last
    block, whose weights its owner may already have updated in place; they
    must not reach the by-product."""
    shapes = [(200, 128), (37, 384), (16, 64)]
    clips = tuple(synth.clip_grid(1.0, 0.7, 8))
    state = [_inputs(r, c, 960 + i, w_bf16, False) for i, (r, c) in enumerate(shapes)]
    amaxes = [torch.tensor([float(oracle.absmax(host(W))), 0, 0, 0], dtype=torch.float32, device="cuda")
              for W, _, _, _ in state]
    kw = dict(step=2, fmt="nvfp4", clips=clips, want_amax_out=True, **HP)

    def single_run():
        res = []
        for (W, m, v, g), a in zip(state, amaxes):
            Ws, ms, vs = W.clone(), m.clone(), v.clone()
            o = Q.adamw_reconstruct(Ws, ms, vs, g, tensor_amax=a, **kw)
            res.append((Ws, ms, vs, o))
        torch.cuda.synchronize()
        return res

    def batch_run():
        cl = [(W.clone(), m.clone(), v.clone(), g, a) for (W, m, v, g), a in zip(state, amaxes)]
        outs = Q.adamw_reconstruct_batch(cl, **kw)
        torch.cuda.synchronize()
        return [(W, m, v, o) for (W, m, v, _, _), o in zip(cl, outs)]

    print(f"[case] adamw.amax-by-product w={'bf16' if w_bf16 else 'f32'} shapes={shapes}", flush=True)
    runs = [single_run(), single_run(), batch_run(), batch_run()]
    keys = ["codes", "scales", "best_clip", "err", "r", "tensor_scale", "amax_out"]
    for i in range(len(shapes)):
        Wn = runs[0][i][0]
        want = Wn.float().abs().max().reshape(1).view(torch.int32).item()
        for ri, run in enumerate(runs):
            W, m, v, o = run[i]
            got = o["amax_out"][:1].view(torch.int32).item()
            assert got == want, f"run {ri} matrix {i} {shapes[i]}: amax_out {got:#x}, max |W'| {want:#x}"
            for name, a, b in (("W", W, Wn), ("m", m, runs[0][i][1]), ("v", v, runs[0][i][2])):
                assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), (ri, i, name)
            for k in keys:
                x, y = o[k], runs[0][i][3][k]
                if k in ("tensor_scale", "amax_out"):
                    x, y = x[:1], y[:1]
                assert torch.equal(x.view(torch.uint8), y.view(torch.uint8)), (ri, i, k)
