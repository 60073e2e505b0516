"""The benchmark's own launches against the oracle, on every group.

bench.py times each layer set as one batched launch per step with the
per-group diagnostics off (best clip and score not written).  Here the same
launch runs twice on the same inputs, once exactly so and once with the
diagnostics on; the two must agree byte for byte on everything both write,
and the second is compared with the oracle on every group of every matrix
(tests/_parity.py).  So the configuration the throughput is quoted for is the
one pinned to the oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_13966_amd import quasar as Q
from paper_2608_13966_amd import synth
from tests import _parity
from tests.test_gpu_parity import THREADS, host, record

pytestmark = pytest.mark.gpu

BENCH_HP = dict(lr=1e-5, beta1=0.9, eps=1e-8, weight_decay=0.01)  # bench.py's fused-step constants


def _bytes(t):
    return t.contiguous().view(torch.uint8)


def _outputs(d, W, want_diag, r_bf16=False):
    o = Q.alloc_outputs(d, W, want_r=not r_bf16, want_diag=want_diag, has_amax=True)
    if r_bf16:
        o["r"] = torch.empty(W.shape, dtype=torch.bfloat16, device=W.device)
    return o


@pytest.mark.parametrize("wl_name", ["c3", "c4"])
def test_bench_launch_matches_oracle(wl_name):
    wl = synth.workloads()[wl_name]
    nv = wl.fmt == "nvfp4"
    mats = [synth.gen_matrix(r, c, seed, w_bf16=wl.w_bf16, ema=wl.ema, device="cuda")
            for (_, r, c), seed in zip(wl.shapes, wl.seeds)]
    v_in = [v.clone() for _, v, _ in mats]  # the EMA overwrites v: each launch starts from a copy
    descs = [Q.Descriptor(*W.shape, fmt=wl.fmt, bits=wl.bits, group=wl.group, clips=wl.clips,
                          w_dtype=Q.BF16 if wl.w_bf16 else Q.F32, g_dtype=Q.BF16, beta2=wl.beta2)
             for W, _, _ in mats]
    stream = torch.cuda.current_stream().cuda_stream
    runs = []
    for want_diag in (False, True):
        vs = [v.clone() for v in v_in]
        outs = [_outputs(d, W, want_diag) for d, (W, _, _) in zip(descs, mats)]
        amax = [torch.zeros(4, dtype=torch.float32, device="cuda") if nv else None for _ in mats]
        arr = [Q.matrix(W, v, g, o, a) for (W, _, g), v, o, a in zip(mats, vs, outs, amax)]
        print(f"[case] bench launch {wl_name} diag={want_diag}", flush=True)
        if nv:
            assert Q.quasar_absmax_batch(descs[0], arr, amax, stream) == Q.OK
        assert Q.quasar_reconstruct_batch(descs[0], arr, stream) == Q.OK
        torch.cuda.synchronize()
        runs.append((vs, outs))
    (v0, o0), (v1, o1) = runs
    for i in range(len(mats)):
        for k in ("codes", "scales", "zeros", "r", "tensor_scale"):
            if o0[i][k] is not None:
                n = 4 if k == "tensor_scale" else None
                assert torch.equal(_bytes(o0[i][k])[:n], _bytes(o1[i][k])[:n]), (wl_name, i, k)
        if wl.ema:
            assert torch.equal(_bytes(v0[i]), _bytes(v1[i])), (wl_name, i, "v'")
    for i, ((name, _, _), (W, _, g)) in enumerate(zip(wl.shapes, mats)):
        Wh, vh, gh = host(W), host(v_in[i]), host(g)
        amax = float(oracle.absmax(Wh)) if nv else None
        o = oracle.reconstruct(Wh, vh, fmt=wl.fmt, bits=wl.bits, group=wl.group, clips=wl.clips, g=gh,
                               beta2=wl.beta2, tensor_amax=amax, want_scores=True, want_diag=True,
                               n_threads=THREADS)
        out = o1[i]
        gpu = {"codes": out["codes"].cpu().numpy(), "scales": out["scales"].cpu().numpy(),
               "best_clip": out["best_clip"].cpu().numpy(), "err": out["err"].cpu().numpy(), "r": host(out["r"])}
        if nv:
            gpu["tensor_scale"] = out["tensor_scale"].cpu().numpy()[0]
        else:
            gpu["zeros"] = out["zeros"].cpu().numpy()
        fails, st = _parity.compare(fmt=wl.fmt, bits=wl.bits, group=wl.group, W=Wh,
                                    h=o["v_out"] if wl.ema else vh, o=o, gpu=gpu,
                                    v_out_gpu=host(v1[i]) if wl.ema else None)
        record(f"bench-launch.{wl_name}.{name}", st)
        assert not fails, f"{wl_name}.{name}:\n" + "\n".join(fails)
        assert st["near_tie"] + st["near_tie_floor"] + st["near_e4m3"] <= max(2, 0.001 * st["groups"]), dict(st)
        del o, gpu
    del mats, runs
    torch.cuda.empty_cache()


def _f32_bits(a):
    return np.ascontiguousarray(a).view(np.uint16 if a.dtype == np.uint16 else np.uint32)


@pytest.mark.parametrize("wl_name", ["c6", "c7"])
def test_adamw_bench_launch_matches_oracle(wl_name):
    """The fused AdamW layer-set step (one quasar_adamw_reconstruct_batch with
    bench.py's constants, fp32 master weights, bf16 r, the NVFP4 max |W'|
    by-product): W', m', v' bit for bit and every group's reconstruction
    against the oracle."""
    wl = synth.workloads()[wl_name]
    nv = wl.fmt == "nvfp4"
    state = []
    for (_, r, c), seed in zip(wl.shapes, wl.seeds):
        W, v, g = synth.gen_matrix(r, c, seed, w_bf16=wl.w_bf16, ema=True, device="cuda")
        m, v = synth.gen_adamw_state(r, c, seed, v, device="cuda")
        state.append((W, m, v, g))
    amax_in = [torch.tensor([float(W.abs().max()), 0, 0, 0], dtype=torch.float32, device="cuda") if nv else None
               for W, _, _, _ in state]
    kw = dict(step=1, beta2=wl.beta2, fmt=wl.fmt, bits=wl.bits, group=wl.group, clips=wl.clips,
              want_amax_out=nv, **BENCH_HP)
    runs = []
    for want_diag in (False, True):
        items = [(W.clone(), m.clone(), v.clone(), g, a) if nv else (W.clone(), m.clone(), v.clone(), g)
                 for (W, m, v, g), a in zip(state, amax_in)]
        print(f"[case] bench launch {wl_name} diag={want_diag}", flush=True)
        outs = Q.adamw_reconstruct_batch(items, want_diag=want_diag, **kw)
        torch.cuda.synchronize()
        runs.append((items, outs))
    (i0, o0), (i1, o1) = runs
    for i in range(len(state)):
        for t in range(3):
            assert torch.equal(_bytes(i0[i][t]), _bytes(i1[i][t])), (wl_name, i, "Wmv"[t])
        for k in ("codes", "scales", "zeros", "r", "tensor_scale", "amax_out"):
            if o0[i].get(k) is not None:
                n = 4 if k in ("tensor_scale", "amax_out") else None
                assert torch.equal(_bytes(o0[i][k])[:n], _bytes(o1[i][k])[:n]), (wl_name, i, k)
    for i, ((name, _, _), (W, m, v, g)) in enumerate(zip(wl.shapes, state)):
        o = oracle.adamw_reconstruct(host(W), host(m), host(v), host(g), step=1, beta2=wl.beta2, fmt=wl.fmt,
                                     bits=wl.bits, group=wl.group, clips=wl.clips,
                                     tensor_amax=float(amax_in[i][0]) if nv else None, want_scores=True,
                                     want_diag=True, n_threads=THREADS, **BENCH_HP)
        for t, k in enumerate(("W_out", "m_out", "v_out")):
            bad = np.count_nonzero(_f32_bits(host(i1[i][t])) != _f32_bits(o[k]))
            assert bad == 0, f"{wl_name}.{name}: {k} differs in {bad} elements"
        out = o1[i]
        gpu = {"codes": out["codes"].cpu().numpy(), "scales": out["scales"].cpu().numpy(),
               "best_clip": out["best_clip"].cpu().numpy(), "err": out["err"].cpu().numpy(), "r": host(out["r"])}
        if nv:
            gpu["tensor_scale"] = out["tensor_scale"].cpu().numpy()[0]
            assert float(out["amax_out"][0]) == float(o["amax_out"]), "max |W'| by-product"
        else:
            gpu["zeros"] = out["zeros"].cpu().numpy()
        o["r"] = synth.to_host(torch.from_numpy(o["r"]).to(torch.bfloat16))  # bf16 r of the fp32 W'
        fails, st = _parity.compare(fmt=wl.fmt, bits=wl.bits, group=wl.group, W=o["W_out"], h=o["v_out"], o=o,
                                    gpu=gpu)
        record(f"bench-launch.{wl_name}.{name}", st)
        assert not fails, f"{wl_name}.{name}:\n" + "\n".join(fails)
        assert st["near_tie"] + st["near_tie_floor"] + st["near_e4m3"] <= max(2, 0.001 * st["groups"]), dict(st)
        del o, gpu
    del state, runs
    torch.cuda.empty_cache()
