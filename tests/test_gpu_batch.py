"""GPU parity of the batched entry point (quasar_reconstruct_batch).

One launch over several matrices of different shapes must give, for every
matrix, the same bytes as a single-matrix call on it (every output: codes,
scales / codebook, zeros, r, best clip, score, tensor scale, the EMA v').
The single-matrix call of each matrix is checked against the oracle in the
same test (tests/test_gpu_parity.run_case), so the batch is pinned to the
oracle through it."""
import numpy as np
import pytest
import torch

from paper_2608_13966_amd import quasar as Q
from paper_2608_13966_amd import synth
from tests.test_gpu_parity import host, run_case

pytestmark = pytest.mark.gpu

KEYS = ("codes", "scales", "zeros", "r", "best_clip", "err", "tensor_scale")


def _bits(t):
    return None if t is None else host(t).view(np.uint8)


def _same(name, a, b, keys=KEYS):
    for k in keys:
        x, y = a.get(k), b.get(k)
        if x is None and y is None:
            continue
        assert (x is None) == (y is None), f"{name}: {k} present on one side only"
        bx, by = _bits(x), _bits(y)
        if k in ("tensor_scale", "amax_out"):  # one fp32 value in a 16-byte slot
            bx, by = bx[:4], by[:4]
        bad = np.count_nonzero(bx != by)
        assert bad == 0, f"{name}: {k} differs in {bad} bytes"


def _draw(shapes, seed0, *, w_bf16, ema, g_fp32=False):
    mats = []
    for i, (r, c) in enumerate(shapes):
        W, v, g = synth.gen_matrix(r, c, seed0 + 7 * i, w_bf16=w_bf16, ema=ema, device="cuda")
        if g is not None and g_fp32:
            g = g.float()
        mats.append((W, v, g))
    return mats


def _check_batch(name, mats, *, fmt, oracle_check=True, amax=False, **kw):
    """Single-matrix calls (oracle-checked) vs one batched call on copies of v."""
    singles, items = [], []
    for i, (W, v, g) in enumerate(mats):
        a = None
        if amax:
            a = torch.zeros(4, dtype=torch.float32, device="cuda")
            a[0] = W.float().abs().max()
        v1, v2 = v.clone(), v.clone()
        if oracle_check:
            out, _ = run_case(f"{name}.{i}", *W.shape, 0, fmt=fmt, W=W, v=v1, g=g, w_bf16=W.dtype == torch.bfloat16,
                              supply_amax=amax, **kw)
        else:
            out = Q.reconstruct(W, v1, g, fmt=fmt, tensor_amax=a, **kw)
        singles.append((out, v1))
        items.append((W, v2, g, a) if amax else (W, v2, g))
    print(f"[case] {name}: batch of {len(items)} fmt={fmt}", flush=True)
    outs = Q.reconstruct_batch(items, fmt=fmt, **kw)
    torch.cuda.synchronize()
    for i, ((o1, v1), o2, it) in enumerate(zip(singles, outs, items)):
        _same(f"{name}.{i}", o1, o2)
        if it[2] is not None:
            assert torch.equal(v1.view(torch.int32), it[1].view(torch.int32)), f"{name}.{i}: EMA v' differs"
    return outs


def test_batch_int4_ragged_mix_ema():
    shapes = [(64, 256), (3, 384), (17, 128), (1, 128), (40, 512)]
    _check_batch("batch.int4", _draw(shapes, 101, w_bf16=True, ema=True), fmt="int", bits=4, group=128,
                 clips=(1.0, 0.95, 0.9, 0.85, 0.8, 0.75, 0.7, 0.65))


def test_batch_int2_g64_fp32_no_ema_k12():
    shapes = [(5, 192), (32, 64), (9, 640)]
    _check_batch("batch.int2", _draw(shapes, 211, w_bf16=False, ema=False), fmt="int", bits=2, group=64,
                 clips=tuple(1.0 - 0.04 * k for k in range(12)))


def test_batch_int3_fp32_gradient_k16():
    shapes = [(4, 256), (11, 128)]
    _check_batch("batch.int3", _draw(shapes, 307, w_bf16=True, ema=True, g_fp32=True), fmt="int", bits=3,
                 group=128, clips=tuple(1.0 - 0.03 * k for k in range(16)))


def test_batch_int_sym():
    shapes = [(8, 256), (13, 128), (2, 384)]
    _check_batch("batch.sym", _draw(shapes, 401, w_bf16=True, ema=True), fmt="int_sym", bits=4, group=128,
                 clips=(1.0, 0.9, 0.8, 0.7))


def test_batch_nvfp4_per_matrix_amax():
    shapes = [(6, 64), (33, 256), (1, 16), (16, 512)]
    _check_batch("batch.nvfp4", _draw(shapes, 503, w_bf16=True, ema=True), fmt="nvfp4", amax=True,
                 clips=(1.0, 0.9, 0.8, 0.7, 0.6, 0.5, 0.45, 0.4))


def test_batch_rubin():
    shapes = [(16, 128), (8, 64), (24, 192)]
    _check_batch("batch.rubin", _draw(shapes, 601, w_bf16=True, ema=True), fmt="rubin", oracle_check=False,
                 clips=synth.PAPER_CLIPS)


def test_batch_weighting_and_param_dtype():
    shapes = [(7, 256), (20, 128)]
    _check_batch("batch.h2fp16", _draw(shapes, 701, w_bf16=True, ema=False), fmt="int", bits=4, group=128,
                 clips=(1.0, 0.9, 0.8), weighting="h2", param_dtype="fp16")


def test_batch_max_size_and_single():
    """Sixteen matrices in one launch (the maximum), and a batch of one (the
    single-matrix launch path)."""
    shapes = [(1 + 3 * i, 128 * (1 + i % 3)) for i in range(Q.MAX_BATCH)]
    mats = _draw(shapes, 809, w_bf16=True, ema=True)
    _check_batch("batch.16", mats, fmt="int", bits=4, group=128, clips=(1.0, 0.9), oracle_check=False)
    _check_batch("batch.1", mats[:1], fmt="int", bits=4, group=128, clips=(1.0, 0.9))


def test_batch_llama_layer_shapes():
    """The seven matrix shapes of one Llama-3.1-8B decoder layer in one
    launch (the benchmark's batched configuration), each compared with its
    single-matrix call."""
    wl = synth.workloads()["c3"]
    mats = []
    for (name, r, c), seed in list(zip(wl.shapes, wl.seeds))[:7]:
        W, v, g = synth.gen_matrix(r, c, seed, w_bf16=wl.w_bf16, ema=wl.ema, device="cuda")
        mats.append((W, v, g))
    _check_batch("batch.llama", mats, fmt=wl.fmt, bits=wl.bits, group=wl.group, clips=wl.clips,
                 oracle_check=False)
    del mats
    torch.cuda.empty_cache()


@pytest.mark.parametrize("w_bf16", [True, False])
def test_absmax_batch_exact(w_bf16):
    """The batched tensor absmax equals max |W| exactly (it is a maximum), for
    matrices that end inside a workgroup's span, a maximum planted at the first
    or last element or negative, and a matrix of zeros."""
    shapes = [(1, 16), (7, 272), (33, 1040), (4096, 4096), (3, 4096 * 16 + 16), (2, 32)]
    Ws = []
    for i, (r, c) in enumerate(shapes):
        W, _, _ = synth.gen_matrix(r, c, 900 + i, w_bf16=w_bf16, ema=False, device="cuda")
        Ws.append(W)
    Ws[1].view(-1)[-1] = -3.5            # largest magnitude, last element, negative
    Ws[2].view(-1)[0] = 7.25             # first element
    Ws[5].zero_()
    print(f"[case] absmax batch of {len(Ws)} w={'bf16' if w_bf16 else 'f32'}", flush=True)
    outs = Q.absmax_batch(Ws)
    torch.cuda.synchronize()
    for i, (W, o) in enumerate(zip(Ws, outs)):
        want = W.float().abs().max().reshape(1).view(torch.int32).item()
        got = o[:1].view(torch.int32).item()
        assert got == want, f"matrix {i} {tuple(W.shape)}: amax bits {got:#x} vs {want:#x}"


def test_batch_nvfp4_amax_from_batched_pass():
    """reconstruct_batch with no tensor amax takes it from one batched absmax
    pass; the results equal single-matrix calls that compute their own."""
    shapes = [(6, 64), (33, 256), (16, 512)]
    mats = _draw(shapes, 1103, w_bf16=True, ema=False)
    singles = [Q.reconstruct(W, v.clone(), g, fmt="nvfp4", clips=(1.0, 0.9, 0.8)) for W, v, g in mats]
    outs = Q.reconstruct_batch([(W, v.clone(), g) for W, v, g in mats], fmt="nvfp4", clips=(1.0, 0.9, 0.8))
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(zip(singles, outs)):
        _same(f"nvfp4.auto.{i}", a, b)
