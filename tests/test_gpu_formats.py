"""The gfx950 FP4 / FP8 conversions the kernels rely on, driven through the
NVFP4 and Rubin kernels with crafted blocks at the formats' edge values, and
compared bit for bit with the oracle (no exception is excused here).

  * E2M1 (Sec. 4.2): scaled weights exactly on every rounding midpoint 0.25,
    0.75, 1.25, 1.75, 2.5, 3.5 and 5 (ties go to the even mantissa), one ulp
    to either side of each, exactly 6, above 6 (saturation), zeros of either
    sign and tiny values (a zero code is +0).  The block maximum m is 2 and the
    clip factors 0.75 and 0.375 make the search multiplier 6/f a power of two,
    so y = w (1/m) (6/f) is exact and lands where it is placed.
  * E4M3 block scale (Sec. 4.2): blocks w = s q with q on the E2M1 grid and
    power-of-two saliency, so the fitted scale s* = sum h q w / sum h q^2 is
    exactly s, and s / S_t (S_t = 2^-10) is exactly each E4M3 rounding
    midpoint, normal and subnormal; blocks whose fitted scale exceeds 448 S_t
    (saturation at 448).
  * E4M3 codebook entries (App. B, Eq. rubin-fit): Rubin blocks whose eight
    INT3 indices each hold copies of one value, with power-of-two saliency, so
    each entry's weighted mean is exactly that value: E4M3 midpoints (signed),
    one fp32 ulp beside them, subnormal midpoints, and magnitudes above 448.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_13966_amd import quasar as Q
from tests.test_gpu_parity import THREADS, host, record
from tests import _exact as X

pytestmark = pytest.mark.gpu

E2M1_MIDS = (0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0)
E2M1_GRID = (0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0)


def _e4m3_pos():
    return np.array(sorted(v for v, _ in X.e4m3_levels()))  # 0 and the 126 positive finite values


def _to_bf16_exact(a):
    t = torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16)
    assert torch.equal(t.float(), torch.from_numpy(np.ascontiguousarray(a, np.float32))), "value not exact in bf16"
    return t


def _nvfp4_exact(name, W, h, clips, amax):
    """GPU against the oracle with every byte equal: codes, E4M3 scales, r,
    chosen clip; the score within 1e-5."""
    Wg = W.cuda()
    vg = torch.from_numpy(h).cuda()
    amax_t = torch.tensor([amax, 0, 0, 0], dtype=torch.float32, device="cuda")
    print(f"[case] {name} shape={tuple(W.shape)} w={W.dtype} K={len(clips)}", flush=True)
    out = Q.reconstruct(Wg, vg, fmt="nvfp4", clips=clips, tensor_amax=amax_t)
    torch.cuda.synchronize()
    Wh = host(W)
    o = oracle.reconstruct(Wh, h, fmt="nvfp4", clips=clips, tensor_amax=amax, want_scores=True, want_diag=True,
                           n_threads=THREADS)
    ng = Wh.size // 16
    st = {"groups": ng}
    gc = out["codes"].cpu().numpy()
    bad = np.flatnonzero(np.any(gc.reshape(ng, 8) != o["codes_packed"].reshape(ng, 8), axis=1))
    assert bad.size == 0, f"{name}: codes differ in blocks {bad[:8].tolist()}"
    ge = out["scales"].cpu().numpy()
    bad = np.flatnonzero(ge != o["e4m3"])
    assert bad.size == 0, (f"{name}: E4M3 bytes differ in blocks {bad[:8].tolist()}: gpu {ge[bad[:8]].tolist()} "
                           f"oracle {o['e4m3'][bad[:8]].tolist()} s*/S_t {o['diag'][bad[:8], 2].tolist()}")
    assert np.array_equal(out["best_clip"].cpu().numpy(), o["best"]), f"{name}: chosen clip differs"
    gr, orr = host(out["r"]), o["r"]
    assert np.array_equal(gr.view(np.uint8), orr.view(np.uint8)), f"{name}: r differs"
    assert float(out["tensor_scale"][0]) == float(o["tensor_scale"])
    oe, gerr = o["err"].astype(np.float64), out["err"].cpu().numpy().astype(np.float64)
    assert np.all(np.abs(gerr - oe) <= 1e-5 * oe + 1e-37), f"{name}: score beyond 1e-5"
    record(name, st)
    return o


def _e2m1_blocks(c6, w_bf16, seed):
    """Blocks of 16 whose maximum is 2 (so 1 / m = 0.5 exactly) and whose
    other weights put y = w * 0.5 * c6 exactly on the chosen values."""
    scale = 2.0 / c6  # w = y * 2 / c6
    ys = []
    for mid in E2M1_MIDS + (6.0,):
        w = np.float32(mid * scale)
        if w_bf16:
            t = torch.tensor([float(w)], dtype=torch.bfloat16)
            up = float(torch.nextafter(t, torch.tensor([np.inf], dtype=torch.bfloat16)))
            dn = float(torch.nextafter(t, torch.tensor([-np.inf], dtype=torch.bfloat16)))
            ws = [float(w), up, dn]
        else:
            ws = [float(w), float(np.nextafter(w, np.float32(np.inf))), float(np.nextafter(w, np.float32(-np.inf)))]
        ys += ws
    ys += [6.5 * scale, 7.75 * scale, 1.999 * scale * 4, 0.0, -0.0, 1e-30, -1e-30, 0.1 * scale, -0.2 * scale]
    vals = np.array(ys + [-y for y in ys], np.float32)
    if w_bf16:  # the filler values to their bf16 neighbours (the placed ones are bf16 values already)
        vals = torch.from_numpy(vals).to(torch.bfloat16).float().numpy()
    rng = np.random.default_rng(seed)
    blocks = []
    for rep in range(4):
        perm = rng.permutation(vals.size)
        for i in range(0, vals.size, 15):
            chunk = vals[perm[i:i + 15]]
            chunk = np.concatenate([chunk, np.zeros(15 - chunk.size, np.float32)])
            blocks.append(np.concatenate([[2.0 if rep % 2 == 0 else -2.0], chunk]).astype(np.float32))
    W = np.stack(blocks).reshape(-1, 64 if len(blocks) % 4 == 0 else 16)
    h = (2.0 ** rng.integers(-3, 4, size=W.shape)).astype(np.float32)
    return W, h


@pytest.mark.parametrize("w_bf16", [False, True])
@pytest.mark.parametrize("f,c6", [(0.75, 8.0), (0.375, 16.0)])
def test_e2m1_midpoints_and_saturation(f, c6, w_bf16):
    W, h = _e2m1_blocks(c6, w_bf16, 1)
    assert np.float32(6.0) / np.float32(f) == np.float32(c6)
    Wt = _to_bf16_exact(W) if w_bf16 else torch.from_numpy(W)
    _nvfp4_exact(f"formats.e2m1.f{f}.{'bf16' if w_bf16 else 'f32'}", Wt, h, (f,), 2.0)


def _e4m3_blocks(seed):
    """Blocks w = s q (q on the E2M1 grid, one q = 6 so the block maximum is 6 s)
    with s / 2^-10 on every E4M3 rounding midpoint, plus blocks whose fitted
    scale lies above 448 S_t, plus one block holding the tensor maximum 2.625
    (S_t = 2.625 / 2688 = 2^-10)."""
    rng = np.random.default_rng(seed)
    pos = _e4m3_pos()
    mids = (pos[1:] + pos[:-1]) / 2
    targets = list(mids) + list(pos[1:])        # every midpoint and every value (normal and subnormal)
    blocks = []
    for x in targets:
        s = np.float32(x * 2.0 ** -10)
        assert float(s) == x * 2.0 ** -10
        q = rng.choice(E2M1_GRID, size=15) * rng.choice([-1.0, 1.0], size=15)
        blocks.append(np.concatenate([[6.0], q]) * float(s))
    # fitted scale above 448 S_t: one weight at the block maximum m (code 6),
    # fifteen at 0.8 m (y = 4.8, code 4) with far larger saliency, so
    # s* ~ 0.2 m = 1.2 m / 6; with m near the tensor maximum that is beyond 448 S_t
    sat = []
    for m in (2.625, 2.5, 2.375, 2.25, 2.2):
        blocks.append(np.array([m] + [0.8 * m] * 15, np.float64) * rng.choice([-1.0, 1.0]))
        sat.append(len(blocks) - 1)
    blocks.append(np.array([2.625] + [0.5] * 15))
    W = np.stack(blocks).astype(np.float32)
    h = (2.0 ** rng.integers(-3, 4, size=W.shape)).astype(np.float32)
    for b in sat:
        h[b, 0] = 2.0 ** -20
    return W, h, len(targets), sat


def test_e4m3_block_scale_midpoints_subnormals_and_saturation():
    W, h, n_mid, sat = _e4m3_blocks(2)
    assert float(np.abs(W).max()) == 2.625
    o = _nvfp4_exact("formats.e4m3-scale", torch.from_numpy(W), h, (1.0,), 2.625)
    # the crafted ratios arrived: s*/S_t exactly on the target, and above 448 where meant
    pos = _e4m3_pos()
    mids = (pos[1:] + pos[:-1]) / 2
    targets = np.array(list(mids) + list(pos[1:]))
    assert np.array_equal(o["diag"][:n_mid, 2], targets)
    assert np.all(o["diag"][sat, 2] > 448.0) and np.all(o["e4m3"][sat] == 0x7E)
    # ties went to the even mantissa: every midpoint's byte is even
    assert np.all(o["e4m3"][:len(mids)] % 2 == 0)


def test_nvfp4_crafted_blocks_full_grid():
    """All crafted blocks together with an 8-factor grid, through the regular
    parity protocol."""
    from tests.test_gpu_parity import run_case
    W1, _ = _e2m1_blocks(8.0, False, 3)
    W2, _, _, _ = _e4m3_blocks(4)
    W = np.ascontiguousarray(np.concatenate([W1.reshape(-1, 16), W2]))  # one 16-block per row
    rng = np.random.default_rng(5)
    h = (2.0 ** rng.integers(-3, 4, size=W.shape)).astype(np.float32)
    run_case("formats.nvfp4-grid", 0, 0, 0, fmt="nvfp4", clips=(1.0, 0.9, 0.8, 0.75, 0.6, 0.5, 0.375, 0.3),
             W=torch.from_numpy(W).cuda(), v=torch.from_numpy(h).cuda(), w_bf16=False)


# ---------------------------------------------------------------------------- Rubin codebook entries

def _rubin_block(values, rng):
    """One 8 x 64 block holding 64 copies of each of the eight values (sorted:
    value k sits on INT3 level k of the block's range at clip 1)."""
    vals = np.repeat(np.asarray(values, np.float32), 64)
    return vals[rng.permutation(512)].reshape(8, 64)


def _on_levels(values):
    """The eight values lie within 0.3 of a step of their INT3 levels."""
    v = np.asarray(values, np.float64)
    lev = v[0] + np.arange(8) * (v[7] - v[0]) / 7
    return np.all(np.abs(v - lev) <= 0.3 * (v[7] - v[0]) / 7)


def _rubin_sets():
    pos = _e4m3_pos()
    mids = (pos[1:] + pos[:-1]) / 2
    smids = np.array(sorted(set(mids) | set(-mids)))
    sets = []
    # normal midpoints over several ranges: each level takes its nearest midpoint
    for lo, hi in ((-3.25, 3.75), (0.21875, 3.75), (-0.4375, -0.0546875), (1.0625, 13.0), (-104.0, 232.0)):
        lo, hi = (smids[np.argmin(np.abs(smids - x))] for x in (lo, hi))
        lev = lo + np.arange(8) * (hi - lo) / 7
        vals = [smids[np.argmin(np.abs(smids - x))] for x in lev]
        assert _on_levels(vals), (lo, hi, vals)
        sets.append(("mid", vals))
        up = [float(np.nextafter(np.float32(x), np.float32(np.inf))) for x in vals]
        dn = [float(np.nextafter(np.float32(x), np.float32(-np.inf))) for x in vals]
        sets += [("mid+ulp", up), ("mid-ulp", dn)]
    # subnormal midpoints (m + 1/2) 2^-9, evenly spaced, ties to the even m
    sets.append(("subnormal", [(-7.5 + 2 * k) * 2.0 ** -9 for k in range(8)]))
    sets.append(("subnormal-small", [(-3.5 + k) * 2.0 ** -9 for k in range(8)]))
    # magnitudes above 448 (saturation), positive and negative
    sets.append(("saturate", [float(np.float32(380 + k * 220 / 7)) for k in range(8)]))
    sets.append(("saturate-neg", [float(np.float32(-620 + k * 240 / 7)) for k in range(8)]))
    return sets


@pytest.mark.parametrize("w_bf16", [False, True])
def test_rubin_codebook_midpoints_subnormals_and_saturation(w_bf16):
    rng = np.random.default_rng(7)
    sets = [s for s in _rubin_sets() if not (w_bf16 and s[0] in ("mid+ulp", "mid-ulp"))]
    if w_bf16:
        sets += [("mid-bf16-ulp", [float(torch.nextafter(torch.tensor([x], dtype=torch.bfloat16),
                                                         torch.tensor([np.inf], dtype=torch.bfloat16)))
                                   for x in vals]) for kind, vals in _rubin_sets() if kind == "mid"]
        sets = [(k, [float(torch.tensor([x], dtype=torch.bfloat16)) for x in v]) for k, v in sets]
    blocks = [_rubin_block(vals, rng) for _, vals in sets]
    for (kind, vals) in sets:
        assert _on_levels(vals), (kind, vals)
    n = len(blocks)
    cols = 64 * n
    W = np.concatenate(blocks, axis=1).astype(np.float32)  # 8 rows, blocks side by side
    h = (2.0 ** rng.integers(-3, 4, size=W.shape)).astype(np.float32)
    Wt = _to_bf16_exact(W) if w_bf16 else torch.from_numpy(W)
    name = f"formats.rubin.{'bf16' if w_bf16 else 'f32'}"
    print(f"[case] {name} shape={tuple(W.shape)} blocks={n}", flush=True)
    out = Q.reconstruct(Wt.cuda(), torch.from_numpy(h).cuda(), fmt="rubin", clips=(1.0,))
    torch.cuda.synchronize()
    o = oracle.rubin_reconstruct(host(Wt), h, clips=(1.0,), want_scores=True, n_threads=THREADS)
    glut = out["scales"].cpu().numpy().reshape(-1, 8)
    for b, (kind, vals) in enumerate(sets):
        assert np.array_equal(glut[b], o["lut"][b]), (f"{kind}: codebook {glut[b].tolist()} vs oracle "
                                                      f"{o['lut'][b].tolist()} for values {vals}")
        want = [oracle.e4m3_code_signed(x) for x in vals]  # each entry is E4M3 of its (exact) mean
        assert o["lut"][b].tolist() == want, (kind, o["lut"][b].tolist(), want)
    assert np.array_equal(out["codes"].cpu().numpy(), o["codes_packed"]), "codes differ"
    assert np.array_equal(host(out["r"]).view(np.uint8), o["r"].view(np.uint8)), "r differs"
    sat = [b for b, (k, _) in enumerate(sets) if k.startswith("saturate")]
    assert all(((o["lut"][b] & 0x7F) == 0x7E).sum() >= 3 for b in sat)
    record(name, {"groups": n})
