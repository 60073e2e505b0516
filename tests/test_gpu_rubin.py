"""GPU parity of the Rubin INT3 LUT reconstruction (QUASAR_RUBIN_INT3)
against the oracle on the same seeded bytes.

Bit-exact: EMA v', chosen clip, codes, codebook bytes, r.  Excused and
counted: a different clip whose oracle scores are within 1e-6 (plus the
score's rounding floor), and a codebook byte whose oracle mean lies within
1e-6 of an E4M3 rounding midpoint (the GPU rounds the mean through fp32);
r of that index then follows the GPU's entry."""
import itertools
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2608_13966_amd import quasar as Q
from paper_2608_13966_amd import synth
from tests.test_gpu_parity import THREADS, host, record
from tests import _exact as X

pytestmark = pytest.mark.gpu

_LEVELS = np.array(sorted({v for v, _ in X.e4m3_levels()} | {-v for v, _ in X.e4m3_levels()}))
_MIDS = (_LEVELS[1:] + _LEVELS[:-1]) / 2


def _blocks(a, rows, cols):
    return a.reshape(rows // 8, 8, cols // 64, 64).transpose(0, 2, 1, 3).reshape(-1, 512)


def _f32(a):
    return (a.astype(np.uint32) << 16).view(np.float32) if a.dtype == np.uint16 else a


class rubin_path:
    """Run the Rubin kernel with the cells found one way: "auto" (the
    library's choice) or "tree" (the binary search for every grid), set with
    QUASAR_RUBIN_PATH."""

    def __init__(self, path):
        self.path = path

    def __enter__(self):
        self.old = os.environ.get("QUASAR_RUBIN_PATH")
        if self.path == "auto":
            os.environ.pop("QUASAR_RUBIN_PATH", None)
        else:
            os.environ["QUASAR_RUBIN_PATH"] = self.path

    def __exit__(self, *exc):
        if self.old is None:
            os.environ.pop("QUASAR_RUBIN_PATH", None)
        else:
            os.environ["QUASAR_RUBIN_PATH"] = self.old


def run_rubin(name, W, v, g=None, *, clips, weighting="h", row_step_blocks=1):
    """Both ways of finding the cells (when the library's choice is the bucket
    table, the tree search too), each from the same v, against one oracle run;
    the first run updates the caller's v, as a single call does."""
    R, C = W.shape
    Wh, vh, gh = host(W), host(v), host(g)
    brows = np.arange(0, R // 8, row_step_blocks)
    rows = (brows[:, None] * 8 + np.arange(8)[None, :]).ravel()
    bpr = C // 64
    bidx = (brows[:, None] * bpr + np.arange(bpr)[None, :]).ravel()
    o = oracle.rubin_reconstruct(Wh[rows], vh[rows], clips=clips, g=None if gh is None else gh[rows], beta2=0.999,
                                 weighting=weighting, want_scores=True, n_threads=THREADS)
    d = Q.Descriptor(R, C, fmt="rubin", clips=clips)
    paths = ("auto", "tree") if Q.quasar_int_path(d) == 1 else ("auto",)
    v0 = v.clone() if len(paths) > 1 else None
    for i, path in enumerate(paths):
        vv = v if i == 0 else v0.clone()
        with rubin_path(path):
            form = "buckets" if Q.quasar_int_path(d) == 1 else "tree"
            print(f"[case] {name} shape={(R, C)} K={len(clips)} ema={g is not None} w={weighting} path={path} "
                  f"cells={form}", flush=True)
            out = Q.reconstruct(W, vv, g, fmt="rubin", clips=clips, weighting=weighting)
            torch.cuda.synchronize()
        _check_rubin(name if path == "auto" else f"{name}.{path}", out, o, Wh, vv, g, rows, bidx, C, weighting)


def _check_rubin(name, out, o, Wh, v, g, rows, bidx, C, weighting):
    fails, st = [], {"groups": len(bidx), "near_tie": 0, "near_e4m3": 0}
    vh = host(v)
    if g is not None:
        bad = np.count_nonzero(o["v_out"].view(np.uint32) != vh[rows].view(np.uint32))
        if bad:
            fails.append(f"EMA v' differs in {bad} elements")
    h = o["v_out"] if g is not None else vh[rows]
    h = (h * h).astype(np.float32) if weighting == "h2" else np.ones_like(h) if weighting == "none" else h
    Rs = len(rows)
    wb = _blocks(_f32(Wh[rows]), Rs, C).astype(np.float64)
    hb = _blocks(h, Rs, C).astype(np.float64)
    ob, gb = o["best"].astype(int), out["best_clip"].cpu().numpy()[bidx].astype(int)
    floor = 1e-12 * np.sum(hb * wb * wb, axis=1)
    same = ob == gb
    for i in np.flatnonzero(~same):
        so, sg = o["scores"][i, ob[i]], o["scores"][i, gb[i]]
        if abs(sg - so) <= 1e-6 * so + floor[i]:
            st["near_tie"] += 1
        else:
            fails.append(f"block {i}: clip {gb[i]} vs oracle {ob[i]}, scores {sg} vs {so}")
    gcodes = out["codes"].cpu().numpy().reshape(-1, 192)[bidx]
    glut = out["scales"].cpu().numpy().reshape(-1, 8)[bidx]
    gr = _blocks(host(out["r"])[rows], Rs, C)
    orr = _blocks(o["r"], Rs, C)
    qb = _blocks(o["codes"], Rs, C)
    ge = out["err"].cpu().numpy()[bidx].astype(np.float64)
    for i in np.flatnonzero(same):
        if not np.array_equal(gcodes[i], o["codes_packed"].reshape(-1, 192)[i]):
            fails.append(f"block {i}: codes differ")
            continue
        lut_ok = glut[i] == o["lut"][i]
        for k in np.flatnonzero(~lut_ok):
            m = qb[i] == k
            mean = np.sum(hb[i][m] * wb[i][m]) / np.sum(hb[i][m])
            d = np.min(np.abs(_MIDS - mean) / np.maximum(np.abs(_MIDS), 1e-30))
            if d <= 1e-6:
                st["near_e4m3"] += 1
            else:
                fails.append(f"block {i}: codebook entry {k} {glut[i][k]:#x} vs {o['lut'][i][k]:#x} (mean {mean})")
        ok_el = lut_ok[qb[i]]
        if not np.array_equal(gr[i][ok_el], orr[i][ok_el]):
            fails.append(f"block {i}: r differs")
        oe = float(o["err"][i])
        if abs(ge[i] - oe) > 1e-5 * oe + floor[i] + 1e-37:
            fails.append(f"block {i}: err {ge[i]} vs {oe}")
    record(name, st)
    assert not fails, "\n".join(fails[:20])
    assert st["near_tie"] + st["near_e4m3"] <= max(2, 0.001 * st["groups"]), st


GRID = [(rows, cols, wb, ema, K) for (rows, cols), wb, ema, K in itertools.product(
    [(8, 64), (16, 192), (40, 128)], [True, False], ["none", "bf16", "f32"], [1, 8, 15])
    if (rows + cols + int(wb) + K + ["none", "bf16", "f32"].index(ema)) % 2 == 0 or K == 15]


@pytest.mark.parametrize("rows,cols,wb,ema,K", GRID)
def test_rubin_grid(rows, cols, wb, ema, K):
    W, v, g = synth.gen_matrix(rows, cols, 800 + K + rows, w_bf16=wb, ema=ema != "none", device="cuda")
    if g is not None and ema == "f32":
        g = g.float()
    clips = tuple(synth.clip_grid(1.0, 0.3, K)) if K > 1 else (1.0,)
    run_rubin(f"rubin.{rows}x{cols}.{'bf16' if wb else 'f32'}.ema-{ema}.K{K}", W, v, g, clips=clips)


@pytest.mark.parametrize("weighting", ["h2", "none"])
def test_rubin_weightings(weighting):
    W, v, g = synth.gen_matrix(32, 256, 851, w_bf16=True, ema=True, device="cuda")
    run_rubin(f"rubin.weighting-{weighting}", W, v, g, clips=tuple(synth.clip_grid(1.0, 0.3, 15)),
              weighting=weighting)


def test_rubin_degenerate_blocks():
    torch.manual_seed(3)
    W = (torch.randn(16, 256) * 0.02).float()
    v = torch.rand(16, 256).float()
    W[0:8, 0:64] = 0.125                    # constant block
    v[8:16, 64:128] = 0.0                   # no saliency in a block
    v[0:8, 128:192] = 0.0
    v[3, 130] = 2.0                         # all saliency on one weight
    W[8:16, 192:256] = torch.tensor([-0.5, 0.5]).repeat(8, 32)   # two values
    run_rubin("rubin.degenerate", W.cuda(), v.cuda(), clips=(1.0, 0.8, 0.6, 0.4))
    run_rubin("rubin.degenerate.bf16", W.to(torch.bfloat16).cuda(), v.cuda(), clips=(1.0, 0.7))


def test_rubin_llama_gate_sampled():
    """A full Llama-3.1-8B gate projection in the benchmark's configuration
    (bf16 W, fused EMA, the paper's 15-factor grid); every 23rd block row is
    checked against the oracle."""
    W, v, g = synth.gen_matrix(14336, 4096, 4, w_bf16=True, ema=True, device="cuda")
    clips = tuple(np.float32(x) for x in np.round(np.arange(1.0, 0.29, -0.05), 2))
    run_rubin("rubin.llama-gate", W, v, g, clips=clips, row_step_blocks=23)
    del W, v, g
    torch.cuda.empty_cache()


def _f32_fma(a, b, c):
    """fp32 fma on fp32 arrays: the fp64 product is exact and, at these
    magnitudes, so is the fp64 sum, so one rounding to fp32 remains."""
    return (a.astype(np.float64) * b.astype(np.float64) + c.astype(np.float64)).astype(np.float32)


def _entries_below_range(W, v, clips):
    """Number of (block, clip, index) whose weights all have a saliency below
    2^-101 of their block's largest (and at least one such weight): far below
    both the fixed point's range and the recompute threshold."""
    n = 0
    for blk_w, blk_v in zip(_blocks(W, *W.shape), _blocks(v, *v.shape)):
        mn, mx = blk_w.min(), blk_w.max()
        c, rho = np.float32(0.5) * (mx + mn), np.float32(0.5) * (mx - mn)
        rrho = np.float32(1.0) / rho
        u = _f32_fma(blk_w, np.float32(rrho), np.float32(-(c * rrho)))
        for f in clips:
            al = np.float32(7.0) / (np.float32(2.0) * np.float32(f))
            q = np.clip(np.rint(_f32_fma(u, al, np.float32(3.5))), 0, 7)
            for b in range(8):
                sel = blk_v[q == b]
                n += int(sel.size > 0 and (sel.max() < blk_v.max() * 2.0 ** -101))
    return n


def test_rubin_saliency_beyond_fixed_point_range():
    """Blocks whose saliency spans more than 2^101: the kernel's fixed-point
    cell sums drop the smallest saliencies (and round the others to units of
    2^-72 or so of the block's largest), and a codebook entry whose saliency
    sum lies below about 2^-33 of the block's largest, or made only of dropped
    weights, is recomputed in fp64.  In every block one weight has v = 1e20
    and the weights above the block's 90th percentile of w have v = 1e-15 (a
    ratio of 1e-35), so the top index of most clips holds only those;
    codebook bytes, codes, r and scores must still match the oracle's direct
    sums."""
    torch.manual_seed(5)
    W = (torch.randn(16, 128) * 0.02).float()
    v = torch.rand(16, 128).float() + 0.5
    for rb in range(2):
        for cb in range(2):
            blk = W[8 * rb:8 * rb + 8, 64 * cb:64 * cb + 64]
            vb = v[8 * rb:8 * rb + 8, 64 * cb:64 * cb + 64]
            top = blk >= torch.quantile(blk, 0.9)
            vb[top] = 1e-15
            vb[0, 0] = 1e20
    clips = tuple(synth.clip_grid(1.0, 0.3, 15))
    assert _entries_below_range(W.numpy(), v.numpy(), clips) > 0  # the case is exercised
    run_rubin("rubin.saliency-range", W.cuda(), v.cuda(), clips=clips)
    run_rubin("rubin.saliency-range.bf16", W.to(torch.bfloat16).cuda(), v.cuda(), clips=(1.0, 0.9, 0.75, 0.6))


def test_rubin_saliency_near_recompute_threshold():
    """Saliencies around the point where the kernel stops trusting its
    fixed-point sums: one weight per block has v = 1 and the others v = 2^-e
    with e uniform in [26, 42], so a codebook entry's saliency sum falls on
    either side of about 2^-33 of the block's largest.  Entries above it are
    served from the cell sums (whose low limbs then drop bits: a weight with
    v = 2^-42 keeps about 12 of its 24), those below are recomputed in fp64;
    both must match the oracle."""
    rng = np.random.default_rng(17)
    W = torch.from_numpy((rng.standard_normal((32, 256)) * 0.02).astype(np.float32))
    e = rng.uniform(26.0, 42.0, size=(32, 256))
    v = torch.from_numpy(np.exp2(-e).astype(np.float32))
    v[0::8, 0::64] = 1.0
    clips = tuple(synth.clip_grid(1.0, 0.3, 15))
    run_rubin("rubin.saliency-threshold", W.cuda(), v.cuda(), clips=clips)
    run_rubin("rubin.saliency-threshold.bf16", W.to(torch.bfloat16).cuda(), v.cuda(), clips=clips)


def test_rubin_weights_in_split_cells():
    """Blocks whose weights sit almost all within 0.085 of the block's centre
    (in units of its half-range), where every clip of the paper's grid has
    only its tie threshold at 0 and the host adds its extra cell boundaries:
    each of those boundaries then has many weights on both sides.  The codes
    do not change at an extra boundary, so the kernel must still match the
    oracle on every block, in both cell forms."""
    rng = np.random.default_rng(23)
    W = (rng.uniform(-0.085, 0.085, size=(16, 256)) * 0.1).astype(np.float32)
    for rb in range(2):
        for cb in range(4):
            W[8 * rb, 64 * cb] = -0.1  # the block's range: u = w / 0.1
            W[8 * rb + 1, 64 * cb] = 0.1
    W = torch.from_numpy(W)
    v = torch.from_numpy(rng.uniform(0.1, 1.0, size=(16, 256)).astype(np.float32))
    clips = tuple(synth.clip_grid(1.0, 0.3, 15))
    run_rubin("rubin.split-cells", W.cuda(), v.cuda(), clips=clips)
    run_rubin("rubin.split-cells.bf16", W.to(torch.bfloat16).cuda(), v.cuda(), clips=clips)


def test_rubin_weights_among_tie_thresholds():
    """Weights whose normalised position lies between the clips' tie
    thresholds T(k, 3) (just below u = 0, where the fp32 code rounding ties at
    3.5), which the bucket table merges into one cell boundary: their blocks'
    code-3 and code-4 entries are summed directly.  Every block has c = 0 and
    rho = 1, so u = w, and 40 weights spread over the span."""
    torch.manual_seed(11)
    W = (torch.randn(16, 128) * 0.3).clamp(-0.9, 0.9).float()
    v = torch.rand(16, 128).float() + 0.1
    for rb in range(2):
        for cb in range(2):
            blk = W[8 * rb:8 * rb + 8, 64 * cb:64 * cb + 64]
            blk[0, 0], blk[0, 1] = -1.0, 1.0
            blk[1:6, 2:10] = -torch.linspace(3.3e-8, 1.0e-8, 40).reshape(5, 8)
    clips = tuple(synth.clip_grid(1.0, 0.3, 15))
    run_rubin("rubin.tie-span", W.cuda(), v.cuda(), clips=clips)
    run_rubin("rubin.tie-span.bf16", W.to(torch.bfloat16).cuda(), v.cuda(), clips=clips)


def test_rubin_dense_grid_takes_tree():
    """A clip grid too dense for the bucket table (16 factors in [0.9, 1]):
    the tree search serves it."""
    clips = tuple(synth.clip_grid(1.0, 0.9, 16))
    assert Q.quasar_int_path(Q.Descriptor(16, 128, fmt="rubin", clips=clips)) == 0
    W, v, g = synth.gen_matrix(16, 128, 861, w_bf16=True, ema=True, device="cuda")
    run_rubin("rubin.dense-grid", W, v, g, clips=clips)
