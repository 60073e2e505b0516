"""GPU-vs-oracle comparison for the parity tests (test code only).

Protocol (what must match and which exceptions are counted, not failed):
  * bit-exact: v' (EMA), the chosen clip index, the packed codes of the chosen
    clip, the NVFP4 E4M3 byte, and r whenever the fitted (s, z) are bit-identical;
  * a clip mismatch is excused iff the oracle's own scores of the two clips are
    within 1e-6 relative (counted "near_tie"); where the difference exceeds
    that but lies within an absolute floor of 1e-12 * sum h w^2 (the rounding
    floor of a score made of terms of size h w^2) it is counted separately
    ("near_tie_floor").  The group's other outputs follow from the excused
    choice and are not compared;
  * an E4M3 mismatch is excused iff the oracle's s*/S_t lies within 1e-6
    relative of an E4M3 rounding midpoint (counted "near_e4m3"); that block's
    r and score follow from it and are not compared;
  * relative 1e-5: |da| <= 1e-5 |a|, |db| <= 1e-5 max(|b|, |a| qmax),
    |derr| <= 1e-5 err (an error inside the 1e-12 * sum h w^2 floor but
    outside 1e-5 is counted "err_floor"); fp32 r within 1e-5 of the group's
    max |r|;
  * bf16 r where (s, z) differ from the oracle's in the last bits (counted
    "ab_last_bit"): every element equal, or one bf16 ulp apart where the
    oracle's fp32 r = s q + z lies within 1e-6 relative of a bf16 rounding
    midpoint (elements counted "bf16_midpoint"), or -- as fp32 r -- within
    1e-5 of the group's max |r| (elements near zero; counted
    "bf16_within_scale").
"""
from __future__ import annotations

from collections import Counter

import numpy as np

import oracle


def f32_of(x):
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << 16).view(np.float32)
    return x


def _e4m3_midpoint_distance(x):
    """Relative distance of x > 0 from the nearest E4M3 rounding midpoint."""
    vals = np.array([oracle.e4m3_value(c) for c in range(0x7F)])
    mids = (vals[:-1] + vals[1:]) / 2
    x = np.asarray(x, np.float64)
    i = np.clip(np.searchsorted(mids, x), 1, len(mids) - 1)
    d = np.minimum(np.abs(mids[i] - x), np.abs(mids[i - 1] - x))
    return d / np.maximum(np.abs(x), 1e-300)


def _bf16_midpoint_distance(r32):
    """Relative distance of fp32 values from the midpoint of their two bf16
    neighbours (the point where round-to-nearest-even to bf16 switches)."""
    r32 = np.ascontiguousarray(r32, dtype=np.float32)
    u = r32.view(np.uint32)
    lo = (u & np.uint32(0xFFFF0000)).view(np.float32).astype(np.float64)
    hi = ((u & np.uint32(0xFFFF0000)) + np.uint32(0x10000)).view(np.float32).astype(np.float64)
    x = r32.astype(np.float64)
    return np.abs(x - (lo + hi) / 2) / np.maximum(np.abs(x), 1e-300)


def _oracle_r32(fmt, bits, o, groups, G):
    """The oracle's fp32 r of the given groups, s q + z from its emitted
    (s, z) and codes (single rounding of the exact fp64 value)."""
    q = o["codes"].reshape(-1, G)[groups].astype(np.int64)
    if fmt == "int_sym":
        q = np.where(q >= (1 << (bits - 1)), q - (1 << bits), q)
        z = np.zeros(len(groups))
    else:
        z = o["zero"][groups].astype(np.float64)
    s = o["scale"][groups].astype(np.float64)
    return (s[:, None] * q + z[:, None]).astype(np.float32)


def compare(*, fmt, bits, group, W, h, o, gpu, v_out_gpu=None):
    """W: host W (fp32 or bf16 bits) [R, C]; h: the saliency actually used
    (oracle's v_out with an EMA, else v); o: oracle dict (want_scores and
    want_diag); gpu: dict of host numpy arrays (codes, scales, zeros, r,
    best_clip, err, tensor_scale).  Returns (failures: list[str], stats: Counter)."""
    fails, st = [], Counter()
    nv = fmt == "nvfp4"
    G = 16 if nv else group
    nb = 4 if nv else bits
    qmax = (1 << nb) - 1
    w = f32_of(W).reshape(-1, G).astype(np.float64)
    hh = h.reshape(-1, G).astype(np.float64)
    ng = w.shape[0]
    st["groups"] = ng
    floor = 1e-12 * np.sum(hh * w * w, axis=1)

    if v_out_gpu is not None:
        bad = np.count_nonzero(o["v_out"].view(np.uint32) != v_out_gpu.view(np.uint32))
        if bad:
            fails.append(f"EMA v' differs in {bad} elements")

    ob, gb = o["best"].astype(np.int64), gpu["best_clip"].astype(np.int64)
    same = ob == gb
    diff = np.flatnonzero(~same)
    if diff.size:
        so = o["scores"][diff, ob[diff]]
        sg = o["scores"][diff, gb[diff]]
        rel = np.abs(sg - so) <= 1e-6 * so
        ok = rel | (np.abs(sg - so) <= 1e-6 * so + floor[diff])
        st["near_tie"] += int(rel.sum())
        st["near_tie_floor"] += int((ok & ~rel).sum())
        if not ok.all():
            k = diff[~ok][:5]
            fails.append(f"{int((~ok).sum())} clip mismatches outside the near-tie window, e.g. groups {k.tolist()} "
                         f"oracle {ob[k].tolist()} gpu {gb[k].tolist()} scores "
                         f"{[(o['scores'][i, ob[i]], o['scores'][i, gb[i]]) for i in k]}")

    bpg = G * nb // 8
    oc = o["codes_packed"].reshape(ng, bpg)
    gc = gpu["codes"].reshape(ng, bpg)
    code_bad = same & np.any(oc != gc, axis=1)
    if code_bad.any():
        k = np.flatnonzero(code_bad)[:5]
        fails.append(f"{int(code_bad.sum())} groups with the same clip but different codes, e.g. {k.tolist()}")

    ab_same = np.ones(ng, bool)
    cmp = same.copy()  # groups whose r and score are compared: same clip, no excused E4M3 byte
    if nv:
        e_bad = same & (o["e4m3"] != gpu["scales"])
        if e_bad.any():
            idx = np.flatnonzero(e_bad)
            near = _e4m3_midpoint_distance(o["diag"][idx, 2]) <= 1e-6
            st["near_e4m3"] += int(near.sum())
            if not near.all():
                fails.append(f"{int((~near).sum())} E4M3 scale mismatches away from a rounding midpoint, e.g. "
                             f"{idx[~near][:5].tolist()}")
            cmp[idx] = False
        if float(o["tensor_scale"]) != float(gpu["tensor_scale"]):
            fails.append(f"tensor scale {float(gpu['tensor_scale'])} != {float(o['tensor_scale'])}")
    else:
        oa, ga = o["scale"].astype(np.float64), gpu["scales"].astype(np.float64)
        oz, gz = o["zero"].astype(np.float64), gpu["zeros"].astype(np.float64)
        a_ok = np.abs(ga - oa) <= 1e-5 * np.abs(oa) + 1e-30
        z_ok = np.abs(gz - oz) <= 1e-5 * np.maximum(np.abs(oz), np.abs(oa) * qmax) + 1e-30
        bad = same & ~(a_ok & z_ok)
        if bad.any():
            k = np.flatnonzero(bad)[:5]
            fails.append(f"{int(bad.sum())} groups with (s, z) outside 1e-5, e.g. {k.tolist()} "
                         f"oracle {[(oa[i], oz[i]) for i in k]} gpu {[(ga[i], gz[i]) for i in k]}")
        ab_same = (o["scale"].view(np.uint32) == gpu["scales"].view(np.uint32)) & \
                  (o["zero"].view(np.uint32) == gpu["zeros"].view(np.uint32))
        st["ab_last_bit"] += int((same & ~ab_same).sum())

    if gpu.get("r") is not None:
        orr = o["r"].reshape(ng, G)
        grr = gpu["r"].reshape(ng, G)
        if orr.dtype == np.uint16:
            exact = np.all(orr == grr, axis=1)
            bad = cmp & ab_same & ~exact
            if bad.any():
                fails.append(f"{int(bad.sum())} groups with identical (s, z) but different bf16 r")
            loose = np.flatnonzero(cmp & ~ab_same & ~exact)
            if loose.size:
                # (s, z) within 1e-5 but not bit-identical: a bf16 r may differ
                # by one ulp only where the oracle's fp32 r lies next to a bf16
                # rounding midpoint
                r32 = _oracle_r32(fmt, bits, o, loose, G)
                ob16, gb16 = orr[loose].astype(np.int64), grr[loose].astype(np.int64)
                neq = ob16 != gb16
                one_ulp = (np.abs(ob16 - gb16) == 1) & ((ob16 ^ gb16) < 0x8000)  # adjacent, same sign
                near = _bf16_midpoint_distance(r32) <= 1e-6
                # the relative 1e-5 of the group's scale that fp32 r is held to
                of, gf = f32_of(orr[loose]).astype(np.float64), f32_of(grr[loose]).astype(np.float64)
                small = np.abs(of - gf) <= 1e-5 * np.max(np.abs(r32.astype(np.float64)), axis=1, keepdims=True)
                ok = ~neq | (one_ulp & near) | small
                st["bf16_midpoint"] += int((neq & one_ulp & near).sum())
                st["bf16_within_scale"] += int((neq & small & ~(one_ulp & near)).sum())
                if not ok.all():
                    i, e = np.argwhere(~ok)[0]
                    fails.append(f"{int((~ok.all(axis=1)).sum())} groups with a bf16 r that differs by more than "
                                 f"one ulp or away from a rounding midpoint, e.g. group {int(loose[i])} element "
                                 f"{int(e)}: oracle {ob16[i, e]:#06x} gpu {gb16[i, e]:#06x} fp32 r {r32[i, e]!r}")
        else:
            scale = np.max(np.abs(orr), axis=1, keepdims=True)
            ok = np.abs(orr.astype(np.float64) - grr.astype(np.float64)) <= 1e-5 * scale + 1e-30
            bad = cmp & ~np.all(ok, axis=1)
            if bad.any():
                fails.append(f"{int(bad.sum())} groups with fp32 r outside 1e-5")
            bad = cmp & ab_same & ~np.all(orr == grr, axis=1)
            if bad.any():
                fails.append(f"{int(bad.sum())} groups with identical (s, z) but different fp32 r")

    if gpu.get("err") is not None:
        oe, ge = o["err"].astype(np.float64), gpu["err"].astype(np.float64)
        rel = np.abs(ge - oe) <= 1e-5 * oe + 1e-37
        ok = rel | (np.abs(ge - oe) <= 1e-5 * oe + floor + 1e-37)
        st["err_floor"] += int((cmp & ok & ~rel).sum())
        bad = cmp & ~ok
        if bad.any():
            k = np.flatnonzero(bad)[:5]
            fails.append(f"{int(bad.sum())} groups with err outside 1e-5, e.g. {k.tolist()} "
                         f"oracle {oe[k].tolist()} gpu {ge[k].tolist()}")
    st["clip_lt_1"] = int(np.count_nonzero(o["best"] != 0))
    return fails, st
