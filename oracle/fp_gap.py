"""Where the integer block departs from the floating-point block (test infrastructure).

The whole-block check compares S_y y of the integer block (Sec. 3.1: Eq. 7 projections,
Eq. 8 scores with Phi, the fused requantization of Eq. 11, I-BERT's integer softmax,
A.V requantized by Eq. 7, the output projection) with the real-valued block of
Eq. 8-9 on the same dequantized inputs (``fp_block``).  This module evaluates the
block with a switch per integer stage, so that the gap can be attributed:

  proj   Q, K, V and P requantized to int8 (Eq. 7)
  score  the fused score requantized to int8 (Eq. 11)
  exp    I-BERT's second-order polynomial exp with the shift by z (instead of exp)
  norm   the 8-bit probabilities floor(e floor(2^32 / sum) / 2^24), clamped to 255
         (instead of e / sum)
  ctx    the context requantized to int8 (Eq. 7 with m_o)
  out    the block output requantized to int8 (Eq. 7)

A stage that is on and receives integers evaluates exactly the integer formula of the
oracle; a stage that is on and receives real numbers (an earlier stage is off) applies
the same grid to them: round half up onto the stage's output grid and clamp to +-127
(score, ctx, out), the polynomial on the real distance (exp), floor onto the 2^-8
probability grid (norm).  A stage that is off passes real numbers on.  With every
stage on the result equals the C oracle byte for byte, and with every stage off it
is ``fp_block.block`` (both pinned in the tests), so the switches sit between two
independently written ends.

Integer contractions are evaluated in float64 matrix products: every partial sum is
an integer below 2^53, so they are exact.  F = floor(2^32 / sum) is taken in int64.

Run as a script, it prints the tables reported in the design notes and writes
``oracle/fp_gap_results.json``.
"""

from __future__ import annotations

import json
import math
import os
import sys
import time
from typing import Dict, Optional

import numpy as np

STAGES = ("proj", "score", "exp", "norm", "ctx", "out")
ALL_ON = {s: True for s in STAGES}
ALL_OFF = {s: False for s in STAGES}


def _rs(acc: np.ndarray, m, n: int) -> np.ndarray:
    """Eq. 7's RS(a, m, n) = floor((a m + 2^(n-1)) / 2^n) on integer-valued float64
    arrays (a m below 2^53 here, so exact)."""
    return np.floor((acc * np.asarray(m, dtype=np.float64) + float(1 << (n - 1))) / float(1 << n))


def _clamp8(v: np.ndarray) -> np.ndarray:
    return np.clip(v, -127.0, 127.0)


def _round_grid(v: np.ndarray, S: float) -> np.ndarray:
    """A real value onto an int8 grid of step S: round half up, clamp (the real-input
    form of a requantization)."""
    return _clamp8(np.floor(v / S + 0.5))


def block(blk, stages: Dict[str, bool], x: Optional[np.ndarray] = None, x_real: Optional[np.ndarray] = None,
          lengths=None) -> np.ndarray:
    """Real-valued output [B][T][d] of the block with the given stages integer.

    ``x`` is the int8 input (default: the block's); ``x_real``, when given, is a real
    input used instead (a stack fed by a real-valued previous block); rows i >= L_b are
    zero.  Returns S_y y when ``out`` is on, the real output otherwise.
    """
    st = dict(ALL_OFF, **stages)
    sc, c = blk.scales, blk.consts
    sh = blk.shape
    H, dk, d = sh.n_heads, sh.d_k, sh.d_model
    lengths = blk.lengths if lengths is None else lengths
    Wr = {w: np.asarray(sc["S_W" + w], dtype=np.float64)[:, None] * getattr(blk, "w_" + w).astype(np.float64)
          for w in ("q", "k", "v", "pos", "out")}
    Wi = {w: getattr(blk, "w_" + w).astype(np.float64) for w in ("q", "k", "v", "pos", "out")}
    pe = blk.pos_table.astype(np.float64)

    # ---- projections (Eq. 7): integers on the Q, K, V, P grids, or real values
    if x_real is None:
        xi = (blk.x if x is None else x).astype(np.float64)
        B, T, _ = xi.shape
        integer_in = True
    else:
        xr_in = np.asarray(x_real, dtype=np.float64)
        B, T, _ = xr_in.shape
        integer_in = False
    proj_int = st["proj"] and integer_in
    grids = {"q": "S_Q", "k": "S_K", "v": "S_V"}
    Qi = {}  # integer tensors (when proj_int)
    R = {}  # real tensors
    for w in ("q", "k", "v"):
        if integer_in:
            acc = xi @ Wi[w].T
            if st["proj"]:
                Qi[w] = _clamp8(_rs(acc, c["mult_" + w], c["shift_" + w]))
                R[w] = sc[grids[w]] * Qi[w]
            else:
                R[w] = sc["S_x"] * (xi @ Wr[w].T)
        else:
            r = xr_in @ Wr[w].T
            R[w] = sc[grids[w]] * _round_grid(r, sc[grids[w]]) if st["proj"] else r
    acc_p = pe @ Wi["pos"].T
    if st["proj"]:
        Pi = _clamp8(_rs(acc_p, c["mult_pos"], c["shift_pos"]))
        Pr = sc["S_P"] * Pi
    else:
        Pr = sc["S_pe"] * (pe @ Wr["pos"].T)
    ui = blk.pos_bias_u.astype(np.float64)
    vi = blk.pos_bias_v.astype(np.float64)

    S_s, S_A, S_O, S_y = sc["S_s"], sc["S_A"], sc["S_O"], sc["S_y"]
    q_ln2, q_b, q_c = c["q_ln2"], c["q_b"], c["q_c"]
    ctx_int = st["ctx"] and proj_int and st["norm"] and st["exp"] and st["score"]
    ctx = np.zeros((B, T, d))  # real context
    ctx_i = np.zeros((B, T, d))  # integer context (when ctx_int)
    rows = np.arange(T)[:, None]
    cols = np.arange(T)[None, :]
    for b in range(B):
        L = int(lengths[b])
        for h in range(H):
            hs = slice(h * dk, (h + 1) * dk)
            # ---- Eq. 8 with Phi as the index map r = j - i + T - 1
            if proj_int:
                qi = Qi["q"][b, :, hs]
                cm = (qi + ui[h]) @ Qi["k"][b, :, hs].T  # integers
                pm = ((qi + vi[h]) @ Pi[:, hs].T)[rows, cols - rows + T - 1]
                z = (cm * sc["S_Q"] * sc["S_K"] + pm * sc["S_Q"] * sc["S_P"]) / math.sqrt(dk)
            else:
                q = R["q"][b, :, hs]
                z = ((q + sc["S_Q"] * ui[h]) @ R["k"][b, :, hs].T +
                     ((q + sc["S_Q"] * vi[h]) @ Pr[:, hs].T)[rows, cols - rows + T - 1]) / math.sqrt(dk)
            z = z[:L, :L]
            # ---- Eq. 11: int8 score on the grid S_s
            score_int = st["score"] and proj_int
            if st["score"]:
                if proj_int:
                    s = _clamp8(_rs(c["m_c"] * cm[:L, :L] + c["m_p"] * pm[:L, :L], 1, c["shift_s"]))
                else:
                    s = _round_grid(z, S_s)
                dist = s.max(axis=1, keepdims=True) - s  # in score steps
                dreal = S_s * dist
            else:
                dreal = z.max(axis=1, keepdims=True) - z
                dist = dreal / S_s
            # ---- exp: I-BERT's polynomial (integer or on the real distance), or exp
            exp_int = st["exp"] and score_int
            if st["exp"]:
                zq = np.floor(dist / q_ln2)
                r = zq * q_ln2 - dist
                Lr = (r + q_b) ** 2 + q_c
                e = np.where(zq >= 62, 0.0, Lr / np.exp2(np.minimum(zq, 62)))
                if exp_int:
                    e = np.floor(e)
            else:
                e = np.exp(-dreal)
            # ---- normalization: 8-bit floored probabilities, or e / sum
            if st["norm"]:
                if exp_int:
                    ei = e.astype(np.int64)
                    tot = ei.sum(axis=1, keepdims=True)
                    F = np.where(tot > 0, (np.int64(1) << 32) // np.maximum(tot, 1), 0)
                    a = np.minimum((ei * F) >> 24, 255).astype(np.float64)
                else:
                    a = np.minimum(np.floor(256.0 * e / e.sum(axis=1, keepdims=True)), 255.0)
                prob = S_A * a
            else:
                prob = e / e.sum(axis=1, keepdims=True)
            # ---- A.V and the context grid (Eq. 7 with m_o)
            if ctx_int:
                acc = a @ Qi["v"][b, :L, hs]
                ctx_i[b, :L, hs] = _clamp8(_rs(acc, c["m_o"], c["shift_o"]))
            else:
                cr = prob @ R["v"][b, :L, hs]
                ctx[b, :L, hs] = S_O * _round_grid(cr, S_O) if st["ctx"] else cr
    # ---- output projection (Eq. 7)
    if ctx_int:
        y = (S_y * _clamp8(_rs(ctx_i @ Wi["out"].T, c["mult_out"], c["shift_out"])) if st["out"]
             else S_O * (ctx_i @ Wr["out"].T))
    else:
        yr = ctx @ Wr["out"].T
        y = S_y * _round_grid(yr, S_y) if st["out"] else yr
    for b in range(B):
        y[b, int(lengths[b]):] = 0.0
    return y


def rel_l2(approx: np.ndarray, ref: np.ndarray) -> float:
    return float(np.linalg.norm((approx - ref).ravel()) / max(np.linalg.norm(ref.ravel()), 1e-300))


def row_mass(blk) -> np.ndarray:
    """Sum of the 8-bit probability codes of every valid (utterance, head, row), as the
    integer block computes them (256 is a full row)."""
    from oracle import core

    _, tr = core.relpos_attn(blk, trace_scores=True)
    out = []
    for b in range(blk.x.shape[0]):
        L = int(blk.lengths[b])
        out.append(tr["a"][b, :, :L, :L].astype(np.int64).sum(axis=-1).ravel())
    return np.concatenate(out)


def attribution(blk) -> Dict[str, float]:
    """rel-L2 against the FP block for: every stage integer, every stage but one
    integer ("-stage"), only one stage integer ("+stage"), and none."""
    ref = block(blk, ALL_OFF)
    res = {"all": rel_l2(block(blk, ALL_ON), ref)}
    for s in STAGES:
        res["-" + s] = rel_l2(block(blk, dict(ALL_ON, **{s: False})), ref)
    for s in STAGES:
        res["+" + s] = rel_l2(block(blk, dict(ALL_OFF, **{s: True})), ref)
    return res


def stack_gap(wl) -> float:
    """rel-L2 of the integer stack's output against the FP stack on the same inputs
    (each FP block fed by the FP output of the one before)."""
    from oracle import core

    x = wl.blocks[0].x
    xr = None
    for i, blk in enumerate(wl.blocks):
        x = core.relpos_attn(blk, x=x)
        yr = block(blk, ALL_OFF, x=wl.blocks[0].x if i == 0 else None, x_real=xr)
        xr = yr
    last = wl.blocks[-1]
    return rel_l2(last.scales["S_y"] * x.astype(np.float64), xr)


def main(out_path: Optional[str] = None):
    here = os.path.dirname(os.path.abspath(__file__))
    sys.path.insert(0, os.path.dirname(here))
    from oracle import core
    from workloads import make_workload

    results = {"regime": "calibrated", "configs": {}, "attribution": {}, "sweep": []}
    t0 = time.time()
    for name in ("tiny", "parakeet", "batched", "longform"):
        blk = make_workload(name, "calibrated").blocks[0]
        y = core.relpos_attn(blk)
        ref = block(blk, ALL_OFF)
        err = rel_l2(blk.scales["S_y"] * y.astype(np.float64), ref)
        mass = row_mass(blk) if name != "longform" else None
        results["configs"][name] = {
            "T": int(blk.T), "B": int(blk.x.shape[0]), "rel_l2": err,
            "mean_row_mass": None if mass is None else float(mass.mean()),
            "rows_below_128": None if mass is None else float(np.mean(mass < 128)),
        }
        print(f"[gap] {name}: rel-L2 {err:.4f}  ({time.time() - t0:.0f} s)", flush=True)
        if name in ("tiny", "parakeet", "longform"):
            results["attribution"][name] = attribution(blk)
            print(f"[gap] {name} attribution: " + ", ".join(f"{k} {v:.4f}" for k, v in results["attribution"][name].items()),
                  flush=True)
    wl = make_workload("stack", "calibrated")
    results["configs"]["stack"] = {"T": int(wl.blocks[0].T), "B": int(wl.blocks[0].x.shape[0]),
                                   "layers": len(wl.blocks), "rel_l2": stack_gap(wl)}
    wl1 = make_workload("stack", "calibrated", layers=1)
    results["configs"]["stack"]["rel_l2_first_block"] = rel_l2(
        wl1.blocks[0].scales["S_y"] * core.relpos_attn(wl1.blocks[0]).astype(np.float64), block(wl1.blocks[0], ALL_OFF))
    print(f"[gap] stack: {results['configs']['stack']}", flush=True)
    # the scale sweep on the tiny workload: S_x S_W over [2^-18, 2^-14] in quarter
    # octaves (S_x fixed, every weight matrix's per-channel scales moved together)
    probe = make_workload("tiny", "calibrated").blocks[0]
    best = None
    for k in range(17):
        prod = 2.0 ** (-18 + 0.25 * k)
        blk = make_workload("tiny", "calibrated", w_scale=prod / probe.scales["S_x"]).blocks[0]
        y = core.relpos_attn(blk)
        ref = block(blk, ALL_OFF)
        rec = {
            "SxSW": prod, "log2_SxSW": -18 + 0.25 * k, "S_s": blk.scales["S_s"],
            "rel_l2": rel_l2(blk.scales["S_y"] * y.astype(np.float64), ref),
            "rel_l2_norm_float": rel_l2(block(blk, dict(ALL_ON, norm=False)), ref),
            "rel_l2_score_float": rel_l2(block(blk, dict(ALL_ON, score=False)), ref),
        }
        results["sweep"].append(rec)
        if best is None or rec["rel_l2"] < best[0]["rel_l2"]:
            best = (rec, blk)
        print(f"[gap] sweep {rec}", flush=True)
    results["sweep_best"] = dict(best[0], attribution=attribution(best[1]))
    print(f"[gap] best {results['sweep_best']}", flush=True)
    # the stack: how the gap grows through the layers (first six)
    x = wl.blocks[0].x
    xr = None
    per_layer = []
    for i, blk in enumerate(wl.blocks[:6]):
        x = core.relpos_attn(blk, x=x)
        xr = block(blk, ALL_OFF, x=wl.blocks[0].x if i == 0 else None, x_real=xr)
        per_layer.append({"layer": i, "rel_l2": rel_l2(blk.scales["S_y"] * x.astype(np.float64), xr),
                          "saturated": float(np.mean(np.abs(x) == 127))})
    results["configs"]["stack"]["first_layers"] = per_layer
    out_path = out_path or os.path.join(here, "fp_gap_results.json")
    with open(out_path, "w") as fh:
        json.dump(results, fh, indent=1)
    print(f"[gap] wrote {out_path} in {time.time() - t0:.0f} s")
    return results


if __name__ == "__main__":
    main()
