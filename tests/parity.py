"""Tolerances of the GPU-vs-reference comparisons, and helpers that run the
GPU library through its C ABI binding.

Gates (fp32 GPU against the fp64 reference, same seeded inputs):

* parameters, every tensor t, every element i:
      |gpu_i - ref_i| <= 1e-4 * max(|ref_i|, f * rms(ref_t))
  a relative error of 1e-4 with a floor on the denominator.  The error of a
  weight that lands near zero after a step is the fp32 error of its update
  (eta/B) * G, not a fraction of its own value, so a floor is needed.  The
  full-size workloads are gated with f = 1e-3 (SMALL_FLOOR), in every
  step-along comparison and in the free-running ones of networks without
  kinks; the chaotic free-running relu schedule and the small edge-case
  networks use f = 1 (an independent fp32 computation of the same step,
  numpy float32 products on the CPU, reaches 1.0-1.7e-4 under f = 1e-3 on
  the first layer of the 784-30-10 and 784-100-100-10 workloads, so f = 1e-3
  holds only for an implementation whose sums are that accurate).  Every
  comparison reports the error under both floors and the unfloored largest
  relative error with the element that holds it (tensor_report).
* update, every tensor, in the step-along comparisons (both sides start from
  the same theta_t): with d_gpu = theta_gpu - theta_t and the exact
  d_ref = -(eta/B) G_ref,
      max_i (|d_gpu,i - d_ref,i| - ulp(theta_gpu,i) / 2) <= 1e-3 * max_i |d_ref,i|
  The half ulp is the rounding of the stored fp32 result, which no fp32
  implementation can avoid; where the step is small against the parameters
  (the 4096^4-10 workload moves b_1 by ~1e-4 of its size) it is of the same
  order as the gate.  This check is what sees an update that was not applied:
  the parameter gate alone passes a parameter that did not move when the
  step is below 1e-4 of the tensor's rms.
* tendencies (the batch-summed gradient of the last step): the parameter
  rule elementwise with tolerance 1e-4.  For networks with relu units the
  tendencies depend on which side of the kink each unit falls, and a unit
  whose pre-activation lies within rounding of zero may fall on either side
  in any fp32 computation, both results being correct.  Such comparisons
  take the GPU's own decisions for the units within KINK_BAND * rms(z of the
  layer) of the kink (nf_get_fprime), require the GPU to decide every other
  unit as the reference does, and then compare elementwise: the result is
  unique once those decisions are fixed.
* network outputs (inference): the parameter rule with tolerance 1e-4.
"""

from __future__ import annotations

import json
import sys
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

PARAM_TOL = 1e-4
GRAD_TOL = 1e-4
UPDATE_TOL = 1e-3
OUT_TOL = 1e-4
SMALL_FLOOR = 1e-3      # the smaller floor, reported beside the gated one
KINK_BAND = 1e-4        # relu units within this * rms(z) of the kink take the GPU's side


def tensor_slices(dims: Sequence[int]) -> List[Tuple[str, slice]]:
    out, off = [], 0
    for l in range(1, len(dims)):
        n = dims[l] * dims[l - 1]
        out.append((f"W{l}", slice(off, off + n)))
        off += n
        out.append((f"b{l}", slice(off, off + dims[l])))
        off += dims[l]
    return out


def floored_rel(got, ref, floor: float = 1.0) -> Tuple[float, int]:
    """Largest |got - ref| / max(|ref|, floor * rms(ref)) and where it is."""
    got = np.asarray(got, dtype=np.float64).ravel()
    ref = np.asarray(ref, dtype=np.float64).ravel()
    if ref.size == 0:
        return 0.0, -1
    if not np.all(np.isfinite(got)):
        return float("inf"), int(np.argmax(~np.isfinite(got)))
    rms = float(np.sqrt(np.mean(ref * ref)))
    den = np.maximum(np.abs(ref), floor * rms)
    den[den == 0] = 1.0
    err = np.abs(got - ref) / den
    i = int(np.argmax(err))
    return float(err[i]), i


def tensor_report(got, ref) -> Dict:
    """The gated error (rms floor), the error under the 1e-3 * rms floor, and
    the unfloored largest relative error with its element and values."""
    g = np.asarray(got, dtype=np.float64).ravel()
    r = np.asarray(ref, dtype=np.float64).ravel()
    e, i = floored_rel(g, r, 1.0)
    e3, i3 = floored_rel(g, r, SMALL_FLOOR)
    nz = r != 0
    if np.any(nz) and np.all(np.isfinite(g)):
        rel = np.full(r.shape, 0.0)
        rel[nz] = np.abs(g[nz] - r[nz]) / np.abs(r[nz])
        j = int(np.argmax(rel))
        raw = {"rel": float(rel[j]), "at": j, "gpu": float(g[j]), "ref": float(r[j])}
    else:
        raw = None
    return {"gated": e, "at": i, "floor_1e-3": e3, "floor_1e-3_at": i3, "unfloored": raw}


def check_params(got, ref, dims, tol=PARAM_TOL, what="params", report=None,
                 floor: float = 1.0) -> List[str]:
    """Elementwise gate per tensor, the denominator floored at floor * rms of
    the tensor (1: the rms floor; SMALL_FLOOR: the 1e-3 * rms floor); report
    (a dict) collects tensor_report."""
    fails = []
    for name, sl in tensor_slices(dims):
        rep = tensor_report(got[sl], ref[sl])
        if report is not None:
            report[name] = rep
        e, i = (rep["gated"], rep["at"]) if floor == 1.0 else floored_rel(got[sl], ref[sl], floor)
        if not e <= tol:
            fails.append(f"{what} {name}: relative error {e:.3e} (floor {floor:g} rms) > {tol:g} "
                         f"at {i} (gpu {got[sl][i]!r}, ref {ref[sl][i]!r})")
    return fails


def check_grads(got, ref, dims, tol=GRAD_TOL, report=None) -> List[str]:
    """Tendencies, elementwise.  Relu networks must be compared against a
    reference that took the GPU's decisions at the kink (see kink_sides)."""
    return check_params(got, ref, dims, tol, "grads", report)


def check_update(got, theta_t, ref_grad, scale: float, dims, tol=UPDATE_TOL,
                 report=None) -> List[str]:
    """The applied step against the exact step -(eta/B) G_ref from the same
    theta_t, allowing the half ulp of the stored fp32 result (module doc)."""
    fails = []
    for name, sl in tensor_slices(dims):
        p = np.asarray(got[sl], dtype=np.float32)
        d_gpu = p.astype(np.float64) - np.asarray(theta_t[sl], dtype=np.float32).astype(np.float64)
        d_ref = -scale * np.asarray(ref_grad[sl], dtype=np.float64)
        dinf = float(np.max(np.abs(d_ref))) if d_ref.size else 0.0
        if not np.all(np.isfinite(d_gpu)):
            fails.append(f"update {name}: non-finite parameters")
            continue
        half_ulp = np.spacing(np.abs(p)).astype(np.float64) / 2
        diff = np.abs(d_gpu - d_ref)
        if dinf == 0.0:
            if np.any(diff > half_ulp):
                fails.append(f"update {name}: parameters moved where the step is zero")
            if report is not None:
                report[name] = {"raw": 0.0, "gated": 0.0, "storage": 0.0}
            continue
        raw = float(np.max(diff)) / dinf
        adj = float(np.max(np.maximum(diff - half_ulp, 0.0))) / dinf
        if report is not None:
            report[name] = {"raw": raw, "gated": adj, "storage": float(np.max(half_ulp)) / dinf}
        if not adj <= tol:
            i = int(np.argmax(np.maximum(diff - half_ulp, 0.0)))
            fails.append(f"update {name}: {adj:.3e} of the largest step > {tol:g} at {i} "
                         f"(gpu step {d_gpu[i]!r}, reference step {d_ref[i]!r})")
    return fails


def full_acts(dims, acts) -> List[str]:
    return list(acts) * (len(dims) - 1) if len(acts) == 1 else list(acts)


def has_kinks(acts) -> bool:
    return any(a in ("relu", "step") for a in acts)


def gpu_kink_sides(nf, h, dims, acts, batch) -> Optional[list]:
    """The GPU's relu decisions of the last training step, per layer (None for
    other layers and for the output layer, whose f' is not kept), or None when
    the step kept f' in registers."""
    acts = full_acts(dims, acts)
    L = len(dims) - 1
    out = []
    for l in range(1, L + 1):
        if acts[l - 1] != "relu" or l == L:
            out.append(None)
            continue
        try:
            out.append(nf.nf_get_fprime(h, l, batch, dims[l]))
        except nf.NfError as e:
            if e.status != nf.NF_EINVAL:
                raise
            return None
    return out


def check_kink_sides(sides, theta, dims, acts, X, band=KINK_BAND, stats=None) -> List[str]:
    """The GPU's relu decisions must equal the reference's own for every unit
    outside the band; stats collects, per layer, the units in the band and how
    many of them the GPU put on the other side from the reference."""
    from oracle import mlp
    acts = full_acts(dims, acts)
    Z, _ = mlp.forward(theta, dims, acts, X)
    fails = []
    for l, sd in enumerate(sides):
        if sd is None:
            continue
        z = Z[l + 1]
        own = z > 0
        gpu = np.asarray(sd) > 0
        near = mlp.kink_band(z, band)
        off = (gpu != own) & ~near
        if stats is not None:
            stats[f"z{l + 1}"] = {"in_band": int(near.sum()),
                                  "other_side_in_band": int(((gpu != own) & near).sum()),
                                  "other_side_outside": int(off.sum())}
        if off.any():
            s, j = np.argwhere(off)[0]
            rms = float(np.sqrt(np.mean(z * z)))
            fails.append(f"layer {l + 1}: {int(off.sum())} relu decisions differ outside the band, "
                         f"e.g. sample {s} unit {j} at z = {z[s, j]:.3e} ({abs(z[s, j]) / rms:.2e} rms)")
    return fails


def emit(tag: str, record: Dict) -> None:
    """One machine-readable line of measured errors on stderr."""
    print(f"[parity-json] {tag} " + json.dumps(record, default=float), file=sys.stderr, flush=True)


def worst(report: Dict, key: str = "gated") -> float:
    vals = [v[key] for v in report.values() if isinstance(v, dict) and key in v]
    return max(vals) if vals else 0.0


def relu_clear(theta, dims, acts, X, rel=1e-3) -> bool:
    """True when no relu / step pre-activation of the reference forward pass on
    X lies within rel * (that layer's rms |z|) of zero, so that rounding cannot
    flip a unit across the kink and gradients can be compared elementwise
    without the GPU's decisions (used where the GPU keeps f' in registers)."""
    from oracle import mlp
    acts = full_acts(dims, acts)
    Z, _ = mlp.forward(theta, dims, acts, X)
    for l, a in enumerate(acts):
        if a in ("relu", "step"):
            z = Z[l + 1]
            if np.min(np.abs(z)) < rel * np.sqrt(np.mean(z * z)):
                return False
    return True
