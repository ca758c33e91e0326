"""GPU library against the CPU reference on the five benchmark workloads at
their full sizes, in the launch configuration bench.py times.

Two comparisons per workload:

* step along the reference: before every step the GPU net is loaded with the
  reference's parameters for that step (data flows from the reference to the
  GPU only), takes one step, and its parameters and tendencies are compared
  with the reference's next step.  Every step of the schedule is gated at the
  fixed tolerances of tests/parity.py.
* free-running trajectory: the GPU trains on its own from the seeded initial
  parameters and is compared after every step.  Where the schedule is chaotic
  the result after t steps is not determined to fp32 precision: for networks
  with relu units the reference is run a second time with the other side of
  the kink taken by every unit within 1e-5 * rms(z) of it (units an fp32
  computation may legitimately put on either side), and the gate after step t
  is max(fixed tolerance, 2 * the spread between those two reference runs).
  Networks without kinks keep the fixed tolerance throughout.
"""

import sys

import numpy as np
import pytest

from oracle import mlp
from paper_1902_06714_amd import workloads as W

from . import parity
from .gpu_run import GpuNet, note, to_dev

pytestmark = pytest.mark.gpu

KINK_TOL = 1e-5


def _tensor_spread(a, b, dims):
    out = {}
    for name, sl in parity.tensor_slices(dims):
        out[name] = parity.floored_rel(b[sl], a[sl])[0]
    return out


def _tensor_fro(a, b, dims):
    out = {}
    for name, sl in parity.tensor_slices(dims):
        n = np.linalg.norm(a[sl])
        out[name] = float(np.linalg.norm(np.asarray(b[sl], np.float64) - a[sl]) / n) if n > 0 else 0.0
    return out


def _reference(w, X, Y, theta, steps, shards, kink_tol=0.0):
    thetas, grads = [theta], []
    for t in range(steps):
        sl = slice(t * w.batch, (t + 1) * w.batch)
        new, G = mlp.train_batch(thetas[-1], w.dims, list(w.acts), X[sl], Y[sl], w.eta, shards,
                                 kink_tol=kink_tol)
        thetas.append(new)
        grads.append(G)
    return thetas, grads


def _run(name, steps=None, shards=None):
    w = W.WORKLOADS[name]
    steps = w.steps if steps is None else steps
    shards = w.shards if shards is None else shards
    acts = list(w.acts)
    kinked = any(a in ("relu", "step") for a in acts)
    X, Y = W.make_data(w, w.batch * steps)
    theta0 = W.make_params(w)
    ref_t, ref_g = _reference(w, X, Y, theta0, steps, shards)
    if kinked:
        alt_t, alt_g = _reference(w, X, Y, theta0, steps, shards, KINK_TOL)
    xd, yd = to_dev(X), to_dev(Y)
    fails, worst = [], {"step_p": 0.0, "step_g": 0.0, "free_p": 0.0}
    note(f"{name}: {w.dims} batch={w.batch} shards={shards} steps={steps}")
    with GpuNet(w.dims, acts, theta0) as net:
        # step along the reference
        for t in range(steps):
            sl = slice(t * w.batch, (t + 1) * w.batch)
            net.nf.nf_set_params(net.h, ref_t[t])
            net.train_batch(xd[sl], yd[sl], w.eta, shards)
            p, g = net.params(), net.grads()
            fails += [f"step-along {t}: {m}" for m in parity.check_params(p, ref_t[t + 1], w.dims)]
            fails += [f"step-along {t}: {m}" for m in parity.check_grads(g, ref_g[t], w.dims, acts)]
            worst["step_p"] = max(worst["step_p"], max(_tensor_spread(ref_t[t + 1], p, w.dims).values()))
        # free-running trajectory
        net.nf.nf_set_params(net.h, theta0)
        for t in range(steps):
            sl = slice(t * w.batch, (t + 1) * w.batch)
            net.train_batch(xd[sl], yd[sl], w.eta, shards)
            p, g = net.params(), net.grads()
            gp = _tensor_spread(ref_t[t + 1], p, w.dims)
            gg = _tensor_fro(ref_g[t], g, w.dims)
            if kinked:
                sp = _tensor_spread(ref_t[t + 1], alt_t[t + 1], w.dims)
                sg = _tensor_fro(ref_g[t], alt_g[t], w.dims)
            for tn, _ in parity.tensor_slices(w.dims):
                tol_p = parity.PARAM_TOL
                tol_g = parity.GRAD_FRO_TOL_RELU if kinked else None
                if kinked:
                    tol_p = max(tol_p, 2 * sp[tn])
                    tol_g = max(tol_g, 2 * sg[tn])
                if not gp[tn] <= tol_p:
                    fails.append(f"free {t}: params {tn} {gp[tn]:.3e} > {tol_p:.3e}")
                if tol_g is not None and not gg[tn] <= tol_g:
                    fails.append(f"free {t}: grads {tn} Frobenius {gg[tn]:.3e} > {tol_g:.3e}")
            if not kinked:
                fails += [f"free {t}: {m}" for m in parity.check_grads(g, ref_g[t], w.dims, acts)]
            worst["free_p"] = max(worst["free_p"], max(gp.values()))
        final = net.params()
        if w.heldout:
            Xh, _ = W.make_data(w, heldout=True)
            note(f"{name}: inference on {Xh.shape[0]} held-out samples")
            net.nf.nf_set_params(net.h, ref_t[-1])
            out = net.forward(to_dev(Xh))
            e, _ = parity.floored_rel(out, mlp.output(ref_t[-1], w.dims, acts, Xh))
            if not e <= parity.OUT_TOL:
                fails.append(f"inference: floored relative error {e:.3e}")
    print(f"[parity] {name}: worst step-along param error {worst['step_p']:.2e}, "
          f"worst free-running param error {worst['free_p']:.2e}", file=sys.stderr, flush=True)
    assert not fails, "\n".join(fails[:30])
    return w, X, Y, theta0, final


def test_c1_784_30_10_batch100():
    _run("c1")


def test_c2_784_30_10_epoch_and_inference():
    w, X, Y, theta, final = _run("c2")
    # the whole epoch in one call gives the same bits as step-by-step calls
    note("c2: nf_train_epoch")
    with GpuNet(w.dims, list(w.acts), theta) as net:
        net.train_epoch(to_dev(X), to_dev(Y), w.batch, w.eta, w.shards)
        assert np.array_equal(net.params(), final)


def test_c3_784_100_100_10_sixteen_shards():
    _run("c3")


@pytest.mark.timeout(600)
def test_c4_784_1024x3_10():
    _run("c4")


@pytest.mark.timeout(900)
def test_c5_4096x4_10():
    _run("c5")
