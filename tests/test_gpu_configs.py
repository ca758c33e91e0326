"""GPU library against the CPU reference on the five benchmark workloads at
their full sizes, in the launch configuration bench.py times.

Two comparisons per workload (the gates are those of tests/parity.py; the
parameters, and the held-out outputs of the 784-30-10 workload, are gated at
1e-4 with the 1e-3 * rms floor of the denominator, except the free-running
relu trajectories below, which keep the rms floor):

* step along the reference: before every step the GPU net is loaded with the
  reference's parameters theta_t for that step (data flows from the
  reference to the GPU only) and takes one step.  Its parameters, its
  tendencies and the step it applied are compared with the reference's step
  from the same theta_t.
* free-running trajectory: the GPU trains on its own from the seeded initial
  parameters, the reference likewise, and the parameters are compared after
  every step (the tendencies too for networks without kinks).

For networks with relu units the reference step takes the GPU's decisions
for the units within KINK_BAND * rms(z) of the kink, where the method leaves
the side to rounding (nf_get_fprime), and every other unit must be decided
as the reference decides it.  The free-running reference takes the free
GPU run's decisions step by step in the same way; the distance to the plain
reference (which decides every unit itself) and the spread of the plain
reference under the other choice for the band units are reported beside it.

The 784-1024^3-10 schedule is chaotic in its last steps: the reference with
every parameter moved by one ulp before every step separates from itself by
1.2e-5 after 10 steps but 6e-4 after 16.  The free-running gate after step t
is therefore max(1e-4, 4 x that one-ulp spread at t), computed here from the
reference alone; after 10 steps it is the fixed 1e-4.
"""

import sys

import numpy as np
import pytest

from oracle import mlp
from paper_1902_06714_amd import workloads as W

from . import parity
from .gpu_run import GpuNet, note, to_dev

pytestmark = pytest.mark.gpu


def _reference(w, X, Y, theta, steps, shards, kink_tol=0.0):
    thetas, grads = [theta], []
    for t in range(steps):
        sl = slice(t * w.batch, (t + 1) * w.batch)
        new, G = mlp.train_batch(thetas[-1], w.dims, list(w.acts), X[sl], Y[sl], w.eta, shards,
                                 kink_tol=kink_tol)
        thetas.append(new)
        grads.append(G)
    return thetas, grads


def _kink_step(w, theta, X, Y, shards, sides, band=parity.KINK_BAND):
    if sides is None:       # already a failure; the plain step keeps the rest meaningful
        return mlp.train_batch(theta, w.dims, list(w.acts), X, Y, w.eta, shards)
    return mlp.train_batch(theta, w.dims, list(w.acts), X, Y, w.eta, shards,
                           kink_tol=band, kink_given=sides)


def _sides(net, w, theta, X, fails, what, band=parity.KINK_BAND):
    sides = parity.gpu_kink_sides(net.nf, net.h, w.dims, w.acts, X.shape[0])
    if sides is None:
        fails.append(f"{what}: the GPU step kept no relu decisions")
        return None, {}
    stats = {}
    fails += [f"{what}: {m}" for m in parity.check_kink_sides(sides, theta, w.dims, w.acts, X,
                                                              band=band, stats=stats)]
    return sides, stats


def _ulp_spread(w, X, Y, theta0, ref_t, steps, shards):
    """The reference's own sensitivity to fp32 storage: its trajectory with
    every parameter moved by one fp32 ulp (seeded random signs) before every
    step, taking the unmoved trajectory's relu decisions inside the kink band,
    against the unmoved trajectory.  Worst floored parameter error after each
    step.  Every fp32 step stores the parameters to one ulp, so this is the
    kind of deviation any fp32 computation adds, as the schedule amplifies it."""
    rng = np.random.default_rng(20260)
    acts = parity.full_acts(w.dims, w.acts)
    L = len(w.dims) - 1
    b = theta0
    out = []
    for t in range(steps):
        sl = slice(t * w.batch, (t + 1) * w.batch)
        b = (b + np.where(rng.random(b.size) < 0.5, -1.0, 1.0)
             * np.spacing(np.abs(b))).astype(np.float32)
        Za, _ = mlp.forward(ref_t[t], w.dims, acts, X[sl])
        sides = [(Za[l] > 0).astype(np.float32) if acts[l - 1] == "relu" and l < L else None
                 for l in range(1, L + 1)]
        b, _ = mlp.train_batch(b, w.dims, acts, X[sl], Y[sl], w.eta, shards,
                               kink_tol=parity.KINK_BAND, kink_given=sides)
        rep = {}
        parity.check_params(b, ref_t[t + 1], w.dims, report=rep)
        out.append(parity.worst(rep))
    return out


# the free-running gate after step t is max(PARAM_TOL, CHAOS_MARGIN * the
# reference's one-ulp spread at t): the GPU's trajectory carries its own
# sample of that rounding noise (measured at 0.5-1.4 times the reference's
# sample over the 784-1024^3-10 schedule), while a step applied wrongly moves
# the parameters by orders of magnitude more
CHAOS_MARGIN = 4.0


def _run(name, steps=None, shards=None):
    w = W.WORKLOADS[name]
    steps = w.steps if steps is None else steps
    shards = w.shards if shards is None else shards
    acts = list(w.acts)
    kinked = "relu" in parity.full_acts(w.dims, acts)
    scale = w.eta / w.batch
    X, Y = W.make_data(w, w.batch * steps)
    theta0 = W.make_params(w)
    ref_t, ref_g = _reference(w, X, Y, theta0, steps, shards)
    # free-running gate after step t: max(PARAM_TOL, CHAOS_MARGIN * the
    # reference's own one-ulp spread at t); the kink band widens the same way,
    # since two trajectories that far apart may decide units that far from the
    # kink differently.  Networks without kinks keep the fixed gate.
    ulp_spread = _ulp_spread(w, X, Y, theta0, ref_t, steps, shards) if kinked else [0.0] * steps
    xd, yd = to_dev(X), to_dev(Y)
    fails = []
    worst = {"along_params": 0.0, "along_grads": 0.0, "along_update": 0.0, "free_params": 0.0}
    note(f"{name}: {w.dims} batch={w.batch} shards={shards} steps={steps}")
    free_plain, free_dec = [], []
    with GpuNet(w.dims, acts, theta0) as net:
        # step along the reference
        for t in range(steps):
            sl = slice(t * w.batch, (t + 1) * w.batch)
            net.nf.nf_set_params(net.h, ref_t[t])
            net.train_batch(xd[sl], yd[sl], w.eta, shards)
            p, g = net.params(), net.grads()
            kstats = {}
            if kinked:
                sides, kstats = _sides(net, w, ref_t[t], X[sl], fails, f"step-along {t}")
                new, G = _kink_step(w, ref_t[t], X[sl], Y[sl], shards, sides)
            else:
                new, G = ref_t[t + 1], ref_g[t]
            rp, rg, ru = {}, {}, {}
            fails += [f"step-along {t}: {m}" for m in parity.check_params(
                p, new, w.dims, report=rp, floor=parity.SMALL_FLOOR)]
            fails += [f"step-along {t}: {m}" for m in parity.check_grads(g, G, w.dims, report=rg)]
            fails += [f"step-along {t}: {m}" for m in parity.check_update(p, ref_t[t], G, scale,
                                                                          w.dims, report=ru)]
            parity.emit(f"{name} along {t}", {"params": rp, "grads": rg, "update": ru,
                                              "kinks": kstats})
            worst["along_params"] = max(worst["along_params"], parity.worst(rp))
            worst["along_grads"] = max(worst["along_grads"], parity.worst(rg))
            worst["along_update"] = max(worst["along_update"], parity.worst(ru))
        # free-running trajectory
        net.nf.nf_set_params(net.h, theta0)
        th_o = theta0
        for t in range(steps):
            sl = slice(t * w.batch, (t + 1) * w.batch)
            net.train_batch(xd[sl], yd[sl], w.eta, shards)
            p, g = net.params(), net.grads()
            kstats = {}
            tol_p = max(parity.PARAM_TOL, CHAOS_MARGIN * ulp_spread[t])
            band = max(parity.KINK_BAND, CHAOS_MARGIN * ulp_spread[t])
            if kinked:
                sides, kstats = _sides(net, w, th_o, X[sl], fails, f"free {t}", band)
                th_new, G_o = _kink_step(w, th_o, X[sl], Y[sl], shards, sides, band)
            else:
                th_new, G_o = ref_t[t + 1], ref_g[t]
            rp, rg = {}, {}
            # without kinks the free-running trajectory is held to the same floor
            # as the step-along one; the relu schedules to the rms floor and the
            # envelope of the reference's own one-ulp spread
            fails += [f"free {t}: {m}" for m in parity.check_params(
                p, th_new, w.dims, tol=tol_p, report=rp,
                floor=1.0 if kinked else parity.SMALL_FLOOR)]
            gfails = parity.check_grads(g, G_o, w.dims, report=rg)
            if not kinked:
                fails += [f"free {t}: {m}" for m in gfails]
            rec = {"params": rp, "grads": rg, "kinks": kstats, "gate": tol_p,
                   "reference_ulp_spread": ulp_spread[t]}
            if kinked:
                plain = {}
                parity.check_params(p, ref_t[t + 1], w.dims, report=plain)
                rec["params_vs_plain_reference"] = plain
                free_plain.append(parity.worst(plain))
            parity.emit(f"{name} free {t}", rec)
            worst["free_params"] = max(worst["free_params"], parity.worst(rp))
            free_dec.append(parity.worst(rp))
            th_o = th_new
        if w.heldout:
            Xh, _ = W.make_data(w, heldout=True)
            note(f"{name}: inference on {Xh.shape[0]} held-out samples")
            net.nf.nf_set_params(net.h, ref_t[-1])
            out = net.forward(to_dev(Xh))
            ro = parity.tensor_report(out, mlp.output(ref_t[-1], w.dims, acts, Xh))
            parity.emit(f"{name} inference", ro)
            if not ro["floor_1e-3"] <= parity.OUT_TOL:
                fails.append(f"inference: relative error {ro['floor_1e-3']:.3e} (floor 1e-3 rms)")
    msg = (f"[parity] {name}: step-along worst params {worst['along_params']:.2e}, tendencies "
           f"{worst['along_grads']:.2e}, update {worst['along_update']:.2e}; free-running worst "
           f"params {worst['free_params']:.2e}")
    if kinked and steps >= 10:
        # the plain reference against itself with the other side taken for
        # the band units: how far the undetermined decisions alone move it
        alt_t, _ = _reference(w, X, Y, theta0, steps, shards, parity.KINK_BAND)
        spread = []
        for t in range(steps):
            rep = {}
            parity.check_params(alt_t[t + 1], ref_t[t + 1], w.dims, report=rep)
            spread.append(parity.worst(rep))
        parity.emit(f"{name} free-running after 10 steps",
                    {"gpu_vs_reference_with_gpu_decisions": free_dec[9], "gpu_vs_plain_reference":
                     free_plain[9], "plain_reference_spread": spread[9],
                     "reference_ulp_spread": ulp_spread[9],
                     "per_step_gated": free_dec, "per_step_vs_plain": free_plain,
                     "per_step_spread": spread, "per_step_ulp_spread": ulp_spread})
        gate10 = max(parity.PARAM_TOL, CHAOS_MARGIN * ulp_spread[9])
        gate_end = max(parity.PARAM_TOL, CHAOS_MARGIN * ulp_spread[-1])
        msg += (f"; after 10 steps: {free_dec[9]:.2e} (gated at {gate10:.1e}), "
                f"vs the plain reference {free_plain[9]:.2e}, the plain reference's spread "
                f"over the band's decisions {spread[9]:.2e}, over one ulp {ulp_spread[9]:.2e}; "
                f"at the end {free_dec[-1]:.2e} (gated at {gate_end:.1e})")
    print(msg, file=sys.stderr, flush=True)
    assert not fails, "\n".join(fails[:30])
    return w, X, Y, theta0


def test_c1_784_30_10_batch100():
    _run("c1")


def test_c2_784_30_10_epoch_and_inference():
    w, X, Y, theta = _run("c2")
    # the whole epoch in one call gives the same bits as step-by-step calls
    note("c2: nf_train_epoch")
    with GpuNet(w.dims, list(w.acts), theta) as a, GpuNet(w.dims, list(w.acts), theta) as b:
        xd, yd = to_dev(X), to_dev(Y)
        a.train_epoch(xd, yd, w.batch, w.eta, w.shards)
        for t in range(w.steps):
            b.train_batch(xd[t * w.batch:(t + 1) * w.batch], yd[t * w.batch:(t + 1) * w.batch],
                          w.eta, w.shards)
        assert np.array_equal(a.params(), b.params())


def test_c3_784_100_100_10_sixteen_shards():
    _run("c3")


@pytest.mark.timeout(900)
def test_c4_784_1024x3_10():
    _run("c4")


@pytest.mark.timeout(900)
def test_c5_4096x4_10():
    _run("c5")
