"""Error metrics of the GPU parity tests. No arithmetic of the method lives here.

Three views of the difference between what the HIP path stored and what the
fp64 oracle computed:

* whole: the relative Frobenius error of a whole tensor. It is the gate the
  targets are stated in (1e-5 after one step from the same state, 1e-3 along a
  trajectory), but it is diluted where most of a tensor is common to both
  sides: a factor is a multiple of the identity plus a small part that the
  gradients put there, and one step moves a parameter by well under 1% of
  its norm.
* factor: the error of a factor relative to its informative part
  A - (tr A / d) I, the part that differs from a multiple of the identity
  (Algorithm 2 starts every factor at eps^(-1/4) I).
* theta: the error of a parameter relative to the step the oracle applied,
  theta_t - theta_{t-1} (1 - lr wd) (the grafted momentum step of
  Algorithm 3, apart from the decoupled decay of Section 4).

The last two gates also allow a floor for the fp32 storage of the result,
which no computation in fp32 can go below: one rounding of each stored
element is up to 2^-24 of its magnitude. For a factor the floor is 2^-22 of
its norm (its own rounding, and the fp32 rounding of the scale s that
multiplies the whole factor, with a factor two of margin); for a parameter
2^-23 of its norm (its rounding, with the same margin).
"""
from __future__ import annotations

import numpy as np

# Gates after one step from the same state, and along a trajectory.
STEP = {"whole": 1e-5, "factor": 1e-3, "theta": 1e-4}
TRAJ = {"whole": 1e-3, "factor": 1e-2, "theta": 1e-2}
FACTOR_FLOOR = 2.0 ** -22
THETA_FLOOR = 2.0 ** -23
# A factor whose informative part is below this fraction of its norm carries
# nothing beyond rounding (a 1 x 1 factor, or one a zero gradient left alone):
# only the whole-tensor gate applies to it.
INFORMATIVE_MIN = 1e-6


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def rel(a, b) -> float:
    """||a - b||_F / ||b||_F (or ||a - b||_F when b = 0)."""
    a, b = _f64(a), _f64(b)
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (nb if nb > 0 else 1.0))


def informative(A) -> np.ndarray:
    """A - (tr A / d) I."""
    A = _f64(A)
    d = A.shape[0]
    return A - (np.trace(A) / d) * np.eye(d)


def factor_error(A_gpu, A_orc):
    """(error / ||informative part||, allowed floor / ||informative part||, ||informative|| / ||A||),
    or None when the informative part is negligible."""
    A_gpu, A_orc = _f64(A_gpu), _f64(A_orc)
    na = np.linalg.norm(A_orc)
    ni = np.linalg.norm(informative(A_orc))
    if na == 0 or ni <= INFORMATIVE_MIN * na:
        return None
    return (float(np.linalg.norm(A_gpu - A_orc) / ni), float(FACTOR_FLOOR * na / ni), float(ni / na))


def theta_error(th_gpu, th_orc, th_prev_orc, lr, weight_decay):
    """(error / ||applied step||, allowed floor / ||applied step||), or None for a zero step."""
    th_gpu, th_orc, th_prev = _f64(th_gpu), _f64(th_orc), _f64(th_prev_orc)
    step = np.linalg.norm(th_orc - th_prev * (1.0 - lr * weight_decay))
    if step == 0:
        return None
    return (float(np.linalg.norm(th_gpu - th_orc) / step), float(THETA_FLOOR * np.linalg.norm(th_orc) / step))


def check_layer(gpu: dict, orc: dict, th_gpu, th_orc, th_prev_orc, lr, weight_decay, gates: dict, what: str):
    """Gates one layer; returns its metrics.

    gpu, orc: {"L", "R", "mom", "mom_sgd"} -> arrays. Every tensor passes the
    whole-tensor gate; L and R the factor gate; theta the whole and the
    theta gate.
    """
    out = {"whole": {}, "factor": {}, "theta": None}
    for k in ("L", "R", "mom", "mom_sgd"):
        out["whole"][k] = rel(gpu[k], orc[k])
    out["whole"]["theta"] = rel(th_gpu, th_orc)
    bad = [k for k, v in out["whole"].items() if not v <= gates["whole"]]
    for k in ("L", "R"):
        fe = factor_error(gpu[k], orc[k])
        out["factor"][k] = fe
        if fe is not None and not fe[0] <= gates["factor"] + fe[1]:
            bad.append(f"{k} (informative part)")
    te = theta_error(th_gpu, th_orc, th_prev_orc, lr, weight_decay)
    out["theta"] = te
    if te is not None and not te[0] <= gates["theta"] + te[1]:
        bad.append("theta (relative to the applied step)")
    assert not bad, f"{what}: {bad} over the gates {gates}: {out}"
    return out


def worst(metrics: list) -> dict:
    """The largest value of each metric over a list of check_layer results."""
    w = {"whole": 0.0, "factor": 0.0, "theta": 0.0}
    for m in metrics:
        w["whole"] = max(w["whole"], max(m["whole"].values()))
        for fe in m["factor"].values():
            if fe is not None:
                w["factor"] = max(w["factor"], fe[0])
        if m["theta"] is not None:
            w["theta"] = max(w["theta"], m["theta"][0])
    return w
