"""Plain fp64 CPU oracle for the Jorge optimizer step.

TEST INFRASTRUCTURE ONLY. Nothing in the GPU library imports, links or runs
this module; only the tests, the smoke check and the CPU-baseline leg of the
benchmark do. It shares no code with the HIP path.

What it follows (Singh, Sating, Bhatele, "Jorge: Approximate Preconditioning
for GPU-efficient Second-order Optimization", arXiv 2310.12298):

* Algorithm 2 (Jorge, Section 3): factors initialised to eps^(-1/4) I;
  X_L = L_hat^4 G G^T and X_R = R_hat^4 G^T G; each factor updated as
  beta^(-1/4) A_hat (I - (1-beta)/(4 beta) X + 5 (1-beta)^2/(32 beta^2) X^2);
  gradient preconditioned as L_hat G R_hat; momentum on the preconditioned
  gradient; weight update.
* Eq. 5-7 (Section 3): the binomial series of (I + A)^(-p) with p = 1/4,
  truncated after the quadratic term. The coefficients are computed here
  from the general term of Eq. 5 rather than typed in. Section 3 drops the
  cubic and higher terms; series_order=3 keeps the cubic one (the ablation of
  that choice).
* Appendix A.1, Eq. 8-9: the dynamic beta_2 = ||X||_F / (||X||_F + 1), which
  turns the update into ((nu+1)/nu)^(1/4) A_hat (I - X/(4 nu) + 5 X^2/(32 nu^2)).
* Appendix A.2, Algorithm 3: SGD grafting (step magnitude from the heavy-ball
  SGD momentum, direction from Jorge's momentum).
* Section 4, "Weight Decay Penalty": decoupled (AdamW-style) weight decay.

Readings taken where the paper is silent or ambiguous (each is listed, with its
justification, in the design notes of the repository):

* beta mode: FIXED uses beta_2 as given (Algorithm 2 literally); DYNAMIC uses
  Eq. 8 with equality (Appendix A.1), falling back to FIXED when ||X|| = 0;
  CLAMPED (the default) uses beta_eff = max(beta_2, nu/(nu+1)), i.e. the
  dynamic value exactly when the series would otherwise leave its domain.
  In every mode c = (1-beta)/beta and s = beta^(-1/4) are formed without the
  1-beta cancellation: c = 1/nu and s = (1+1/nu)^(1/4) on the dynamic branch
  (the form of Eq. 9).
* nu is the Frobenius norm over all entries of X = A_hat^4 M (Appendix A.1
  names the Frobenius norm; X is not symmetric).
* symmetrize: the literal product A_hat P(X) is symmetric only when A_hat and
  G G^T commute (the substitution of Eq. 3-4 assumes they do); by default the
  updated factor is replaced by (Z + Z^T)/2. symmetrize=False keeps Z.
* the factors that precondition the gradient are the ones after this step's
  update (Algorithm 2 preconditions with L_hat_t, R_hat_t).
* preconditioner interval k: the factors are updated on steps t with
  (t-1) mod k == 0, so the first step always updates.
* Algorithm 3's G-hat is Algorithm 2's G-tilde; its "theta_t = theta_t - ..."
  is read as theta_t = theta_{t-1} - ....
* grafting is per layer with Frobenius norms of the whole m x n tensors; if
  ||m||_F = 0 the grafted step is zero.
* decoupled weight decay: theta <- theta (1 - lr wd) - g m, applied to
  theta_{t-1} and not grafted.
* m_SGD accumulates the raw gradient (no dampening, no weight-decay term).
* G-tilde is evaluated as (L_hat G) R_hat.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

BETA_FIXED = 0
BETA_DYNAMIC = 1
BETA_CLAMPED = 2


def binomial_series_coefficient(p: float, r: int) -> float:
    """Coefficient of A^r in (I + A)^(-p): (-1)^r p (p+1) ... (p+r-1) / r!  (Eq. 5)."""
    coef = 1.0
    for i in range(r):
        coef *= (p + i) / (i + 1)
    return (-1.0) ** r * coef


# Eq. 6 with p = 1/4: the linear and the quadratic coefficient (-1/4 and 5/32),
# and the cubic one of Eq. 5 (-15/128) that Section 3 drops.
SERIES_C1 = binomial_series_coefficient(0.25, 1)
SERIES_C2 = binomial_series_coefficient(0.25, 2)
SERIES_C3 = binomial_series_coefficient(0.25, 3)


def init_factor(d: int, eps: float) -> np.ndarray:
    """Algorithm 2 initialisation: A_hat_0 = eps^(-1/4) I_d."""
    return np.eye(d, dtype=np.float64) * eps ** -0.25


def gram_factors(G: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """The two Kronecker statistics of Algorithm 2: G G^T (m x m) and G^T G (n x n)."""
    G = np.asarray(G, dtype=np.float64)
    return G @ G.T, G.T @ G


def beta_select(nu: float, beta2: float, mode: int) -> tuple[float, float, float]:
    """Return (c, s, beta_eff) with c = (1-beta)/beta and s = beta^(-1/4).

    FIXED: beta = beta2 (Algorithm 2). DYNAMIC: beta = nu/(nu+1) (Eq. 8 with
    equality), which gives c = 1/nu and s = ((nu+1)/nu)^(1/4) (Eq. 9); at
    nu = 0 it falls back to FIXED. CLAMPED: beta = max(beta2, nu/(nu+1)).
    """
    beta2 = float(beta2)
    c_fixed = (1.0 - beta2) / beta2
    s_fixed = beta2 ** -0.25
    if mode == BETA_FIXED:
        return c_fixed, s_fixed, beta2
    if mode == BETA_DYNAMIC:
        use_dynamic = nu > 0.0
    elif mode == BETA_CLAMPED:
        # nu/(nu+1) > beta2  <=>  nu > beta2/(1-beta2)
        use_dynamic = nu > beta2 / (1.0 - beta2)
    else:
        raise ValueError(f"unknown beta mode {mode}")
    if not use_dynamic:
        return c_fixed, s_fixed, beta2
    return 1.0 / nu, (1.0 + 1.0 / nu) ** 0.25, nu / (nu + 1.0)


def update_factor(A_hat: np.ndarray, M: np.ndarray, beta2: float,
                  mode: int = BETA_CLAMPED, symmetrize: bool = True, series_order: int = 2):
    """One preconditioner update of Algorithm 2 (the same form for L_hat and R_hat).

    A_hat is the previous factor (L_hat or R_hat), M the matching statistic
    (G G^T or G^T G). series_order is the last power of X kept from the
    series of Eq. 5: 2 as in Eq. 6-7, or 3. Returns the new factor and a dict
    of intermediates.
    """
    if series_order not in (2, 3):
        raise ValueError("series_order must be 2 or 3")
    A_hat = np.asarray(A_hat, dtype=np.float64)
    M = np.asarray(M, dtype=np.float64)
    d = A_hat.shape[0]
    A2 = A_hat @ A_hat
    A4 = A2 @ A2
    X = A4 @ M                                   # X = A_hat^4 G G^T (Algorithm 2)
    nu = float(np.sqrt(np.sum(X * X)))           # Frobenius norm (Appendix A.1)
    c, s, beta_eff = beta_select(nu, beta2, mode)
    # Truncated series of (I + c X)^(-1/4) (Eq. 6-7, Algorithm 2's factor update)
    X2 = X @ X
    P = np.eye(d) + SERIES_C1 * c * X + SERIES_C2 * (c * c) * X2
    if series_order == 3:                        # the next term of Eq. 5
        P = P + SERIES_C3 * (c * c * c) * (X2 @ X)
    Z = s * (A_hat @ P)
    A_new = 0.5 * (Z + Z.T) if symmetrize else Z
    return A_new, {"X": X, "nu": nu, "c": c, "s": s, "beta_eff": beta_eff,
                   "P": P, "Z": Z}


def precondition(L_hat: np.ndarray, G: np.ndarray, R_hat: np.ndarray) -> np.ndarray:
    """G_tilde = L_hat G R_hat (Algorithm 2's preconditioned gradient), evaluated as (L_hat G) R_hat."""
    return (L_hat @ np.asarray(G, dtype=np.float64)) @ R_hat


def update_weights(theta, m, m_sgd, G_tilde, G, lr, beta1, weight_decay, graft=True):
    """Momentum, SGD grafting and decoupled weight decay.

    m = beta1 m + (1-beta1) G_tilde (the momentum of Algorithms 2 and 3);
    m_SGD = beta1 m_SGD + G (Algorithm 3's SGD momentum);
    theta = theta (1 - lr wd) - g m with g = lr ||m_SGD|| / ||m|| when grafting
    (Algorithm 3's grafted step, Section 4's decoupled weight decay), g = lr otherwise.
    """
    G = np.asarray(G, dtype=np.float64)
    m = beta1 * m + (1.0 - beta1) * G_tilde
    m_sgd = beta1 * m_sgd + G
    norm_m = float(np.sqrt(np.sum(m * m)))
    norm_sgd = float(np.sqrt(np.sum(m_sgd * m_sgd)))
    if graft:
        g = lr * norm_sgd / norm_m if norm_m > 0.0 else 0.0
    else:
        g = lr
    theta = np.asarray(theta, dtype=np.float64) * (1.0 - lr * weight_decay) - g * m
    return theta, m, m_sgd, {"norm_m": norm_m, "norm_sgd": norm_sgd, "g": g}


@dataclass
class LayerState:
    L: np.ndarray
    R: np.ndarray
    m: np.ndarray
    m_sgd: np.ndarray


@dataclass
class JorgeOracle:
    """Per-layer Jorge state for a list of m x n layers, stepped one layer at a time."""
    shapes: list
    eps: float = 1e-6
    precond_interval: int = 1
    beta_mode: int = BETA_CLAMPED
    graft: bool = True
    symmetrize: bool = True
    series_order: int = 2
    t: int = 0                                   # steps taken so far
    layers: list = field(default_factory=list)
    last_diag: list = field(default_factory=list)

    def __post_init__(self):
        if not self.layers:
            self.layers = [LayerState(init_factor(m, self.eps), init_factor(n, self.eps),
                                      np.zeros((m, n)), np.zeros((m, n)))
                           for (m, n) in self.shapes]

    def step(self, params, grads, lr, beta2, beta1, weight_decay):
        """One Jorge step over all layers. params/grads: lists of m x n arrays.

        Returns the list of updated parameters (fp64).
        """
        self.t += 1
        update = (self.t - 1) % self.precond_interval == 0
        out, self.last_diag = [], []
        for st, theta, G in zip(self.layers, params, grads):
            G = np.asarray(G, dtype=np.float64)
            diag = {}
            if update:
                ML, MR = gram_factors(G)
                st.L, dL = update_factor(st.L, ML, beta2, self.beta_mode, self.symmetrize,
                                         self.series_order)
                st.R, dR = update_factor(st.R, MR, beta2, self.beta_mode, self.symmetrize,
                                         self.series_order)
                diag.update(nu_L=dL["nu"], nu_R=dR["nu"], beta_L=dL["beta_eff"],
                            beta_R=dR["beta_eff"])
            Gt = precondition(st.L, G, st.R)
            theta, st.m, st.m_sgd, dw = update_weights(theta, st.m, st.m_sgd, Gt, G, lr,
                                                       beta1, weight_decay, self.graft)
            diag.update(dw)
            self.last_diag.append(diag)
            out.append(theta)
        return out
