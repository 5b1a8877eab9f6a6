"""torch.optim front end of the Jorge library, with the paper's single-shot tuning.

JorgeOptimizer hands the parameters of two or more dimensions of each
parameter group to one Jorge context (the C ABI of include/jorge.h): an N-d
weight is the out x (numel / out) matrix its storage already is (Section 3
collapses weights to 2-D). The order of the collapsed columns does not matter: permuting them
permutes R_hat the same way (Jorge commutes with orthogonal changes of basis
of either side, and the initial eps^(-1/4) I is invariant), so channels-last
weights are used in place. Parameters of fewer than two dimensions (biases,
normalisation scales) take heavy-ball SGD, which the paper does not address.

sgd_to_jorge() and step_decay_milestones() implement the single-shot tuning
of Section 4: the learning rate is SGD's, carried over by grafting
(Appendix A.2, Algorithm 3, done inside the library); the decoupled weight
decay is lambda_SGD / (1 - beta_SGD) (Eq. 10); the schedule is a step decay by
10x at one third and two thirds of the run.
"""
from __future__ import annotations

import ctypes

import torch

from .jorge import Jorge


def sgd_to_jorge(lr: float, momentum: float, weight_decay: float) -> dict:
    """Jorge hyperparameters bootstrapped from a tuned SGD baseline (Section 4).

    lr carries over unchanged (the grafted step takes SGD's magnitude), beta1 is
    SGD's momentum, and the decoupled weight decay is weight_decay / (1 - momentum).
    """
    if not 0.0 <= momentum < 1.0:
        raise ValueError("SGD momentum must be in [0, 1)")
    return dict(lr=float(lr), beta1=float(momentum), weight_decay=float(weight_decay) / (1.0 - momentum))


def step_decay_milestones(total_steps: int) -> list[int]:
    """Steps at which the learning rate drops 10x: one third and two thirds of the run (Section 4)."""
    if total_steps < 3:
        raise ValueError("total_steps must be at least 3")
    return [total_steps // 3, (2 * total_steps) // 3]


def matrix_view(t: torch.Tensor) -> tuple[int, int]:
    """(rows, cols) of the matrix a parameter's storage holds: rows = size(0).

    The tensor must be dense with dimension 0 outermost (standard or
    channels-last layout); the other dimensions, in memory order, form the
    columns.
    """
    if t.dim() < 2:
        raise ValueError("matrix_view needs a tensor of two or more dimensions")
    rows = t.shape[0]
    cols = t.numel() // rows
    dense = t.is_contiguous() or t.is_contiguous(memory_format=torch.channels_last)
    if not dense or t.stride(0) != cols:
        raise ValueError(f"parameter of shape {tuple(t.shape)} and strides {t.stride()} is not a dense "
                         f"row-major matrix of {rows} rows")
    return rows, cols


def split_params(params) -> tuple[list, list]:
    """(matrices, vectors): parameters for Jorge (dim >= 2) and for SGD (dim < 2)."""
    mats, vecs = [], []
    for p in params:
        (mats if p.dim() >= 2 else vecs).append(p)
    return mats, vecs


class JorgeOptimizer(torch.optim.Optimizer):
    """torch.optim-style Jorge: one grouped library step per parameter group.

    Hyperparameters (per group, as in torch.optim): lr (grafted step size),
    beta1 (momentum of both m and m_SGD), beta2 (the floor of the dynamic beta
    by default), weight_decay (decoupled, lr-scaled, on matrices),
    vector_weight_decay (coupled L2 of the SGD update of vector parameters).
    Each group's matrix parameters form one Jorge context, stepped with that
    group's values (one group keeps every layer in the same grouped launches,
    which is the fastest). Context options (eps, precond_interval, beta_mode,
    graft, symmetrize, factor_form, ...) apply to every group's context. lr
    and the other values are read from the groups on every step, so torch
    learning-rate schedulers work.
    """

    def __init__(self, params, lr: float, beta1: float = 0.9, beta2: float = 0.9, weight_decay: float = 0.0,
                 vector_weight_decay: float = 0.0, **context_options):
        self._context_options = dict(context_options)
        self._groups = []   # per parameter group: matrices, vectors, context, pointer array
        self._zero = {}
        defaults = dict(lr=lr, beta1=beta1, beta2=beta2, weight_decay=weight_decay,
                        vector_weight_decay=vector_weight_decay)
        super().__init__(params, defaults)

    def add_param_group(self, param_group):
        super().add_param_group(param_group)
        mats, vecs = split_params(self.param_groups[-1]["params"])
        for p in mats:
            if not (p.is_cuda and p.dtype == torch.float32):
                raise ValueError("matrix parameters must be fp32 CUDA tensors")
        ctx = Jorge([matrix_view(p) for p in mats], **self._context_options) if mats else None
        self._groups.append({"mats": mats, "vecs": vecs, "ctx": ctx,
                             "ptrs": Jorge.pointer_array(mats) if mats else None})

    @property
    def ctx(self):
        """The Jorge context of the first parameter group that has matrix parameters (or None)."""
        return next((g["ctx"] for g in self._groups if g["ctx"] is not None), None)

    @property
    def mats(self):
        """Every matrix parameter, group by group."""
        return [p for g in self._groups for p in g["mats"]]

    def _grad_ptrs(self, mats):
        """Device pointers of the matrix gradients, each in its parameter's layout."""
        ptrs = []
        for p in mats:
            g = p.grad
            if g is None:  # no gradient this step: a zero gradient of the same layout
                g = self._zero.get(id(p))
                if g is None:
                    g = self._zero[id(p)] = torch.zeros_like(p)
            elif g.dtype != torch.float32 or g.stride() != p.stride():
                g = torch.empty_like(p).copy_(g)   # empty_like keeps p's memory format
                self._keep.append(g)
            ptrs.append(g.data_ptr())
        return (ctypes.c_void_p * len(ptrs))(*ptrs)

    @torch.no_grad()
    def step(self, closure=None):
        loss = None
        if closure is not None:
            with torch.enable_grad():
                loss = closure()
        self._keep = []
        for group, g in zip(self.param_groups, self._groups):
            lr, b1, b2, wd = group["lr"], group["beta1"], group["beta2"], group["weight_decay"]
            if g["ctx"] is not None:
                g["ctx"].set_stream(torch.cuda.current_stream().cuda_stream)
                g["ctx"].step_ptrs(g["ptrs"], self._grad_ptrs(g["mats"]), lr, b2, b1, wd)
            vec = [p for p in g["vecs"] if p.grad is not None]
            if vec:
                grads = [p.grad for p in vec]
                vwd = group["vector_weight_decay"]
                if vwd:
                    grads = torch._foreach_add(grads, [p for p in vec], alpha=vwd)
                bufs = []
                for p, gr in zip(vec, grads):
                    st = self.state[p]
                    if "momentum_buffer" not in st:
                        st["momentum_buffer"] = torch.clone(gr).detach()
                    else:
                        st["momentum_buffer"].mul_(b1).add_(gr)
                    bufs.append(st["momentum_buffer"])
                torch._foreach_add_(vec, bufs, alpha=-lr)
        return loss

    def state_dict(self):
        """The torch state plus, per parameter group, its Jorge context's state tensors and step counter
        (host copies)."""
        sd = super().state_dict()
        sd["jorge"] = [None if g["ctx"] is None else
                       {"t": g["ctx"].t,
                        "tensors": [{k: g["ctx"].get_state(l, k).cpu() for k in ("L", "R", "mom", "mom_sgd")}
                                    for l in range(len(g["mats"]))]}
                       for g in self._groups]
        return sd

    def load_state_dict(self, state_dict):
        sd = dict(state_dict)
        jorge = sd.pop("jorge", None)
        super().load_state_dict(sd)
        if isinstance(jorge, dict):   # a single group's record
            jorge = [jorge]
        for g, rec in zip(self._groups, jorge or []):
            if rec is None or g["ctx"] is None:
                continue
            for l, tensors in enumerate(rec["tensors"]):
                for k, v in tensors.items():
                    g["ctx"].set_state(l, k, v)
            g["ctx"].t = rec["t"]
