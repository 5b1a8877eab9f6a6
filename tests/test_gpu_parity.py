"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Gates (tests/parity_metrics.py): after one step from the same state, relative
Frobenius error <= 1e-5 on every tensor, <= 1e-3 on the factors' informative
part A - (tr A / d) I, <= 1e-4 on the parameters relative to the step the
oracle applied; along a trajectory 1e-3, 1e-2 and 1e-2. Exact (bitwise)
properties: factor symmetry, pure beta-scaling at G = 0, determinism,
grouping invariance, the update interval and checkpoint/resume.
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import JorgeOracle  # noqa: E402
from paper_2310_12298_amd.jorge import Jorge, JorgeError  # noqa: E402
from paper_2310_12298_amd.workloads import gradient, initial_params  # noqa: E402
from parity_metrics import STEP, TRAJ, check_layer, rel, worst  # noqa: E402

pytestmark = pytest.mark.gpu

# Evaluation orders of the factor update: the paper's explicit powers, the
# factored order through the statistic's factor H, the squared order (A^2
# formed, the chain through H in steps of A^2; symmetric factors only), all
# through the grouped levels, and the default per-factor choice, where a
# context whose factors all have padded size <= 64 runs them in the
# one-workgroup LDS chain.
FORMS = ("explicit", "factored", "squared", "auto")
FORM_KW = {"explicit": dict(factor_form="explicit", lds_chain_max=0),
           "factored": dict(factor_form="factored", lds_chain_max=0),
           "squared": dict(factor_form="squared", lds_chain_max=0),
           "auto": dict(factor_form="auto")}
HP = dict(lr=0.1, beta2=0.9, beta1=0.9, weight_decay=5e-5)
KINDS = ("L", "R", "mom", "mom_sgd")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def oracle_state(orc, l):
    st = orc.layers[l]
    return {"L": st.L, "R": st.R, "mom": st.m, "mom_sgd": st.m_sgd}


def gpu_state(opt, l):
    return {k: opt.get_state(l, k).cpu().numpy() for k in KINDS}


def compare(opt, orc, params_gpu, params_orc, params_prev, gates, what, hp=HP):
    """Gates every layer (tests/parity_metrics.py); params_prev: the oracle's parameters
    before the step just taken. Returns the worst value of each metric."""
    ms = [check_layer(gpu_state(opt, l), oracle_state(orc, l), params_gpu[l].cpu().numpy(), params_orc[l],
                      params_prev[l], hp["lr"], hp["weight_decay"], gates, f"{what} layer {l}")
          for l in range(len(params_orc))]
    return worst(ms)


def run_pair(shapes, steps, sigma, seed=0, check_every=None, gpu_kw=None, orc_kw=None, hp=HP):
    gpu_kw = gpu_kw or {}
    orc_kw = orc_kw or {}
    opt = Jorge(shapes, **gpu_kw)
    orc = JorgeOracle(shapes, **orc_kw)
    p0 = [initial_params(seed, l, s) for l, s in enumerate(shapes)]
    pg = [to_dev(p) for p in p0]
    po = [p.astype(np.float64) for p in p0]
    w = {"whole": 0.0, "factor": 0.0, "theta": 0.0}
    for t in range(1, steps + 1):
        G = [gradient(seed, l, t, s, sigma) for l, s in enumerate(shapes)]
        opt.step(pg, [to_dev(g) for g in G], hp["lr"], hp["beta2"], hp["beta1"], hp["weight_decay"])
        prev = po
        po = orc.step(po, G, hp["lr"], hp["beta2"], hp["beta1"], hp["weight_decay"])
        if t == steps or (check_every and t % check_every == 0):
            m = compare(opt, orc, pg, po, prev, STEP if t == 1 else TRAJ, f"step {t}", hp)
            w = {k: max(w[k], m[k]) for k in w}
    return opt, orc, pg, po, w


@pytest.mark.parametrize("form", FORMS)
@pytest.mark.parametrize("shapes", [
    [(64, 576)],                       # 3x3 conv 64 -> 64
    [(64, 147)],                       # ragged stem
    [(33, 65)],
    [(1, 1)], [(1, 40)], [(40, 1)],
    [(200, 300)],                      # several tiles, ragged tail
    [(130, 260)],
    [(64, 576), (100, 70), (256, 64), (5, 3)],
])
def test_first_step_parity(shapes, form):
    say("first step", shapes, form)
    say("  worst", run_pair(shapes, 1, 1e-2, gpu_kw=FORM_KW[form])[4])


@pytest.mark.parametrize("form", FORMS)
def test_trajectory_64x576_100_steps(form):
    say("trajectory 64x576 x 100", form)
    say("  worst", run_pair([(64, 576)], 100, 1e-2, check_every=10, gpu_kw=FORM_KW[form])[4])


@pytest.mark.parametrize("form", FORMS)
def test_trajectory_multitile_30_steps(form):
    say("trajectory (256x1152, 300x200) x 30", form)
    run_pair([(256, 1152), (300, 200)], 30, 1e-3, check_every=15, gpu_kw=FORM_KW[form])


@pytest.mark.parametrize("form", FORMS)
@pytest.mark.parametrize("t_inject", [2, 5, 20, 50])
def test_per_step_parity_from_injected_state(t_inject, form):
    """Oracle state after t-1 steps (rounded to fp32) is injected; one step on both."""
    shapes = [(64, 576)]
    say("inject at", t_inject)
    orc = JorgeOracle(shapes)
    po = [initial_params(0, 0, shapes[0]).astype(np.float64)]
    for t in range(1, t_inject):
        po = orc.step(po, [gradient(0, 0, t, shapes[0], 1e-2)], **HP)
    st = orc.layers[0]
    for k in ("L", "R", "m", "m_sgd"):
        setattr(st, k, getattr(st, k).astype(np.float32).astype(np.float64))
    po = [po[0].astype(np.float32).astype(np.float64)]
    opt = Jorge(shapes, **FORM_KW[form])
    for k, v in oracle_state(orc, 0).items():
        opt.set_state(0, k, to_dev(v))
    opt.t = t_inject - 1
    pg = [to_dev(po[0])]
    G = [gradient(0, 0, t_inject, shapes[0], 1e-2)]
    opt.step(pg, [to_dev(G[0])], **HP)
    prev = po
    po = orc.step(po, G, **HP)
    say("  worst", compare(opt, orc, pg, po, prev, STEP, f"injected step {t_inject}"))


@pytest.mark.parametrize("form", FORMS)
@pytest.mark.parametrize("mode,sigma,beta2", [("fixed", 1e-4, 0.9), ("dynamic", 1e-2, 0.9),
                                              ("clamped", 3e-4, 0.9)])
def test_beta_modes(mode, sigma, beta2, form):
    say("mode", mode, form)
    code = {"fixed": 0, "dynamic": 1, "clamped": 2}[mode]
    run_pair([(48, 96), (70, 40)], 6, sigma, check_every=3, gpu_kw=dict(FORM_KW[form], beta_mode=mode),
             orc_kw=dict(beta_mode=code), hp=dict(HP, beta2=beta2))


@pytest.mark.parametrize("form", FORMS)
def test_literal_mode_without_symmetrization(form):
    say("literal mode", form)
    if form == "squared":  # needs symmetric factors: rejected before any GPU work
        with pytest.raises(JorgeError):
            Jorge([(48, 96)], symmetrize=False, factor_form="squared")
        return
    run_pair([(48, 96), (160, 40), (300, 130)], 6, 1e-2, check_every=3,
             gpu_kw=dict(FORM_KW[form], symmetrize=False), orc_kw=dict(symmetrize=False))


def test_without_grafting():
    say("no graft")
    run_pair([(64, 200)], 5, 1e-2, gpu_kw=dict(graft=False), orc_kw=dict(graft=False),
             hp=dict(HP, lr=1e-4))


def test_update_interval_parity_and_frozen_factors():
    shapes = [(64, 200), (96, 32)]
    say("interval k=3")
    opt = Jorge(shapes, precond_interval=3)
    orc = JorgeOracle(shapes, precond_interval=3)
    pg = [to_dev(initial_params(0, l, s)) for l, s in enumerate(shapes)]
    po = [initial_params(0, l, s).astype(np.float64) for l, s in enumerate(shapes)]
    for t in range(1, 8):
        before = [opt.get_state(l, "L").clone() for l in range(2)]
        G = [gradient(0, l, t, s, 1e-2) for l, s in enumerate(shapes)]
        opt.step(pg, [to_dev(g) for g in G], **HP)
        prev = po
        po = orc.step(po, G, **HP)
        for l in range(2):
            same = torch.equal(before[l], opt.get_state(l, "L"))
            assert same == ((t - 1) % 3 != 0), (t, l)
    compare(opt, orc, pg, po, prev, TRAJ, "k=3")


@pytest.mark.parametrize("form", FORMS)
def test_factors_bitwise_symmetric_and_deterministic(form):
    shapes = [(200, 300), (64, 147), (130, 600)]
    say("symmetry + determinism", form)
    a = run_pair(shapes, 4, 1e-2, gpu_kw=FORM_KW[form])
    b = run_pair(shapes, 4, 1e-2, gpu_kw=FORM_KW[form])
    for l in range(len(shapes)):
        for k in ("L", "R"):
            A = a[0].get_state(l, k)
            assert torch.equal(A, A.T), (l, k)
        for k in KINDS:
            assert torch.equal(a[0].get_state(l, k), b[0].get_state(l, k)), (l, k)
        assert torch.equal(a[2][l], b[2][l])


def test_grouping_invariance():
    """Each tile is computed the same way whatever else shares its launch.

    Split-K is off: its split plan depends on every layer of the context.
    """
    shapes = [(64, 576), (256, 64), (130, 90), (256, 2304)]
    say("grouping invariance")
    grouped = Jorge(shapes, split_k=False)
    singles = [Jorge([s], split_k=False) for s in shapes]
    pg = [to_dev(initial_params(0, l, s)) for l, s in enumerate(shapes)]
    ps = [p.clone() for p in pg]
    for t in range(1, 4):
        G = [to_dev(gradient(0, l, t, s, 1e-2)) for l, s in enumerate(shapes)]
        grouped.step(pg, G, **HP)
        for l in range(len(shapes)):
            singles[l].step([ps[l]], [G[l]], **HP)
    for l in range(len(shapes)):
        for k in KINDS:
            assert torch.equal(grouped.get_state(l, k), singles[l].get_state(0, k)), (l, k)
        assert torch.equal(pg[l], ps[l])


@pytest.mark.parametrize("form", FORMS)
def test_zero_gradient_is_exact_beta_scaling(form):
    shapes = [(64, 96)]
    say("G = 0", form)
    opt, _, pg, _, _ = run_pair(shapes, 3, 1e-2, gpu_kw=FORM_KW[form])
    before = {k: opt.get_state(0, k) for k in KINDS}
    theta = pg[0].clone()
    opt.step(pg, [torch.zeros(shapes[0], device="cuda")], 0.1, 0.8, 0.9, 1e-3)
    sf = torch.tensor(0.8 ** -0.25, dtype=torch.float32, device="cuda")
    b1 = torch.tensor(0.9, dtype=torch.float32, device="cuda")
    for k in ("L", "R"):
        assert torch.equal(opt.get_state(0, k), sf * before[k]), k
    assert torch.equal(opt.get_state(0, "mom"), b1 * before["mom"])
    assert torch.equal(opt.get_state(0, "mom_sgd"), b1 * before["mom_sgd"])
    d = opt.read_diag(0)
    assert d["nu_L"] == 0.0 and d["nu_R"] == 0.0 and d["beta_L"] == 0.8
    g = 0.1 * d["norm_sgd"] / d["norm_m"]
    expect = theta.double() * (1 - 0.1 * 1e-3) - g * opt.get_state(0, "mom").double()
    assert rel(pg[0].cpu().numpy(), expect.cpu().numpy()) < 1e-6


def test_checkpoint_resume_bitwise():
    shapes = [(64, 147), (128, 256)]
    say("resume")
    full = Jorge(shapes)
    pf = [to_dev(initial_params(0, l, s)) for l, s in enumerate(shapes)]
    grads = [[to_dev(gradient(0, l, t, s, 1e-2)) for l, s in enumerate(shapes)] for t in range(1, 9)]
    for t in range(4):
        full.step(pf, grads[t], **HP)
    saved = {(l, k): full.get_state(l, k).clone() for l in range(2) for k in KINDS}
    pr = [p.clone() for p in pf]
    resumed = Jorge(shapes)
    for (l, k), v in saved.items():
        resumed.set_state(l, k, v)
    resumed.t = full.t
    for t in range(4, 8):
        full.step(pf, grads[t], **HP)
        resumed.step(pr, grads[t], **HP)
    for l in range(2):
        assert torch.equal(pf[l], pr[l])
        for k in KINDS:
            assert torch.equal(full.get_state(l, k), resumed.get_state(l, k))


def test_many_small_layers():
    rng = np.random.default_rng(5)
    shapes = [tuple(int(x) for x in rng.choice([32, 64, 128, 256], 2)) for _ in range(24)]
    say("many small", len(shapes))
    run_pair(shapes, 3, 1e-2)


def test_full_size_512x4608_first_step():
    say("512x4608 first step")
    opt, _, _, _, _ = run_pair([(512, 4608)], 1, 1e-3)
    assert (opt.factor_form(0, 0), opt.factor_form(0, 1)) == ("explicit", "factored")


def test_auto_form_choice():
    """The cheapest order by tile work: factored when the statistic's rank k is well below d,
    squared for k about d/2, explicit from about 2d/3 up."""
    opt = Jorge([(64, 576), (512, 512), (256, 2304), (2048, 512), (64, 64), (1024, 512), (2048, 1024)])
    forms = [(opt.factor_form(l, 0), opt.factor_form(l, 1)) for l in range(7)]
    assert forms == [("explicit", "factored"), ("explicit", "explicit"), ("explicit", "factored"),
                     ("factored", "explicit"), ("explicit", "explicit"), ("squared", "explicit"),
                     ("squared", "explicit")], forms
    # The literal mode has no squared order.
    lit = Jorge([(1024, 512)], symmetrize=False)
    assert lit.factor_form(0, 0) == "factored"


def test_diagnostics_match_oracle():
    shapes = [(64, 576)]
    opt, orc, _, _, _ = run_pair(shapes, 2, 1e-2)
    d = opt.read_diag(0)
    od = orc.last_diag[0]
    assert d["nu_L"] == pytest.approx(od["nu_L"], rel=1e-5)
    assert d["nu_R"] == pytest.approx(od["nu_R"], rel=1e-5)
    assert d["beta_L"] == pytest.approx(od["beta_L"], rel=1e-9)
    assert d["norm_m"] == pytest.approx(od["norm_m"], rel=1e-5)
    assert d["norm_sgd"] == pytest.approx(od["norm_sgd"], rel=1e-6)
    assert d["g"] == pytest.approx(od["g"], rel=1e-5)


def test_invalid_step_arguments():
    opt = Jorge([(8, 8)])
    p = [torch.zeros((8, 8), device="cuda")]
    g = [torch.zeros((8, 8), device="cuda")]
    for kw in (dict(lr=-1.0), dict(lr=float("nan")), dict(lr=0.1, beta2=1.0), dict(lr=0.1, beta2=0.0),
               dict(lr=0.1, beta1=1.0), dict(lr=0.1, weight_decay=-1.0)):
        with pytest.raises(JorgeError):
            opt.step(p, g, **kw)
    assert opt.t == 0
    with pytest.raises(ValueError):
        opt.step([torch.zeros((8, 9), device="cuda")], g, 0.1)
    with pytest.raises(ValueError):
        opt.step(p, [torch.zeros((8, 8), device="cuda", dtype=torch.float64)], 0.1)


def test_stage_timing_reports_every_update_stage():
    opt = Jorge([(256, 1024)])
    p = [torch.zeros((256, 1024), device="cuda")]
    g = [to_dev(gradient(0, 0, 1, (256, 1024), 1e-2))]
    opt.set_timing(True)
    opt.step(p, g, 0.1)
    tm = opt.read_timing()
    # L_hat (256) is explicit and R_hat (1024, rank 256) factored, so every update stage runs once.
    assert (opt.factor_form(0, 0), opt.factor_form(0, 1)) == ("explicit", "factored")
    for name in ("stage_in", "gram", "pow4", "xform", "chain4", "chain5", "factor_finalize", "poly",
                 "update", "symmetrize", "uprecond_L", "uprecond_R", "layer_finalize", "weight"):
        assert tm[name][1] == 1 and tm[name][0] > 0, name
    assert tm["precond_L"][1] == 0      # the non-update steps' preconditioning
    fl = opt.stage_flops()
    m, n = 256, 1024
    assert fl["precond_L"] == 2 * m * m * n and fl["precond_R"] == 2 * m * n * n
    assert fl["stage_in"] == 0 and fl["weight"] == 0
    # The literal mode launches the powers of non-symmetric factors apart (MN-major B).
    lit = Jorge([(256, 512)], symmetrize=False)
    lit.set_timing(True)
    lit.step([torch.zeros((256, 512), device="cuda")], [to_dev(gradient(0, 0, 1, (256, 512), 1e-2))], 0.1)
    assert lit.read_timing()["gram"][1] == 2 and lit.read_timing()["pow4"][1] == 2
    opt.reset_timing()
    assert all(v == (0.0, 0) for v in opt.read_timing().values())


@pytest.mark.parametrize("form", ["explicit", "factored", "auto"])
def test_split_k_parity_and_determinism(form):
    """Levels with few, long tiles split K; the fixup sums the parts in a fixed order."""
    shapes = [(128, 2048), (64, 4096)]
    say("split-K", form)
    probe = Jorge(shapes, **FORM_KW[form])
    probe.set_timing(True)
    probe.step([torch.zeros(s, device="cuda") for s in shapes],
               [to_dev(gradient(0, l, 1, s, 1e-2)) for l, s in enumerate(shapes)], **HP)
    assert probe.read_timing()["split_fixup"][1] >= 1          # the plan does split
    a = run_pair(shapes, 3, 1e-2, gpu_kw=FORM_KW[form])                 # vs the oracle
    b = run_pair(shapes, 3, 1e-2, gpu_kw=FORM_KW[form])
    c = run_pair(shapes, 3, 1e-2, gpu_kw=dict(FORM_KW[form], split_k=False))
    for l in range(len(shapes)):
        assert torch.equal(a[2][l], b[2][l])
        for k in KINDS:
            x, y, z = (r[0].get_state(l, k) for r in (a, b, c))
            assert torch.equal(x, y), (l, k)                     # deterministic
            assert rel(x.cpu().numpy(), z.cpu().numpy()) < 1e-5, (l, k)   # split vs unsplit rounding


SMALL_SHAPES = [(64, 64), (32, 48), (5, 3), (40, 1), (33, 60), (64, 32), (1, 64), (50, 17)]
# Padded sizes 96 and 128 (and smaller ones beside them), for lds_chain128_kernel.
SMALL128_SHAPES = [(128, 128), (96, 128), (100, 70), (128, 40), (65, 97), (3, 128), (128, 90)]


@pytest.mark.parametrize("symmetrize", [True, False])
def test_lds_chain_small_factors(symmetrize):
    """A context whose factors all have padded size <= 64 runs each whole update in
    one workgroup, in LDS, instead of the grouped levels."""
    shapes = SMALL_SHAPES
    say("LDS chain, symmetrize", symmetrize)
    opt = Jorge(shapes, symmetrize=symmetrize)
    opt.set_timing(True)
    opt.step([torch.zeros(s, device="cuda") for s in shapes],
             [to_dev(gradient(0, l, 1, s, 1e-2)) for l, s in enumerate(shapes)], **HP)
    tm = opt.read_timing()
    assert tm["lds_chain"][1] == 1 and tm["gram"][1] == 0 and tm["update"][1] == 0
    # One larger factor brings the levels back, and the small factors join them.
    mixed = Jorge(shapes + [(64, 576)], symmetrize=symmetrize)
    mixed.set_timing(True)
    mixed.step([torch.zeros(s, device="cuda") for s in shapes + [(64, 576)]],
               [to_dev(gradient(0, l, 1, s, 1e-2)) for l, s in enumerate(shapes + [(64, 576)])], **HP)
    assert mixed.read_timing()["lds_chain"][1] == 0 and mixed.read_timing()["gram"][1] >= 1
    a = run_pair(shapes, 6, 1e-2, check_every=3, gpu_kw=dict(symmetrize=symmetrize),
                 orc_kw=dict(symmetrize=symmetrize))
    b = run_pair(shapes, 6, 1e-2, gpu_kw=dict(symmetrize=symmetrize, lds_chain_max=0),
                 orc_kw=dict(symmetrize=symmetrize))
    for l in range(len(shapes)):
        for k in KINDS:
            x, y = a[0].get_state(l, k), b[0].get_state(l, k)
            assert rel(x.cpu().numpy(), y.cpu().numpy()) < 1e-5, (l, k)
        if symmetrize:
            for k in ("L", "R"):
                A = a[0].get_state(l, k)
                assert torch.equal(A, A.T), (l, k)
        d = a[0].read_diag(l)
        assert d["nu_L"] == pytest.approx(a[1].last_diag[l]["nu_L"], rel=1e-5)
        assert d["nu_R"] == pytest.approx(a[1].last_diag[l]["nu_R"], rel=1e-5)


@pytest.mark.parametrize("series_order", [2, 3])
def test_lds_chain128_small_factors(series_order):
    """In a context whose factors all have padded size <= 128, those of 96 and 128 run
    their whole update in lds_chain128_kernel (and the smaller ones in lds_chain_kernel):
    against the oracle, against the grouped levels, bitwise symmetric."""
    shapes = SMALL128_SHAPES
    say("LDS chain 128, series order", series_order)
    kw = dict(series_order=series_order)
    opt = Jorge(shapes, **kw)
    opt.set_timing(True)
    opt.step([torch.zeros(s, device="cuda") for s in shapes],
             [to_dev(gradient(0, l, 1, s, 1e-2)) for l, s in enumerate(shapes)], **HP)
    tm = opt.read_timing()
    assert tm["lds_chain"][1] == 2 and tm["gram"][1] == 0     # both chain kernels, no levels
    a = run_pair(shapes, 6, 1e-2, check_every=2, gpu_kw=kw, orc_kw=kw)
    b = run_pair(shapes, 6, 1e-2, gpu_kw=dict(kw, lds_chain_max=0), orc_kw=kw)
    for l in range(len(shapes)):
        for k in KINDS:
            x, y = a[0].get_state(l, k), b[0].get_state(l, k)
            assert rel(x.cpu().numpy(), y.cpu().numpy()) < 1e-5, (l, k)
        for k in ("L", "R"):
            A = a[0].get_state(l, k)
            assert torch.equal(A, A.T), (l, k)
        d = a[0].read_diag(l)
        assert d["nu_L"] == pytest.approx(a[1].last_diag[l]["nu_L"], rel=1e-5)
        assert d["nu_R"] == pytest.approx(a[1].last_diag[l]["nu_R"], rel=1e-5)


@pytest.mark.parametrize("interval", [1, 2])
def test_lowrank_preconditioning(interval):
    """A factored factor with d > 3k preconditions through A_new H on update steps."""
    shapes = [(64, 576), (256, 1152), (512, 128), (100, 1000), (300, 200)]
    say("low-rank preconditioning, interval", interval)
    a = run_pair(shapes, 6, 1e-2, check_every=2, gpu_kw=dict(precond_interval=interval),
                 orc_kw=dict(precond_interval=interval))
    b = run_pair(shapes, 6, 1e-2, gpu_kw=dict(precond_interval=interval, precond_lowrank=False),
                 orc_kw=dict(precond_interval=interval))
    for l in range(len(shapes)):
        for k in KINDS:
            x, y = a[0].get_state(l, k), b[0].get_state(l, k)
            assert rel(x.cpu().numpy(), y.cpu().numpy()) < 1e-5, (l, k)
        assert rel(a[2][l].cpu().numpy(), b[2][l].cpu().numpy()) < 1e-5
    fl_a, fl_b = a[0].stage_flops(), b[0].stage_flops()
    assert fl_a["uprecond_L"] + fl_a["uprecond_R"] < fl_b["uprecond_L"] + fl_b["uprecond_R"]


# ---------------------------------------------------------------- cubic series term
# series_order=3 keeps the cubic term of Eq. 5 that Section 3 drops: the
# explicit order forms V = b X - e X X and then P = I - a X + X V, the factored
# order V = b S - e S S and W = a A^5 H - A^5 H V, the LDS chain the explicit
# steps in LDS. The shapes put factors in every path of the grouped levels:
# explicit, factored, low-rank preconditioning (factored with d > 3k), and a
# long-K layer whose sparse levels split; an all-small context takes the LDS
# chain.
CUBIC_SHAPES = [(64, 576), (48, 96), (300, 130), (256, 1152), (512, 128), (128, 2048)]


# The squared order needs symmetric factors (its rejection in the literal mode is
# test_literal_mode_without_symmetrization), so it runs with symmetrize only.
@pytest.mark.parametrize("form,symmetrize", [(f, s) for f in FORMS for s in (True, False)
                                             if f != "squared" or s])
def test_cubic_series_term(form, symmetrize):
    say("cubic series term", form, "symmetrize", symmetrize)
    kw = dict(series_order=3, symmetrize=symmetrize)
    opt, orc, pg, po, w = run_pair(CUBIC_SHAPES, 6, 1e-2, check_every=2,
                                   gpu_kw=dict(FORM_KW[form], **kw), orc_kw=kw)
    say("  worst", w)
    # The test discriminates: the quadratic truncation is far from the cubic one here.
    orc2 = JorgeOracle(CUBIC_SHAPES, symmetrize=symmetrize)
    po2 = [initial_params(0, l, s).astype(np.float64) for l, s in enumerate(CUBIC_SHAPES)]
    for t in range(1, 7):
        po2 = orc2.step(po2, [gradient(0, l, t, s, 1e-2) for l, s in enumerate(CUBIC_SHAPES)], **HP)
    gap = max(rel(orc2.layers[l].R, orc.layers[l].R) for l in range(len(CUBIC_SHAPES)))
    assert gap > 100 * w["whole"], (gap, w)


@pytest.mark.parametrize("symmetrize", [True, False])
def test_cubic_series_term_lds_chain(symmetrize):
    say("cubic series term, LDS chain, symmetrize", symmetrize)
    kw = dict(series_order=3, symmetrize=symmetrize)
    a = run_pair(SMALL_SHAPES, 6, 1e-2, check_every=2, gpu_kw=kw, orc_kw=kw)
    b = run_pair(SMALL_SHAPES, 6, 1e-2, gpu_kw=dict(kw, lds_chain_max=0), orc_kw=kw)
    for l in range(len(SMALL_SHAPES)):
        for k in KINDS:
            x, y = a[0].get_state(l, k), b[0].get_state(l, k)
            assert rel(x.cpu().numpy(), y.cpu().numpy()) < 1e-5, (l, k)


@pytest.mark.parametrize("shapes", [[(1, 1)], [(40, 1)], [(33, 65)], [(200, 300)], [(130, 260)]])
@pytest.mark.parametrize("form", FORMS)
def test_cubic_series_first_step(shapes, form):
    say("cubic first step", shapes, form)
    run_pair(shapes, 1, 1e-2, gpu_kw=dict(FORM_KW[form], series_order=3), orc_kw=dict(series_order=3))


def test_cubic_series_launches_and_flops():
    shapes = [(256, 512)]     # L_hat explicit; R_hat (rank 256) squared, with the factored order's poly products
    g = [to_dev(gradient(0, 0, 1, shapes[0], 1e-2))]
    runs = {}
    for order in (2, 3):
        opt = Jorge(shapes, series_order=order)
        opt.set_timing(True)
        opt.step([torch.zeros(shapes[0], device="cuda")], g, 0.1)
        runs[order] = (opt.read_timing(), opt.stage_flops())
    assert runs[2][0]["poly2"][1] == 0 and runs[3][0]["poly2"][1] == 1
    m, n = shapes[0]
    # Explicit L_hat: X V (2 m^3) one level after V; R_hat (k = m): S S (m^3, symmetric).
    f2, f3 = runs[2][1], runs[3][1]
    assert f3["poly2"] == 2 * m ** 3 + 2 * n * m * m
    assert f3["poly"] == 2 * m ** 3 + m ** 3
    assert f2["poly"] == 2 * m ** 3 + 2 * n * m * m


# ---------------------------------------------------------------- HIP graph capture
def test_graph_capture_replays_match_eager():
    """jorge_step launches kernels only (no allocation, memset or host sync), so a
    caller can capture an update step in a HIP graph and replay it with new
    gradients copied into the captured buffers. Each replay, with unrelated eager
    work and synchronisations in between, equals an eager step bitwise."""
    shapes = [(64, 576), (130, 260), (512, 128), (128, 2048)]
    say("graph capture")
    grads = [torch.zeros(s, device="cuda") for s in shapes]
    eager, graphed = Jorge(shapes), Jorge(shapes)
    pe = [to_dev(initial_params(0, l, s)) for l, s in enumerate(shapes)]
    pg = [p.clone() for p in pe]

    def load(t):
        for l, s in enumerate(shapes):
            grads[l].copy_(to_dev(gradient(0, l, t, s, 1e-2)))

    load(1)
    eager.step(pe, grads, **HP)
    graphed.step(pg, grads, **HP)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        graphed.set_stream(torch.cuda.current_stream().cuda_stream)
        graphed.step(pg, grads, **HP)
    graphed.set_stream(torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    for t in range(2, 6):
        load(t)
        eager.step(pe, grads, **HP)
        graph.replay()
        x = torch.randn(1 << 20, device="cuda")
        (x * x).sum().item()
        torch.cuda.synchronize()
        for l in range(len(shapes)):
            assert torch.equal(pe[l], pg[l]), (t, l)
            for k in KINDS:
                assert torch.equal(eager.get_state(l, k), graphed.get_state(l, k)), (t, l, k)


# ---------------------------------------------------------------- maximum size
# A rank-one statistic at the largest dimension the library accepts. For a
# 1 x n layer G = g and R_hat_0 = a I: X = a^4 g^T g = nu u u^T with
# nu = a^4 ||g||^2 and u = g / ||g||, so the series collapses to
# P = I + q u u^T with q = -(c/4) nu + (5c^2/32) nu^2 (- (15c^3/128) nu^3),
# R_hat_1 = s a P, L_hat_1 = s a (1 + q), and since g P = (1 + q) g the grafted
# step is theta_1 = theta_0 (1 - lr wd) - lr g (Eq. 5-7, Alg. 2, Alg. 3). The
# n x n factor (4.3 GB) is checked on sampled entries against this closed form;
# its last element sits at the 2^32 - 4 byte offset of the 32-bit epilogue
# addressing. The n x 1 layer puts the same factor on the L side.
@pytest.mark.parametrize("series_order", [2, 3])
@pytest.mark.parametrize("side", ["R", "L"])
def test_maximum_dimension_rank_one_closed_form(side, series_order):
    from oracle import BETA_CLAMPED, beta_select, init_factor  # noqa: F401
    n = 32768
    shape = (1, n) if side == "R" else (n, 1)
    say("max dimension", shape, "series order", series_order)
    eps, sigma = 1e-6, 1e-2
    g = gradient(0, 0, 1, shape, sigma).astype(np.float64).ravel()
    theta0 = initial_params(0, 0, shape)
    opt = Jorge([shape], eps=eps, series_order=series_order)
    pg = [to_dev(theta0)]
    opt.step(pg, [to_dev(g.reshape(shape))], **HP)
    a = eps ** -0.25
    gg = float(g @ g)
    nu = a ** 4 * gg
    c, s, _ = beta_select(nu, HP["beta2"], BETA_CLAMPED)
    q = -(c / 4) * nu + (5 * c * c / 32) * nu ** 2
    if series_order == 3:
        q -= (15 * c ** 3 / 128) * nu ** 3
    big = opt.get_state(0, side)
    rng = np.random.default_rng(7)
    i = rng.integers(0, n, 4096)
    j = rng.integers(0, n, 4096)
    i = np.concatenate([i, np.arange(0, n, 128), [n - 1, n - 1, 0]])
    j = np.concatenate([j, np.arange(0, n, 128), [n - 1, 0, n - 1]])
    ti, tj = torch.from_numpy(i).cuda(), torch.from_numpy(j).cuda()
    got = big[ti, tj].double().cpu().numpy()
    ref = s * a * ((i == j).astype(np.float64) + q * g[i] * g[j] / gg)
    assert np.abs(got - ref).max() <= 1e-6 * s * a, np.abs(got - ref).max() / (s * a)
    assert torch.equal(big[ti, tj], big[tj, ti])                       # bitwise symmetric
    small = opt.get_state(0, "L" if side == "R" else "R").item()
    assert small == pytest.approx(s * a * (1 + q), rel=1e-6)
    d = opt.read_diag(0)
    assert d["nu_L"] == pytest.approx(nu, rel=1e-4) and d["nu_R"] == pytest.approx(nu, rel=1e-4)
    want = theta0.astype(np.float64).ravel() * (1 - HP["lr"] * HP["weight_decay"]) - HP["lr"] * g
    assert rel(pg[0].cpu().numpy().ravel(), want) <= 1e-6


# ---------------------------------------------------------------- stream switch
def test_stream_switch_orders_the_steps():
    """jorge_set_stream makes later work on the new stream wait for the old stream's work:
    a context stepped on a different side stream every step ends bitwise equal to one that
    stays on the default stream."""
    shapes = [(256, 1152), (64, 576), (130, 260)]
    say("stream switch")
    one, hop = Jorge(shapes), Jorge(shapes)
    p1 = [to_dev(initial_params(0, l, s)) for l, s in enumerate(shapes)]
    p2 = [p.clone() for p in p1]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for t in range(1, 6):
        G = [to_dev(gradient(0, l, t, s, 1e-2)) for l, s in enumerate(shapes)]
        one.step(p1, G, **HP)
        side = streams[t % 2]
        side.wait_stream(torch.cuda.current_stream())     # the gradients' upload
        hop.set_stream(side.cuda_stream)
        with torch.cuda.stream(side):
            hop.step(p2, G, **HP)
        for g in G:
            g.record_stream(side)
    hop.set_stream(torch.cuda.current_stream().cuda_stream)
    hop.synchronize()
    torch.cuda.synchronize()
    for l in range(len(shapes)):
        assert torch.equal(p1[l], p2[l]), l
        for k in KINDS:
            assert torch.equal(one.get_state(l, k), hop.get_state(l, k)), (l, k)
