"""GPU checks of failure detection: non-finite gradients are flagged per layer and
a restored checkpoint recovers from them; a context larger than the device
reports JORGE_ERR_OUT_OF_MEMORY and leaves the library usable.

Every condition is forced from the host with ordinary inputs (a NaN or an
infinity in a gradient, a context too large to allocate); every kernel runs to
its normal end."""
import math

import pytest

torch = pytest.importorskip("torch")

from paper_2310_12298_amd.jorge import Jorge, JorgeError  # noqa: E402

pytestmark = pytest.mark.gpu
HP = dict(lr=0.1, beta2=0.9, beta1=0.9, weight_decay=5e-4)
KINDS = ("L", "R", "mom", "mom_sgd")
# A grouped-level context (one factor above the chains' sizes) and an all-small one (LDS chains).
CONTEXTS = {
    "levels": [(64, 96), (128, 40), (200, 300), (48, 48)],
    "chains": [(64, 96), (128, 40), (100, 70), (48, 48)],
}


def grads_at(shapes, t):
    gen = torch.Generator(device="cuda").manual_seed(7000 + t)
    return [torch.randn(s, generator=gen, device="cuda").mul_(1e-2) for s in shapes]


def checkpoint(opt, params):
    return ({(l, k): opt.get_state(l, k).clone() for l in range(len(params)) for k in KINDS},
            [p.clone() for p in params], opt.t)


def restore(opt, params, ck):
    states, saved, t = ck
    for (l, k), v in states.items():
        opt.set_state(l, k, v)
    for p, s in zip(params, saved):
        p.copy_(s)
    opt.t = t


@pytest.mark.parametrize("ctx", sorted(CONTEXTS))
@pytest.mark.parametrize("value", [math.nan, math.inf, -math.inf])
def test_nonfinite_gradient_is_flagged_and_a_checkpoint_recovers(ctx, value):
    shapes = CONTEXTS[ctx]
    bad_layer = 2
    gen = torch.Generator(device="cuda").manual_seed(11)
    params = [torch.randn(s, generator=gen, device="cuda") for s in shapes]
    ref_params = [p.clone() for p in params]
    opt, ref = Jorge(shapes), Jorge(shapes)
    for t in (1, 2):
        G = grads_at(shapes, t)
        opt.step(params, G, **HP)
        ref.step(ref_params, G, **HP)
    assert opt.nonfinite() == (0, -1)
    ck = checkpoint(opt, params)

    # Step 3 with one non-finite element in one layer's gradient.
    G = grads_at(shapes, 3)
    G_bad = [g.clone() for g in G]
    G_bad[bad_layer][5, 7] = value
    opt.step(params, G_bad, **HP)
    assert opt.nonfinite() == (1, bad_layer)
    assert not torch.isfinite(opt.get_state(bad_layer, "mom_sgd")).all()
    # The other layers' steps are independent of it.
    ref.step(ref_params, G, **HP)
    for l in range(len(shapes)):
        if l != bad_layer:
            assert torch.equal(params[l], ref_params[l]), l
    # The flags were cleared by the read; the layer's m_SGD stays non-finite, so
    # the next step flags it again.
    assert opt.nonfinite() == (0, -1)
    opt.step(params, grads_at(shapes, 4), **HP)
    assert opt.nonfinite() == (1, bad_layer)

    # Recovery: the checkpoint from before the bad step, then the clean step 3
    # and step 4, equal the run that never saw the bad gradient, bitwise.
    restore(opt, params, ck)
    opt.step(params, G, **HP)
    ref.step(ref_params, grads_at(shapes, 4), **HP)
    opt.step(params, grads_at(shapes, 4), **HP)
    assert opt.nonfinite() == (0, -1)
    assert opt.t == ref.t == 4
    for l in range(len(shapes)):
        assert torch.equal(params[l], ref_params[l]), l
        for k in KINDS:
            assert torch.equal(opt.get_state(l, k), ref.get_state(l, k)), (l, k)


def test_flags_cover_every_layer_batch():
    # 300 layers take two batches of the per-layer kernels; each flag is its own.
    shapes = [(32 + 16 * (i % 5), 48 + 8 * (i % 7)) for i in range(300)]
    params = [torch.zeros(s, device="cuda") for s in shapes]
    opt = Jorge(shapes)
    for t in (1, 2):
        opt.step(params, grads_at(shapes, t), **HP)
    assert opt.nonfinite() == (0, -1)
    G = grads_at(shapes, 3)
    for l in (0, 255, 256, 299):
        G[l][0, 0] = math.nan
    opt.step(params, G, **HP)
    assert opt.nonfinite() == (4, 0)


def test_context_larger_than_the_device_reports_out_of_memory():
    # 32 layers of 16384 x 16384 need about 480 GiB of device memory.
    shapes = [(16384, 16384)] * 32
    assert Jorge.plan(shapes) > 400 * 2**30
    with pytest.raises(JorgeError) as err:
        Jorge(shapes)
    assert err.value.status == -2, err.value
    # Nothing of the failed call stays behind: a new context steps normally.
    shapes = [(64, 96), (200, 300)]
    params = [torch.zeros(s, device="cuda") for s in shapes]
    opt = Jorge(shapes)
    opt.step(params, grads_at(shapes, 1), **HP)
    torch.cuda.synchronize()
    assert all(torch.isfinite(p).all() for p in params)
    assert opt.nonfinite() == (0, -1)
