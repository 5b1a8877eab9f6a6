"""C-ABI checks that need no GPU: the library loads, exports every entry point
that include/jorge.h declares, and rejects invalid arguments before any HIP
call is made."""
import ctypes
import os
import re

import pytest

from paper_2310_12298_amd import jorge as J

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "jorge.h")

ERR_INVALID, ERR_UNSUPPORTED = -1, -4


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return re.findall(r"\b(jorge_[a-z_]+)\s*\(", text)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(J.LIB_PATH):
        from paper_2310_12298_amd.build import build_library
        build_library()
    return J.load_library()


def test_header_declares_expected_api():
    names = set(declared_functions())
    assert {"jorge_create", "jorge_step", "jorge_destroy", "jorge_get_state", "jorge_set_state"} <= names


def test_every_declared_symbol_is_exported(lib):
    names = set(declared_functions())
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing
    # The binding marshals exactly the declared entry points.
    assert names == set(J._SIGNATURES)


def test_hparams_default(lib):
    hp = J.HParams()
    assert lib.jorge_hparams_default(ctypes.byref(hp)) == 0
    assert (hp.eps, hp.precond_interval, hp.beta_mode, hp.graft, hp.symmetrize,
            hp.factor_form, hp.split_k, hp.lds_chain_max, hp.precond_lowrank,
            hp.series_order) == (1e-6, 1, 2, 1, 1, 0, 1, 128, 1, 2)
    assert lib.jorge_hparams_default(None) == ERR_INVALID


def _create(lib, shapes, hp=None):
    arr = (J.Shape * max(1, len(shapes)))(*[J.Shape(m, n) for m, n in shapes])
    out = ctypes.c_void_p(12345)
    st = lib.jorge_create(arr, len(shapes), ctypes.byref(hp) if hp else None, None, ctypes.byref(out))
    return st, out.value


@pytest.mark.parametrize("shapes", [[], [(0, 4)], [(4, 0)], [(-1, 3)], [(3, 4), (5, -2)]])
def test_create_rejects_bad_shapes(lib, shapes):
    st, out = _create(lib, shapes)
    assert st == ERR_INVALID and out is None


def test_create_rejects_oversize(lib):
    st, out = _create(lib, [(4, 32769)])
    assert st == ERR_UNSUPPORTED and out is None


@pytest.mark.parametrize("field,value", [("eps", 0.0), ("eps", -1.0), ("eps", float("inf")),
                                         ("eps", float("nan")), ("precond_interval", 0),
                                         ("beta_mode", 3), ("beta_mode", -1), ("graft", 2),
                                         ("symmetrize", -1), ("factor_form", -1),
                                         ("factor_form", 4), ("split_k", 2), ("split_k", -1),
                                         ("lds_chain_max", -1), ("lds_chain_max", 129),
                                         ("precond_lowrank", 2), ("series_order", 1),
                                         ("series_order", 4), ("series_order", 0)])
def test_create_rejects_bad_hparams(lib, field, value):
    hp = J.HParams()
    lib.jorge_hparams_default(ctypes.byref(hp))
    setattr(hp, field, value)
    st, out = _create(lib, [(4, 4)], hp)
    assert st == ERR_INVALID and out is None


def test_null_arguments(lib):
    shp = (J.Shape * 1)(J.Shape(2, 2))
    assert lib.jorge_create(shp, 1, None, None, None) == ERR_INVALID
    assert lib.jorge_create(None, 1, None, None, ctypes.byref(ctypes.c_void_p())) == ERR_INVALID
    P = ctypes.c_void_p
    arr = (P * 1)(P(0))
    assert lib.jorge_step(None, arr, arr, 0.1, 0.9, 0.9, 0.0) == ERR_INVALID
    assert lib.jorge_get_state(None, 0, 0, P(16), 4) == ERR_INVALID
    assert lib.jorge_set_state(None, 0, 0, P(16), 4) == ERR_INVALID
    assert lib.jorge_state_ptr(None, 0, 0, ctypes.byref(P()), ctypes.byref(ctypes.c_int64())) == ERR_INVALID
    assert lib.jorge_get_step(None, ctypes.byref(ctypes.c_int64())) == ERR_INVALID
    assert lib.jorge_set_step(None, 0) == ERR_INVALID
    assert lib.jorge_read_diag(None, 0, (ctypes.c_double * 7)()) == ERR_INVALID
    assert lib.jorge_nonfinite(None, ctypes.byref(ctypes.c_int32()), None) == ERR_INVALID
    assert lib.jorge_set_stream(None, None) == ERR_INVALID
    assert lib.jorge_synchronize(None) == ERR_INVALID
    assert lib.jorge_device_bytes(None, ctypes.byref(ctypes.c_int64())) == ERR_INVALID
    assert lib.jorge_set_timing(None, 1) == ERR_INVALID
    assert lib.jorge_read_timing(None, None, None, 0) == ERR_INVALID
    assert lib.jorge_reset_timing(None) == ERR_INVALID
    assert lib.jorge_stage_flops(None, (ctypes.c_double * 1)(), 1) == ERR_INVALID
    assert lib.jorge_factor_form(None, 0, 0, ctypes.byref(ctypes.c_int32())) == ERR_INVALID
    assert lib.jorge_plan(shp, 1, None, None) == ERR_INVALID
    assert lib.jorge_plan(None, 1, None, ctypes.byref(ctypes.c_int64())) == ERR_INVALID
    lib.jorge_destroy(None)
    assert lib.jorge_last_error(None) == b""


def test_stage_names_and_status_strings(lib):
    n = lib.jorge_num_stages()
    names = [lib.jorge_stage_name(i).decode() for i in range(n)]
    assert names[0] == "stage_in" and "xform" in names and "weight" in names and "split_fixup" in names
    assert len(set(names)) == n
    assert lib.jorge_stage_name(n) is None and lib.jorge_stage_name(-1) is None
    assert lib.jorge_status_string(0) == b"ok"
    assert lib.jorge_status_string(-1) == b"invalid argument"
    assert lib.jorge_status_string(-99) == b"unknown status"


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    monkeypatch.setattr(J, "_LIB", None)
    with pytest.raises(FileNotFoundError):
        J.load_library(str(tmp_path / "missing.so"))


# ---------------------------------------------------------------- host-side plan checks
# jorge_plan builds every launch table exactly as jorge_create does and checks,
# on the host, that each access of each grouped launch stays inside its buffer
# with the alignment and extents the kernels assume. These run without a GPU.

from paper_2310_12298_amd.workloads import CONFIGS  # noqa: E402

FORMS = ("auto", "explicit", "factored", "squared")


def forms_for(symmetrize):
    # The squared order needs symmetric factors.
    return FORMS if symmetrize else tuple(f for f in FORMS if f != "squared")


@pytest.mark.parametrize("name", sorted(CONFIGS))
@pytest.mark.parametrize("symmetrize", [True, False])
def test_plan_tables_of_every_workload(lib, name, symmetrize):
    shapes = CONFIGS[name][0]
    forms = forms_for(symmetrize)
    sizes = {f: J.Jorge.plan(shapes, symmetrize=symmetrize, factor_form=f, split_k=False) for f in forms}
    assert all(v > 0 for v in sizes.values())
    # Per factor, auto takes one of the forms' workspaces.
    assert sizes["auto"] <= max(sizes[f] for f in forms if f != "auto")
    for f in forms:   # split plans are checked too; they only add their workspace
        assert J.Jorge.plan(shapes, symmetrize=symmetrize, factor_form=f) >= sizes[f]
        # The cubic series term adds products (and, factored, one k x k buffer per factor).
        assert J.Jorge.plan(shapes, symmetrize=symmetrize, factor_form=f, series_order=3) > 0


def test_plan_splits_long_tiles_of_sparse_levels(lib):
    # One 512 x 4608 layer: ~150 tiles per level with K up to 4608 get split;
    # the ResNet-50 set keeps its full levels whole.
    one = [(512, 4608)]
    assert J.Jorge.plan(one) > J.Jorge.plan(one, split_k=False)
    r50 = J.Jorge.plan_stages(CONFIGS["resnet50"][0])
    assert all(r50[name][1] == 0 for name in ("gram", "pow4", "xform", "update")), r50


def test_plan_stages_split_choices(lib):
    one = [(512, 4608)]
    plain = J.Jorge.plan_stages(one, split_k=False)
    split = J.Jorge.plan_stages(one)
    assert set(plain) == set(split) and all(v[1] == 0 for v in plain.values())
    for name, (units, nsplit, _) in split.items():
        # A split tile becomes at least two units; an unsplit level keeps its tiles.
        assert units >= plain[name][0] + nsplit, name
        assert (units == plain[name][0]) == (nsplit == 0), name
    # The chain levels hold ~150 tiles of K = 4608 for 512 CUs' worth of slots: split.
    for name in ("gram", "pow4", "xform", "chain4", "chain5"):
        assert split[name][1] >= 144, (name, split[name])
    # The update level's 16 tiles of W^T H (K = 4608) would outlast its 682 short
    # tiles: they are cut.
    assert split["update"][1] >= 16
    # Plans are deterministic.
    assert J.Jorge.plan_stages(one) == split
    # Full levels are left whole.
    r50 = J.Jorge.plan_stages(CONFIGS["resnet50"][0])
    assert all(r50[name][1] == 0 for name in ("gram", "pow4", "xform", "update", "uprecond_L")), r50


def test_plan_stages_small_mode(lib):
    # Full levels of many small layers run their at-most-64-wide products as 64 x 64
    # blocks; a level of a few tiles (one 64 x 576 layer) keeps 128 x 128 tiles.
    many = J.Jorge.plan_stages(CONFIGS["many_small"][0])
    assert many["gram"][2] > 0 and many["pow4"][2] > 0
    for name, (units, nsplit, small) in many.items():
        assert units >= (small + 3) // 4, name   # at most four blocks per unit
    one = J.Jorge.plan_stages([(64, 576)])
    assert all(v[2] == 0 for v in one.values()), one
    # Small layers' preconditioning products too (they update the momentum).
    assert many["precond_R"][2] > 0 and many["uprecond_R"][2] > 0
    # The literal mode's NN launches have no small mode; its NT products still do.
    lit = J.Jorge.plan_stages(CONFIGS["many_small"][0], symmetrize=False)
    assert lit["gram"][2] > 0


def test_plan_stages_rejects_bad_arguments(lib):
    arr = (J.Shape * 1)(J.Shape(4, 4))
    units = (ctypes.c_int64 * 4)()
    assert lib.jorge_plan_stages(arr, 1, None, None, None, None, 4) == ERR_INVALID
    assert lib.jorge_plan_stages(arr, 1, None, units, None, None, -1) == ERR_INVALID
    assert lib.jorge_plan_stages(arr, 1, None, None, None, None, 0) == 0
    assert lib.jorge_plan_stages(arr, 0, None, units, None, None, 4) == ERR_INVALID
    bad = (J.Shape * 1)(J.Shape(4, 0))
    assert lib.jorge_plan_stages(bad, 1, None, units, None, None, 4) == ERR_INVALID


@pytest.mark.parametrize("form", FORMS)
@pytest.mark.parametrize("symmetrize", [True, False])
def test_plan_tables_of_edge_shapes(lib, form, symmetrize):
    if form not in forms_for(symmetrize):
        with pytest.raises(J.JorgeError):
            J.Jorge.plan([(4, 4)], symmetrize=symmetrize, factor_form=form)
        return
    shapes = [(1, 1), (1, 40), (40, 1), (33, 65), (5, 3), (127, 129), (128, 128), (129, 4000),
              (4000, 129), (32, 32), (300, 200), (1, 4608)]
    assert J.Jorge.plan(shapes, symmetrize=symmetrize, factor_form=form) > 0
    for s in shapes:
        assert J.Jorge.plan([s], symmetrize=symmetrize, factor_form=form) > 0
        assert J.Jorge.plan([s], symmetrize=symmetrize, factor_form=form, split_k=False) > 0
        for lds in (0, 32, 64, 96, 128):
            assert J.Jorge.plan([s], symmetrize=symmetrize, factor_form=form, lds_chain_max=lds) > 0
        assert J.Jorge.plan([s], symmetrize=symmetrize, factor_form=form, precond_lowrank=False) > 0
        assert J.Jorge.plan([s], symmetrize=symmetrize, factor_form=form, series_order=3) > 0


def test_plan_tables_of_random_shapes(lib):
    import numpy as np
    rng = np.random.default_rng(11)
    for _ in range(40):
        shapes = [tuple(int(x) for x in rng.integers(1, 700, size=2)) for _ in range(int(rng.integers(1, 6)))]
        for form in FORMS:
            assert J.Jorge.plan(shapes, factor_form=form) > 0, shapes
            sym = bool(rng.integers(2)) or form == "squared"
            assert J.Jorge.plan(shapes, factor_form=form, series_order=3, symmetrize=sym) > 0


def test_plan_rejects_what_create_rejects(lib):
    with pytest.raises(J.JorgeError):
        J.Jorge.plan([(4, 0)])
    with pytest.raises(J.JorgeError):
        J.Jorge.plan([(4, 32769)])
    with pytest.raises(J.JorgeError):
        J.Jorge.plan([(4, 4)], factor_form=7)


def test_plan_small_contexts_take_the_lds_chains(lib):
    """Every factor of padded size <= lds_chain_max: the LDS chains replace the grouped
    levels (no GEMM units); sizes 96 and 128 need symmetric factors; one larger factor
    brings the levels back for all."""
    levels = ("gram", "pow4", "xform", "chain4", "chain5", "poly", "poly2", "update")

    def units(shapes, **kw):   # work units of the factor-update levels (the preconditioning stays)
        st = J.Jorge.plan_stages(shapes, **kw)
        return sum(st[k][0] for k in levels)

    small = [(128, 128), (96, 128), (100, 70), (128, 40), (65, 97), (3, 128), (128, 90)]
    assert units(small) == 0
    assert units(small, lds_chain_max=64) > 0 and units(small, lds_chain_max=0) > 0
    assert units(small, symmetrize=False) > 0                 # the 96- and 128-wide chain needs symmetry
    assert units([(64, 64), (40, 33)], symmetrize=False) == 0
    assert units(small + [(64, 576)]) > 0


# Property-based: any valid combination of shapes and options plans, and its
# launch tables pass the library's own bounds and coverage check (jorge_plan
# builds and checks them on the host); an invalid one is refused, never planned.
from hypothesis import HealthCheck, given, settings  # noqa: E402
from hypothesis import strategies as hs  # noqa: E402

_dims = hs.one_of(hs.integers(1, 300), hs.sampled_from([31, 32, 33, 64, 96, 127, 128, 129, 256, 576, 1152, 2304]))
_opts = hs.fixed_dictionaries({
    "factor_form": hs.sampled_from(FORMS),
    "symmetrize": hs.booleans(),
    "split_k": hs.booleans(),
    "lds_chain_max": hs.sampled_from([0, 32, 64, 96, 128]),
    "precond_interval": hs.integers(1, 60),
    "beta_mode": hs.sampled_from(["fixed", "dynamic", "clamped"]),
    "graft": hs.booleans(),
    "precond_lowrank": hs.booleans(),
    "series_order": hs.sampled_from([2, 3]),
})


@settings(max_examples=120, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])
@given(shapes=hs.lists(hs.tuples(_dims, _dims), min_size=1, max_size=6), opts=_opts)
def test_plan_any_valid_options(lib, shapes, opts):
    if opts["factor_form"] == "squared" and not opts["symmetrize"]:
        with pytest.raises(J.JorgeError):
            J.Jorge.plan(shapes, **opts)
        return
    assert J.Jorge.plan(shapes, **opts) > 0
    st = J.Jorge.plan_stages(shapes, **opts)
    for name, (units, split, small) in st.items():
        assert units >= 0 and 0 <= split <= units and small >= 0, (name, units, split, small)
        if not opts["split_k"]:
            assert split == 0, name
