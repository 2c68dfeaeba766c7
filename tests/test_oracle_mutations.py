"""Planted mistakes in the oracle must fail its pins.

Each mutant is one plausible slip in the oracle -- a one-line change of the C
enumeration (compiled apart into a temporary library) or of one of the Python
functions (the function's own source with one edit) -- and the committed pin
tests are run against it, cheapest first, until one fails.  A mutant that
every pin lets through is a gap in the pins.  The unmutated sources, built and
loaded the same way, pass the same pins (a check on the harness itself).

CPU only: the GPU path is not involved.
"""
import inspect
import itertools
import os
import subprocess

import numpy as np
import pytest

import oracle
import test_oracle_bruteforce as bf
import test_oracle_grad as grad
import test_oracle_invariance as inv
import test_oracle_locations as locs
import test_oracle_pins as pins
import test_oracle_theta as th
import test_oracle_subnetwork as subt
import test_oracle_training as tr
import test_oracle_variable_k as vk
from oracle import subnetwork

_SRC = os.path.join(os.path.dirname(oracle.__file__), "lram_oracle.c")
_counter = itertools.count()


# ---------------------------------------------------------------------------
# Planting

def _build_c(tmp_path, text):
    """Compiles a variant of the C helper under a fresh name (the loader
    caches libraries by path) with the oracle's own flags."""
    n = next(_counter)
    src = tmp_path / ("oracle_variant_%d.c" % n)
    lib = tmp_path / ("liboracle_variant_%d.so" % n)
    src.write_text(text)
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
                    "-fno-fast-math", str(src), "-o", str(lib), "-lm"], check=True)
    return str(lib)


def _plant_c(monkeypatch, tmp_path, old, new):
    text = open(_SRC).read()
    assert text.count(old) == 1, old
    path = _build_c(tmp_path, text.replace(old, new))
    monkeypatch.setattr(oracle, "_LIB_PATH", path)
    monkeypatch.setattr(oracle, "_lib", None)


def _plant_py(monkeypatch, name, old, new, module=oracle):
    """Replaces module.<name> by its own source with one edit."""
    src = inspect.getsource(getattr(module, name))
    assert src.count(old) == 1, (name, old)
    ns = dict(vars(module))
    exec(compile(src.replace(old, new), "<mutant of %s.%s>" % (module.__name__, name), "exec"), ns)
    monkeypatch.setattr(module, name, ns[name])


def _first_failure(battery):
    """Name of the first pin that fails (None: every pin passed)."""
    for name, check in battery:
        try:
            check()
        except Exception:  # an assertion, or the oracle refusing its own result
            return name
    return None


# ---------------------------------------------------------------------------
# Pin batteries (the committed tests, cheapest first)

def _core_battery():
    cache = {}

    def mc():
        if "mc" not in cache:  # the pins module's Monte Carlo sample, drawn with the planted oracle
            rng = np.random.default_rng(20210707)
            cache["mc"] = oracle.neighbors((rng.random((40000, 8)) * 8).astype(np.float32), pins.K8)
        return cache["mc"]

    return [
        ("lattice point returns its value", pins.test_lattice_point_returns_its_value),
        ("deep hole: 16 neighbours of weight 1/16", pins.test_deep_hole_sixteen_sixteenths),
        ("recipe weight is the kernel", pins.test_recipe_weight_is_the_kernel),
        ("total weight 1 at lattice points and deep holes", pins.test_total_weight_one_at_lattice_points_and_deep_holes),
        ("shell of 240 nearest neighbours", pins.test_nearest_neighbour_shell_is_240),
        ("x is the exact fmod of 2q", bf.test_bruteforce_x_is_exact_fmod),
        ("location map is a bijection", lambda: locs.test_location_is_bijection((2, 4, 2, 2, 4, 2, 2, 2))),
        ("location map is periodic", lambda: locs.test_location_is_periodic((4, 6, 8, 2, 4, 10, 2, 4))),
        ("Table 1 mean support", lambda: pins.test_mean_support_matches_table1(mc())),
        ("Table 1 support bounds", lambda: pins.test_support_bounds_table1(mc())),
        ("Table 1 maximum next to a lattice point", pins.test_max_support_121_next_to_lattice_point),
        ("total weight bounds", lambda: pins.test_total_weight_bounds(mc())),
        ("covering radius", lambda: pins.test_covering_radius(mc())),
        ("top-32 weight share", lambda: pins.test_top32_weight_share(mc())),
        ("torus periods", inv.test_torus_period_leaves_everything_unchanged),
        ("lattice translations", inv.test_lattice_translation_shifts_lifts),
        ("table adjoint at K = 2", lambda: grad.test_table_gradient_adjoint((2,) * 8)),
        ("dq against finite differences", lambda: grad.test_dq_matches_central_differences((4,) * 8)),
        ("brute force at K = 4", lambda: bf.test_oracle_matches_bruteforce((4,) * 8)),
    ]


def _theta_battery():
    return [
        ("quarter turns hit lattice points",
         lambda: [th.test_quarter_turns_hit_lattice_points(*a) for a in ((1, 0, 0), (0, 1, 2), (-1, 0, 4), (0, -1, -2))]),
        ("origin row", th.test_origin_row_is_row_zero),
        ("scale of the displayed formula", th.test_scale_is_reciprocal_sum_of_reciprocal_moduli),
        ("zero and non-finite entries", th.test_zero_and_nonfinite_entries),
        ("homogeneity", th.test_homogeneous_of_degree_one),
        ("table adjoint", th.test_grad_table_adjoint),
        ("grad z against finite differences", th.test_grad_z_matches_finite_differences),
    ]


def _variable_k_battery():
    return [
        ("closest k are prefixes", vk.test_closest_k_are_prefixes),
        ("untruncated total weight", vk.test_untruncated_total_weight),
        ("rounding-admitted shell", vk.test_rounding_can_admit_the_shell_but_never_beyond_it),
        ("whole support against the brute force at K = 4", lambda: vk.test_whole_support_matches_bruteforce((4,) * 8)),
    ]


def _subnetwork_battery():
    return [
        ("identity dense parts reduce to theta", subt.test_identity_dense_parts_reduce_to_theta),
        ("training normalisation closed forms", subt.test_training_normalisation_closed_forms),
        ("gradients against finite differences", lambda: subt.test_gradients_match_directional_finite_differences(False)),
        ("training gradients against finite differences",
         lambda: subt.test_gradients_match_directional_finite_differences(True)),
    ]


def _training_battery():
    return [
        ("Adam = torch.optim.Adam", tr.test_adam_matches_torch_when_every_row_is_touched),
        ("Adam laziness and first step", tr.test_adam_is_lazy_on_untouched_rows_and_first_step_closed_form),
        ("statistics uniform on lattice points", tr.test_stats_uniform_at_lattice_points),
        ("statistics invariance and single lookup", tr.test_stats_scale_invariance_and_single_lookup),
    ]


# ---------------------------------------------------------------------------
# Mutants

C_MUTANTS = {
    # Sec. 2.5: the support is the open ball r^2 < 8
    "closed support": ("if (!(d < 8.0f)) return;", "if (!(d <= 8.0f)) return;"),
    # Sec. 2.4: coordinate sum 0 mod 4
    "coordinate sum even instead of 0 mod 4": ("if (floor_mod(sum, 4) != 0) return;",
                                                "if (floor_mod(sum, 2) != 0) return;"),
    "odd coset dropped": ("      enum_coset(&c, 0, 1, k, 0.0, 0);\n", ""),
    # Sec. 2.5: f(r) = (1 - r^2/8)^4
    "kernel cubed": ("  double u2 = u * u;\n  return u2 * u2;", "  double u2 = u * u;\n  return u2 * u;"),
    "kernel radius 2 instead of sqrt 8": ("double u = 1.0 - d2 / 8.0;", "double u = 1.0 - d2 / 4.0;"),
    # the fp32 recipe weight is the same kernel, u^4
    "recipe weight cubed": ("w32[o] = u2 * u2;", "w32[o] = u2 * u;"),
    "recipe weight squared": ("w32[o] = u2 * u2;", "w32[o] = u * u;"),
    "recipe weight with radius 2": ("float u = 1.0f - r->d * 0.125f;", "float u = 1.0f - r->d * 0.25f;"),
    # Sec. 2.6: the closest 32
    "farthest points first": ("if (bx != by) return bx < by ? -1 : 1;", "if (bx != by) return bx < by ? 1 : -1;"),
    "ties by descending location": ("if (x->slot != y->slot) return x->slot < y->slot ? -1 : 1;",
                                    "if (x->slot != y->slot) return x->slot < y->slot ? 1 : -1;"),
    # the user scale: x = 2q on a torus of side 2K
    "query not doubled": ("x[i] = fmodf(2.0f * qi, 2.0f * (float)K[i]);", "x[i] = fmodf(qi, 2.0f * (float)K[i]);"),
    # Sec. 2.2: locations of Lambda / L_K
    "remainder instead of floor mod": ("  return r < 0 ? r + m : r;", "  return r;"),
    "location strides shifted": ("for (int i = 1; i < 7; i++) idx = idx * K[i] + Y[i];",
                                 "for (int i = 1; i < 7; i++) idx = idx * K[i - 1] + Y[i];"),
    "coset offset forgotten": ("return (int32_t)(eps * (N / 2) + idx);", "return (int32_t)(idx);"),
    "pruning without slack": ("const double LIM = 8.0 + 1e-3;", "const double LIM = 7.99;"),
}

PY_CORE_MUTANTS = {
    # Sec. 2.6: dq through w = (1 - r^2/8)^4, x = 2q
    "dq sign": ("grad_query", "a = np.where(valid, -2.0 * u ** 3 * gv, 0.0)",
                "a = np.where(valid, 2.0 * u ** 3 * gv, 0.0)"),
    "dq without dx/dq = 2": ("grad_query", "a = np.where(valid, -2.0 * u ** 3 * gv, 0.0)",
                             "a = np.where(valid, -1.0 * u ** 3 * gv, 0.0)"),
    "dq with u squared": ("grad_query", "a = np.where(valid, -2.0 * u ** 3 * gv, 0.0)",
                          "a = np.where(valid, -2.0 * u ** 2 * gv, 0.0)"),
    "dq from the lattice point minus the query": ("grad_query", 'e = nb["x"].astype(np.float64)[..., None, :] - nb["lift"].astype(np.float64)',
                                                 'e = nb["lift"].astype(np.float64) - nb["x"].astype(np.float64)[..., None, :]'),
    # Sec. 2.2: phi = sum_j w_j v_j
    "forward without weights": ("forward", 'return np.einsum("...j,...jm->...m", w, np.asarray(rows, np.float64))',
                                'return np.einsum("...j,...jm->...m", (w > 0) * 1.0, np.asarray(rows, np.float64))'),
    # dV[s] accumulates every pair that reads s
    "table gradient overwrites": ("grad_table_rows", "np.add.at(acc, inv, contrib)", "acc[inv] = contrib"),
    "table gradient without weights": ("grad_table_rows", "contrib = (w[:, :, None] * Gf[:, None, :])[valid]",
                                       "contrib = (np.ones_like(w)[:, :, None] * Gf[:, None, :])[valid]"),
}

C_VARIABLE_K_MUTANTS = {
    # Sec. 2.2 / 2.5: the untruncated sum runs over the whole support
    "whole support cut at 121 points": ("      if (j < c.n) {", "      if (j < c.n && j < 121) {"),
}

PY_SUBNETWORK_MUTANTS = {
    # Sec. 3.1: y = W2 theta(BN(W1 x + b1)) + b2
    "first dense layer transposed": ("forward", 'pre = x @ p["W1"].T + p["b1"]', 'pre = x @ p["W1"] + p["b1"]'),
    "batch norm without the square root": ("_normalise", 'inv = 1.0 / np.sqrt(var + p["eps"])',
                                           'inv = 1.0 / (var + p["eps"])'),
    "gamma gradient from the unnormalised features": ("backward", 'g["gamma"] = (dz * st["xhat"]).sum(0)',
                                                      'g["gamma"] = (dz * (st["pre"] - st["mu"])).sum(0)'),
    "pre-activation gradient without the normalisation": ("backward", 'dpre = dxhat * st["inv"]',
                                                          'dpre = dxhat'),
    # Sec. 3.1 / 4.1 in training: batch statistics, biased variance, and the
    # gradient through them
    "batch variance unbiased": ("_normalise", "var = ((pre - mu) ** 2).mean(0)",
                                "var = ((pre - mu) ** 2).sum(0) / (pre.shape[0] - 1)"),
    "batch mean from the running mean": ("_normalise", "mu = pre.mean(0)", 'mu = p["mu"]'),
    "training gradient without the batch statistics": (
        "backward", 'dpre = st["inv"] * (dxhat - dxhat.mean(0) - st["xhat"] * (dxhat * st["xhat"]).mean(0))',
        'dpre = st["inv"] * dxhat'),
    "training gradient without the variance term": (
        "backward", 'dpre = st["inv"] * (dxhat - dxhat.mean(0) - st["xhat"] * (dxhat * st["xhat"]).mean(0))',
        'dpre = st["inv"] * (dxhat - dxhat.mean(0))'),
    "training gradient without the mean term": (
        "backward", 'dpre = st["inv"] * (dxhat - dxhat.mean(0) - st["xhat"] * (dxhat * st["xhat"]).mean(0))',
        'dpre = st["inv"] * (dxhat - st["xhat"] * (dxhat * st["xhat"]).mean(0))'),
}

PY_THETA_MUTANTS = {
    # Sec. 2.3: q_i = (K_i / 2 pi) arg z_i, s = (sum 1/|z_i|)^-1
    "arg with swapped atan2 arguments": ("theta_coords", "q = (np.arctan2(b, a) * c).astype(np.float32)",
                                         "q = (np.arctan2(a, b) * c).astype(np.float32)"),
    "arg not divided by 2 pi": ("theta_coords", "c = K.astype(np.float64) / (2.0 * np.pi)",
                                "c = K.astype(np.float64) / np.pi"),
    "harmonic mean as the scale": ("theta_coords", "s = 1.0 / np.sum(1.0 / np.hypot(a, b), axis=-1)",
                                   "s = 8.0 / np.sum(1.0 / np.hypot(a, b), axis=-1)"),
    "output not scaled": ("theta_forward", "return np.asarray(s, np.float64)[..., None] * forward(nb, rows)",
                          "return forward(nb, rows)"),
    "table gradient not scaled": ("theta_grad_table_rows",
                                  "return grad_table_rows(nb, np.asarray(G, np.float64) * np.asarray(s, np.float64)[..., None], weights)",
                                  "return grad_table_rows(nb, np.asarray(G, np.float64), weights)"),
    "d arg / d Re z sign": ("theta_grad_z", "ga = dLds[..., None] * s[..., None] ** 2 * a / r3 - dLdq * c * b / r2",
                            "ga = dLds[..., None] * s[..., None] ** 2 * a / r3 + dLdq * c * b / r2"),
    "d s / d z without s squared": ("theta_grad_z", "gb = dLds[..., None] * s[..., None] ** 2 * b / r3 + dLdq * c * a / r2",
                                    "gb = dLds[..., None] * s[..., None] * b / r3 + dLdq * c * a / r2"),
}

PY_TRAINING_MUTANTS = {
    # Sec. 3.2: Adam (Algorithm 1 of Adam)
    "no bias correction": ("sparse_adam", "mh = m1[rows] / (1 - beta1 ** step)", "mh = m1[rows]"),
    "eps inside the square root": ("sparse_adam", "V[rows] = V[rows] - lr * mh / (np.sqrt(vh) + eps)",
                                   "V[rows] = V[rows] - lr * mh / np.sqrt(vh + eps)"),
    "moments decay on untouched rows": ("sparse_adam", "m1[rows] = beta1 * m1[rows] + (1 - beta1) * g[rows]",
                                        "m1 = beta1 * m1 + (1 - beta1) * g"),
    # Sec. 4.3, Table 5
    "access counts instead of weights": ("access_histogram", "return np.bincount(s[ok], weights=w[ok], minlength=N).astype(np.float64)",
                                         "return np.bincount(s[ok], minlength=N).astype(np.float64)"),
    "KL of uniform from p": ("access_stats", "return float((h > 0).mean()), float(np.sum(p * np.log(p * N)))",
                             "return float((h > 0).mean()), float(np.sum(np.log(1.0 / (p * N))) / N)"),
}


def test_unmutated_c_source_passes_the_pins(monkeypatch, tmp_path):
    """The harness itself: the oracle's own source, compiled apart and loaded
    as the mutants are, passes every core pin."""
    monkeypatch.setattr(oracle, "_LIB_PATH", _build_c(tmp_path, open(_SRC).read()))
    monkeypatch.setattr(oracle, "_lib", None)
    assert _first_failure(_core_battery()) is None


@pytest.mark.parametrize("name", sorted(C_MUTANTS))
def test_c_mutant_is_caught(name, monkeypatch, tmp_path):
    _plant_c(monkeypatch, tmp_path, *C_MUTANTS[name])
    caught = _first_failure(_core_battery())
    print("%s: caught by %s" % (name, caught))
    assert caught is not None, name


@pytest.mark.parametrize("name", sorted(PY_CORE_MUTANTS))
def test_python_mutant_is_caught(name, monkeypatch):
    _plant_py(monkeypatch, *PY_CORE_MUTANTS[name])
    caught = _first_failure(_core_battery())
    print("%s: caught by %s" % (name, caught))
    assert caught is not None, name


@pytest.mark.parametrize("name", sorted(PY_THETA_MUTANTS))
def test_theta_mutant_is_caught(name, monkeypatch):
    _plant_py(monkeypatch, *PY_THETA_MUTANTS[name])
    caught = _first_failure(_theta_battery())
    print("%s: caught by %s" % (name, caught))
    assert caught is not None, name


@pytest.mark.parametrize("name", sorted(PY_TRAINING_MUTANTS))
def test_training_mutant_is_caught(name, monkeypatch):
    _plant_py(monkeypatch, *PY_TRAINING_MUTANTS[name])
    caught = _first_failure(_training_battery())
    print("%s: caught by %s" % (name, caught))
    assert caught is not None, name


@pytest.mark.parametrize("name", sorted(C_VARIABLE_K_MUTANTS))
def test_variable_k_mutant_is_caught(name, monkeypatch, tmp_path):
    _plant_c(monkeypatch, tmp_path, *C_VARIABLE_K_MUTANTS[name])
    caught = _first_failure(_variable_k_battery())
    print("%s: caught by %s" % (name, caught))
    assert caught is not None, name


@pytest.mark.parametrize("name", sorted(PY_SUBNETWORK_MUTANTS))
def test_subnetwork_mutant_is_caught(name, monkeypatch):
    _plant_py(monkeypatch, *PY_SUBNETWORK_MUTANTS[name], module=subnetwork)
    caught = _first_failure(_subnetwork_battery())
    print("%s: caught by %s" % (name, caught))
    assert caught is not None, name


def test_python_batteries_pass_unmutated():
    assert _first_failure(_theta_battery()) is None
    assert _first_failure(_training_battery()) is None
    assert _first_failure(_subnetwork_battery()) is None


def test_unmutated_c_source_passes_the_variable_k_pins(monkeypatch, tmp_path):
    monkeypatch.setattr(oracle, "_LIB_PATH", _build_c(tmp_path, open(_SRC).read()))
    monkeypatch.setattr(oracle, "_lib", None)
    assert _first_failure(_variable_k_battery()) is None
