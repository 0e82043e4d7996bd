"""The workloads, networks and training loop against the settings the paper prints
(tests/golden/paper_settings.json, each value with the place it is stated)."""
import inspect
import json
import os

import oracle
from workloads import get

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_settings.json")))


def _g(key):
    return GOLDEN[key]["value"]


def _params(widths):
    return sum(i * o + o for i, o in zip(widths[:-1], widths[1:]))


def test_paper_shape_step():
    w = get("paper")
    assert w.n_theta == _g("predicted_parameter_samples")
    assert w.events_per_theta == _g("events_per_parameter_sample")
    assert w.n_events == _g("discriminator_batch_size")
    assert 2 * w.d == _g("parameters_per_sample")
    assert w.widths[0] == _g("observables") and w.features == "proxy2"
    assert _params(w.widths) == _g("discriminator_trainable_parameters")


def test_training_step_shape():
    t = get("train")
    assert t.k * t.events_per_theta == _g("discriminator_batch_size")
    assert _params(t.g_widths) == _g("generator_trainable_parameters")
    assert _params(t.d_widths) == _g("discriminator_trainable_parameters")
    assert t.g_widths[-1] == _g("parameters_per_sample")
    assert tuple(oracle.G_WIDTHS) == tuple(t.g_widths)


def test_learning_rates():
    from paper_2407_00051_amd.gan import GanLoop
    for fn in (oracle.gan_step, GanLoop.__init__):
        sig = inspect.signature(fn)
        assert sig.parameters["lr_g"].default == _g("generator_learning_rate")
        assert sig.parameters["lr_d"].default == _g("discriminator_learning_rate")


def test_bootstrap_fraction():
    for name in ("bootstrap", "bootstrap_d3", "bootstrap_rows", "bootstrap_rows_d3"):
        b = get(name)
        assert b.n_out / b.n_data == _g("sub_sample_fraction")


def test_ensemble_size_is_one_the_paper_uses():
    e = get("ensemble")
    assert e.n_members in _g("ensemble_sizes")
    assert _params(e.widths) == _g("generator_trainable_parameters")
