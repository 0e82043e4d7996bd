"""The bf16 reading of the medium and higher-dim workloads, checked on the CPU with
the oracle alone: how far the bf16-operand network (hidden weights, activations and
backward signals rounded to bfloat16, everything else exact) is from the float64
network, per output tensor, and which rounding point causes it.

These facts decide what the GPU parity tests can ask of the bf16 path against the
float64 definition (network of Sec. V-A, objective of Sec. II-B.2):
  * the second rounding of the scaled weight-gradient operand e_D * delta is
    immaterial: the bf16-point oracle is the plain bf16-operand network;
  * the dW / db deviations come from rounding the weights (a hi + lo split of the
    weights removes them);
  * the dL_G/dx deviation comes from rounding the activations, which moves hidden
    units across the LeakyReLU kink; no evaluation with bf16 activations meets the
    2e-2 bar there, while splitting weights and activations into two bf16 terms does.
"""
import numpy as np
import pytest

import oracle
from oracle.mlp import _disc_bf16, round_bf16
from workloads import gen, get
from workloads.configs import scaled

ident = lambda a: np.asarray(a, dtype=np.float64)     # noqa: E731


def split2(a):
    """Two bf16 terms hi + lo of a value (about 16 significant bits)."""
    hi = round_bf16(a)
    return hi + round_bf16(np.asarray(a, dtype=np.float64) - hi)


def nw(a, r):
    a = np.asarray(a, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    return float(np.linalg.norm((a - r).ravel()) / np.linalg.norm(r.ravel()))


@pytest.fixture(scope="module")
def medium_case():
    w = scaled(get("medium"), 4, 1024)
    inp = gen.make_inputs(w)
    fake = oracle.sample(inp["theta"], w.events_per_theta, w.fake_seed)
    real = oracle.sample(inp["theta_star"], w.n_events, w.real_seed)
    ref = oracle.disc_fwd_bwd(inp["W"], inp["b"], fake, real)

    def run(rw, ra, rd, re):
        return _disc_bf16(inp["W"], inp["b"], fake, real, 0.2, rw, ra, rd, re)

    def dev(r):
        out = {k: nw(r[k], ref[k]) for k in ("logits_fake", "logits_real", "dLg_din")}
        out["loss_d"] = abs(r["loss_d"] - ref["loss_d"]) / ref["loss_d"]
        out["loss_g"] = abs(r["loss_g"] - ref["loss_g"]) / ref["loss_g"]
        for l in range(len(inp["W"])):
            out[f"dW{l}"] = nw(r["dW"][l], ref["dW"][l])
            out[f"db{l}"] = nw(r["db"][l], ref["db"][l])
        return out

    R = round_bf16
    runs = {"all": run(R, R, R, R), "no_e": run(R, R, R, ident), "W": run(R, ident, ident, ident),
            "A": run(ident, R, ident, ident), "Wsplit": run(split2, R, R, R),
            "WAsplit": run(split2, split2, R, R)}
    devs = {k: dev(v) for k, v in runs.items()}
    for k, v in devs.items():
        print(k, " ".join(f"{t}={x:.1e}" for t, x in v.items()))
    return inp, runs, devs


def test_second_rounding_of_the_scaled_signal_is_immaterial(medium_case):
    inp, runs, devs = medium_case
    for l in range(len(inp["W"])):
        change = nw(runs["all"]["dW"][l], runs["no_e"]["dW"][l])
        assert change <= 0.15 * max(devs["all"][f"dW{l}"], 1e-12), (l, change)


def test_weight_rounding_causes_the_gradient_deviation(medium_case):
    inp, runs, devs = medium_case
    hidden = range(len(inp["W"]) - 1)          # every layer whose input gradient passes a bf16 weight
    for l in hidden:
        for t in (f"dW{l}", f"db{l}"):
            assert devs["W"][t] >= 0.75 * devs["all"][t], t
            assert devs["Wsplit"][t] <= 2e-2, t
    # the medium network's first-layer gradients miss the 2e-2 bar with bf16 weights
    assert devs["all"]["dW0"] > 2e-2


def test_activation_rounding_causes_the_input_gradient_deviation(medium_case):
    _, _, devs = medium_case
    assert devs["A"]["dLg_din"] > 5e-2          # bf16 activations alone: kinks crossed
    assert devs["Wsplit"]["dLg_din"] > 5e-2     # and splitting only the weights does not help
    assert devs["WAsplit"]["dLg_din"] <= 2e-2   # splitting both does
    # logits and losses stay far inside the bar at every rounding
    for k in ("logits_fake", "logits_real", "loss_d", "loss_g"):
        assert devs["all"][k] <= 2e-2, k
