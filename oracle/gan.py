"""One GAN training step of the loop-closure test, end to end (test infrastructure).

Sec. III and Sec. V: the generator maps noise to parameters theta, the
pipeline samples events from theta and turns them into observables, the
discriminator is trained on them against reference events (Sec. IV-B: a
bootstrapped sub-sample of the rank's data) and the generator is trained
through the discriminator's response.  Readings (the paper is silent):
  * both gradients come from the same discriminator, before either update;
    the discriminator is then updated, and the generator (Sec. IV-B: the
    discriminator is updated right away, the generator's gradient travels);
  * the optimiser is Adam (see optim.py) with the learning rates of Sec. V-A;
  * step t (from 1) samples its fake events with counter base (t - 1) * N,
    so no event is drawn twice, and draws its reference batch as bootstrap
    step t.
"""
from __future__ import annotations

import numpy as np

from .bootstrap import bootstrap
from .generator import generator_backward, generator_forward
from .optim import adam_step
from .step import run_step


def gan_step(state: dict, noise, pool, t: int, E: int, fake_seed: int, boot_seed: int,
             lr_g: float = 1e-5, lr_d: float = 1e-4, slope: float = 0.2, features: str = "proxy2") -> dict:
    """state: G_W, G_b, D_W, D_b (lists of arrays) and their Adam moments
    G_m, G_v, D_m, D_v (lists in the order W0, b0, W1, b1, ...).  Returns the
    new state and the step's intermediates."""
    k = noise.shape[0]
    N = k * E
    theta = generator_forward(state["G_W"], state["G_b"], noise, slope)
    real, _ = bootstrap(pool, N, boot_seed, t)
    r = run_step(theta, E, fake_seed, state["D_W"], state["D_b"], real, features=features, slope=slope,
                 counter_base=(t - 1) * N)
    gW, gb = generator_backward(state["G_W"], state["G_b"], noise, r["dL_dtheta"], slope)

    def update(Ws, bs, dWs, dbs, ms, vs, lr):
        P, G = [], []
        for W, b, dW, db in zip(Ws, bs, dWs, dbs):
            P += [W, b]
            G += [dW, db]
        out_p, out_m, out_v = [], [], []
        for p, g, m, v in zip(P, G, ms, vs):
            p2, m2, v2 = adam_step(p, g, m, v, t, lr)
            out_p.append(p2)
            out_m.append(m2)
            out_v.append(v2)
        return out_p[0::2], out_p[1::2], out_m, out_v

    new = dict(state)
    new["D_W"], new["D_b"], new["D_m"], new["D_v"] = update(state["D_W"], state["D_b"], r["dW"], r["db"],
                                                            state["D_m"], state["D_v"], lr_d)
    new["G_W"], new["G_b"], new["G_m"], new["G_v"] = update(state["G_W"], state["G_b"], gW, gb,
                                                            state["G_m"], state["G_v"], lr_g)
    return {"state": new, "theta": theta, "real": real, "loss_d": r["loss_d"], "loss_g": r["loss_g"],
            "dW_D": r["dW"], "db_D": r["db"], "dL_dtheta": r["dL_dtheta"], "dW_G": gW, "db_G": gb}


def initial_state(G_W, G_b, D_W, D_b) -> dict:
    """Parameters as float64 and zero Adam moments."""
    f = lambda xs: [np.asarray(x, dtype=np.float64) for x in xs]
    z = lambda Ws, bs: [np.zeros(np.shape(a)) for pair in zip(Ws, bs) for a in pair]
    return {"G_W": f(G_W), "G_b": f(G_b), "D_W": f(D_W), "D_b": f(D_b),
            "G_m": z(G_W, G_b), "G_v": z(G_W, G_b), "D_m": z(D_W, D_b), "D_v": z(D_W, D_b)}
