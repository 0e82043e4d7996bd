"""The GAN training loop of the loop-closure test on one GPU (paper Sec. III,
Sec. IV-B, Sec. V), sequenced from the library's calls: every step is six
launches' worth of library work on the context's stream and no host
synchronisation.

Step t (counting from 1):
  1. theta = 1 + softplus(G(noise_t))                       sagips_gen_forward
  2. reference batch = bootstrap step t of the data pool     sagips_bootstrap
  3. events from theta (counter base (t-1) N), observables, discriminator,
     BCE, backward: dL_D/dW_D and dL_G/dtheta                sagips_disc_fwd_bwd
  4. dL_G/dW_G from dL_G/dtheta                             sagips_gen_backward
  5. Adam on the discriminator (lr 1e-4), then on the generator (lr 1e-5)
                                                             sagips_adam_step
Both gradients come from the discriminator before its update.  The normalised
residual r_hat = (theta* - p_hat) / theta* of the generator's mean prediction
tracks convergence (sagips_ensemble_response with one member).
"""
from __future__ import annotations

from typing import List, Optional, Sequence

from . import FEAT_PROXY2, Context


class GanLoop:
    """Generator (one member, parameters updated in place), discriminator and the
    reference data pool, all device tensors owned by the caller; the loop owns
    the step's buffers and the Adam moments."""

    def __init__(self, ctx: Context, G_W: Sequence, G_b: Sequence, D_W: Sequence, D_b: Sequence, pool,
                 k: int, events_per_theta: int, fake_seed: int = 0, boot_seed: int = 5,
                 lr_g: float = 1e-5, lr_d: float = 1e-4, slope: float = 0.2, features: int = FEAT_PROXY2):
        import torch
        self.ctx = ctx
        self.G_W, self.G_b, self.D_W, self.D_b = list(G_W), list(G_b), list(D_W), list(D_b)
        self.pool = pool
        self.k, self.E = int(k), int(events_per_theta)
        self.N = self.k * self.E
        self.fake_seed, self.boot_seed = fake_seed, boot_seed
        self.lr_g, self.lr_d, self.slope, self.features = lr_g, lr_d, slope, features
        self.t = 0
        dev = pool.device
        n_out = self.G_W[-1].shape[0]
        f32 = dict(dtype=torch.float32, device=dev)
        self.theta = torch.empty((1, self.k, n_out), **f32)
        self.real = torch.empty((self.N, pool.shape[1]), **f32)
        self.outs = {"loss_d": torch.empty(1, **f32), "loss_g": torch.empty(1, **f32),
                     "dW": [torch.empty_like(w) for w in self.D_W], "db": [torch.empty_like(v) for v in self.D_b],
                     "dLg_dtheta": torch.empty((self.k, n_out), **f32)}
        self.gW = [torch.empty_like(w) for w in self.G_W]
        self.gb = [torch.empty_like(v) for v in self.G_b]
        self._d_params = self._interleave(self.D_W, self.D_b)
        self._g_params = self._interleave(self.G_W, self.G_b)
        self._d_grads = self._interleave(self.outs["dW"], self.outs["db"])
        self._g_grads = self._interleave(self.gW, self.gb)
        self.D_m = [torch.zeros_like(p) for p in self._d_params]
        self.D_v = [torch.zeros_like(p) for p in self._d_params]
        self.G_m = [torch.zeros_like(p) for p in self._g_params]
        self.G_v = [torch.zeros_like(p) for p in self._g_params]

    @staticmethod
    def _interleave(Ws: List, bs: List) -> List:
        return [t for pair in zip(Ws, bs) for t in pair]

    def step(self, noise) -> None:
        """One training step on the noise batch [k][in] (a device tensor)."""
        self.t += 1
        c = self.ctx
        c.gen_forward(self.G_W, self.G_b, noise, slope=self.slope, out=self.theta)
        c.bootstrap(self.pool, self.N, self.boot_seed, self.t, out=self.real)
        theta = self.theta[0]
        c.disc_fwd_bwd(self.D_W, self.D_b, self.real,
                       fake_source=dict(theta=theta, events_per_theta=self.E, seed=self.fake_seed,
                                        counter_base=(self.t - 1) * self.N),
                       features=self.features, slope=self.slope, want_logits=False, want_dx=False,
                       outputs=self.outs)
        c.gen_backward(self.G_W, self.G_b, noise, self.outs["dLg_dtheta"], slope=self.slope, dW=self.gW, db=self.gb)
        c.adam_step(self._d_params, self._d_grads, self.D_m, self.D_v, self.t, self.lr_d)
        c.adam_step(self._g_params, self._g_grads, self.G_m, self.G_v, self.t, self.lr_g)

    def residual(self, noise, theta_star) -> dict:
        """p_hat (mean prediction over the noise batch) and r_hat = (theta* - p_hat) / theta*."""
        return self.ctx.ensemble_response(self.G_W, self.G_b, noise, p_true=theta_star, slope=self.slope)


def loop_closure(ctx: Context, steps: int, report_every: int = 1000, k: int = 1024, events_per_theta: int = 100,
                 seed: int = 0, log: Optional[callable] = None) -> List[dict]:
    """Train the paper-shape GAN (generator 6-128-128-128-128-6, discriminator
    2-128-128-128-128-1 on the two observables) against reference data drawn at
    theta* = (2, 5, 1.5, 3, 3, 2), recording r_hat every report_every steps."""
    import numpy as np
    import torch

    from workloads import gen

    dev = "cuda:%d" % ctx.device
    ts = torch.tensor([[2.0, 5.0, 1.5, 3.0, 3.0, 2.0]], device=dev)
    N = k * events_per_theta
    pool = ctx.sample_events(ts, 2 * N, seed + 1)                 # the rank's reference data: 2 N events
    GW, Gb = gen.generator_stack((6, 128, 128, 128, 128, 6), 1, seed + 21)
    DW, Db = gen.xavier_mlp((2, 128, 128, 128, 128, 1), seed + 2)
    G_W = [torch.tensor(w[0], device=dev) for w in GW]
    G_b = [torch.tensor(v[0], device=dev) for v in Gb]
    D_W = [torch.tensor(w, device=dev) for w in DW]
    D_b = [torch.tensor(v, device=dev) for v in Db]
    loop = GanLoop(ctx, G_W, G_b, D_W, D_b, pool, k, events_per_theta, fake_seed=seed, boot_seed=seed + 5)
    rng = np.random.default_rng(seed + 22)
    eval_noise = torch.tensor(rng.standard_normal((k, 6)).astype(np.float32), device=dev)
    history = []
    for s in range(1, steps + 1):
        noise = torch.tensor(rng.standard_normal((k, 6)).astype(np.float32), device=dev)
        loop.step(noise)
        if s % report_every == 0 or s == steps:
            r = loop.residual(eval_noise, ts[0])
            rec = {"step": s, "loss_d": loop.outs["loss_d"].item(), "loss_g": loop.outs["loss_g"].item(),
                   "p_hat": r["p_hat"].tolist(), "r_hat": r["r_hat"].tolist()}
            history.append(rec)
            if log:
                log(rec)
    return history


if __name__ == "__main__":
    import argparse
    import json

    ap = argparse.ArgumentParser(description="loop-closure run of the paper-shape GAN on one GPU")
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--report-every", type=int, default=200)
    ap.add_argument("--seed", type=int, default=0)
    a = ap.parse_args()
    ctx = Context(0)
    loop_closure(ctx, a.steps, a.report_every, seed=a.seed, log=lambda r: print(json.dumps(r), flush=True))
    ctx.close()
