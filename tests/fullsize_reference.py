"""Test helper: the discriminator step's reduced outputs (dW, db of every layer,
both losses) at the full sizes of the bf16 workloads, where the CPU oracle would
take tens of minutes.

It restates the oracle's two evaluations (oracle/mlp.py: the float64 network of
Sec. V-A with the BCE objective of Sec. II-B.2, and the same network evaluated
at the bf16 rounding points) in torch float64, so that the matrix products run
as float64 GEMMs on whatever device the inputs are put on, a chunk of events at
a time.  Each event's seeds e_D = dL_D/dz and e_G depend only on its own logit
and the batch sizes, so one forward and backward pass per chunk accumulates the
sums exactly as the whole batch would (up to float64 summation order).

It shares nothing with the HIP library; tests/test_fullsize_reference.py pins
it to the oracle on small batches (CPU, float64)."""
import torch

F64 = torch.float64


def round_bf16(t):
    """Round to the nearest bfloat16 (ties to even) via float32, as the oracle does."""
    return t.to(torch.float32).to(torch.bfloat16).to(F64)


def _leaky(t, s):
    return torch.where(t > 0, t, s * t)


def _leaky_grad(t, s):
    return torch.where(t > 0, torch.ones_like(t), torch.full_like(t, s))


def _softplus(t):
    return torch.clamp(t, min=0.0) + torch.log1p(torch.exp(-torch.abs(t)))


def _sigmoid(t):
    return 0.5 * (1.0 + torch.tanh(0.5 * t))


def reduced_outputs(W, b, fake_in, real_in, slope=0.2, bf16=False, device="cpu", chunk=1 << 18,
                    progress=None):
    """dW, db (lists of float64 tensors on `device`), loss_d, loss_g and, for the
    float64 evaluation, the per-entry sums of |terms| dW_cond and db_cond.

    W, b: the network (torch.nn.Linear layout), any array type.  fake_in,
    real_in: the two batches' input features, [N][F] float64 (numpy or torch);
    they are moved to `device` one chunk at a time."""
    n = len(W)
    Wd = [torch.as_tensor(w, dtype=F64).to(device) for w in W]
    bd = [torch.as_tensor(v, dtype=F64).to(device) for v in b]
    rnd = round_bf16 if bf16 else (lambda t: t)
    # hidden-to-hidden weights are the ones rounded (layers 1 .. n-2)
    Wq = [rnd(w) if 0 < l < n - 1 else w for l, w in enumerate(Wd)]
    dW = [torch.zeros_like(w) for w in Wd]
    db = [torch.zeros_like(v) for v in bd]
    cW = [torch.zeros_like(w) for w in Wd]
    cb = [torch.zeros_like(v) for v in bd]
    nf, nr = len(fake_in), len(real_in)
    sums = {"sp_f": 0.0, "sp_neg_f": 0.0, "sp_neg_r": 0.0}
    for fake, batch in ((True, fake_in), (False, real_in)):
        N = nf if fake else nr
        for r0 in range(0, N, chunk):
            h0 = torch.as_tensor(batch[r0:r0 + chunk], dtype=F64).to(device)
            hs = [h0]
            for l in range(n - 1):
                hs.append(rnd(_leaky(hs[-1] @ Wq[l].T + bd[l], slope)))
            z = (hs[-1] @ Wd[-1].T + bd[-1])[:, 0]
            if fake:
                e = _sigmoid(z) / nf
                sums["sp_f"] += float(_softplus(z).sum())
                sums["sp_neg_f"] += float(_softplus(-z).sum())
            else:
                e = -_sigmoid(-z) / nr
                sums["sp_neg_r"] += float(_softplus(-z).sum())
            dW[n - 1] += (e[:, None] * hs[n - 1]).sum(dim=0)[None, :]
            db[n - 1] += e.sum().reshape(1)
            cW[n - 1] += (e.abs()[:, None] * hs[n - 1].abs()).sum(dim=0)[None, :]
            cb[n - 1] += e.abs().sum().reshape(1)
            d = rnd(Wd[n - 1][0][None, :] * _leaky_grad(hs[n - 1], slope))   # unit-seed signal
            for l in range(n - 2, -1, -1):
                ed = e[:, None] * d
                dW[l] += (rnd(ed) if l > 0 else ed).T @ hs[l]
                db[l] += ed.sum(dim=0)
                cW[l] += ed.abs().T @ hs[l].abs()
                cb[l] += ed.abs().sum(dim=0)
                if l > 0:
                    d = rnd((d @ Wq[l]) * _leaky_grad(hs[l], slope))
            if progress:
                progress(fake, r0 + len(h0), N)
    loss_d = sums["sp_neg_r"] / nr + sums["sp_f"] / nf
    loss_g = sums["sp_neg_f"] / nf
    return {"dW": dW, "db": db, "dW_cond": cW, "db_cond": cb, "loss_d": loss_d, "loss_g": loss_g}
