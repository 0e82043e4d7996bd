"""CPU oracle for the SAGIPS single-rank step (test infrastructure only).

A plain, slow, float64 statement of what the step computes, written from the
paper (Sec. II problem statement, Sec. III GAN optimiser, Sec. V-A loop-closure
settings and its inverse-CDF sampler) and from the stated workload choices
(Philox4x32-10 counter-based draws, a Kumaraswamy inverse CDF, a LeakyReLU
discriminator with a BCE loss).

Only the test-suite, the smoke check and the CPU-baseline leg of the benchmark
may import this package.  It shares no code with the HIP library and imports
nothing from it.

Parity status per function (what pins it, see tests/test_oracle_*.py):
  philox4x32_10      pinned: bit-exact against an independent open-source
                     implementation compiled from source (PyTorch ATen).
  uniform            pinned: exact-arithmetic identities.
  kumaraswamy_icdf   pinned: CDF round trip, a=b=1 identity, Beta(1,b) and
                     Beta(a,1) special cases (scipy), median, moments.
  pathwise           pinned: finite differences, chain-rule form, signs,
                     expectation identities (digamma), theta=1 closed form.
  features_hd8       pinned: definition checks (log features vs values).
  mlp forward/back   pinned: finite differences, torch float64 autograd,
                     zero-last-layer and logistic-regression special cases.
  bce                pinned: closed values at z=0, derivative identity.
  bf16 emulation     pinned: RNE rounding against torch's bfloat16 cast;
                     the bf16 discriminator against torch autograd with
                     straight-through rounding at the same points.
  kink variants      pinned: torch autograd where no unit is near the kink,
                     one-sided finite differences at an exact kink.
  features_proxy2    pinned: Jacobian by finite differences, the means and
                     the covariance of the two observables against the
                     closed-form Kumaraswamy moments, the whole step's
                     dL/dtheta by finite differences.
  generator          pinned: forward against torch float64 modules,
                     backward against torch autograd and finite
                     differences.
  ensemble response  pinned: M = 1 and identical members (sigma = 0), the
                     M = 2 closed form |G1 - G2| / 2, numpy's population
                     standard deviation, member-order invariance.
  adam_step          pinned: torch.optim.Adam (float64) over several steps,
                     the first step's closed form lr g / (|g| + eps).
  gan_step           pinned: the generator gradient by finite differences
                     through generator, sampler, pipeline and discriminator;
                     lr = 0 leaves the parameters and sets the moments to
                     (1 - beta) g, (1 - beta2) g^2; both networks move
                     against their gradients.
  bootstrap          pinned: row ranges, the power-of-two case as a bit
                     shift, the with-replacement statistics (unique
                     fraction 1 - (1 - 1/n)^m, per-row counts binomial),
                     step and seed independence.
"""
from .philox import philox4x32_10, event_words  # noqa: F401
from .sampler import (uniform_from_words, kumaraswamy_icdf, kumaraswamy_cdf,  # noqa: F401
                      pathwise, sample, features_hd8, features_hd8_jacobian,
                      features_proxy2, features_proxy2_jacobian)
from .mlp import mlp_forward, bce_losses, disc_fwd_bwd, round_bf16, input_grad_kink_variants  # noqa: F401
from .step import param_grad, quadratic_critic, run_step  # noqa: F401
from .bootstrap import bootstrap, bootstrap_indices, bootstrap_row_order, STREAM_BOOTSTRAP  # noqa: F401
from .optim import adam_step  # noqa: F401
from .gan import gan_step, initial_state  # noqa: F401
from .generator import G_WIDTHS, generator_forward, generator_backward, ensemble_response, residual  # noqa: F401
