"""Seeded synthetic inputs for the SAGIPS single-rank step.

This package holds shapes and seeded draws (numpy PCG64 streams): the workload
definitions (the step's, the bootstrap draw's and the ensemble's) and
generators for the parameter batches theta, the discriminator and generator
weights and the generator-network noise.  None of the hot path's steps is here
(no Philox, no sampler, no discriminator, no pathwise derivative, no
reduction), so the CPU oracle and the HIP path take the same inputs from here
without sharing any of that code.

The one computation here is input preparation: the small-batch workload's
theta is the output of a fixed 16-64-64-4 LeakyReLU network on N(0,1) noise,
evaluated once in float64 and rounded to float32 (theta_from_generator).  theta
is the step's input, so both sides receive the same rounded values and nothing
of that network is compared.  It is not the library's generator (a different
shape, 6-128-128-128-128-6, whose oracle is oracle/generator.py).
"""
from .configs import CONFIGS, Workload, get  # noqa: F401
from .gen import (make_inputs, theta_uniform, theta_from_generator, xavier_mlp,  # noqa: F401
                  generator_stack, noise)
