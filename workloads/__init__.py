"""Seeded synthetic inputs for the SAGIPS single-rank step.

This package holds only shapes and seeded draws (numpy PCG64 streams): the
workload definitions (the step's, the bootstrap draw's and the ensemble's) and
generators for the parameter batches theta, the discriminator and generator
weights and the generator-network noise.  It contains none of
the step's arithmetic (no Philox, no sampler, no discriminator), so both the
CPU oracle and the HIP path can take their inputs from here without sharing
any of the method's code.
"""
from .configs import CONFIGS, Workload, get  # noqa: F401
from .gen import (make_inputs, theta_uniform, theta_from_generator, xavier_mlp,  # noqa: F401
                  generator_stack, noise)
