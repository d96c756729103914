"""Float64 CPU oracle for the Free Energy Mixer read (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import anything from this package.  The product path (the HIP
library and its Python binding) never imports, calls or links it, and the
oracle shares no code with the product path.
"""

from .fem_oracle import (  # noqa: F401
    elu_plus_one,
    softmax_prior_rows,
    linear_prior_rows,
    free_energy_read,
    expectation_read,
    ltl_read,
    fem_softmax_ltl,
    fem_softmax,
    fem_softmax_grads,
    fem_softmax_encoder,
    fem_softmax_decode,
    softmax_prior_all,
    fem_linear,
    fem_linear_recurrent,
    fem_gla,
    fem_gla_recurrent,
    rope,
    gla_features,
    posterior,
)
