"""MI355X (gfx950) implementation of the Free Energy Mixer read.

``binding`` holds the Python side of the C ABI declared in ``include/fem.h``
(``fem_softmax_fwd``, ``fem_softmax_fwd_ex``, ``fem_softmax_fwd_train``,
``fem_softmax_bwd``, ``fem_softmax_gated_fwd``,
``fem_softmax_decode``, ``fem_linear_fwd``, ``fem_gla_fwd``, ``fem_status_str``); ``inputs``
draws the seeded synthetic workloads.  Nothing is imported eagerly, so the
package can be imported on a machine without a GPU or a built library.
"""

__all__ = ["binding", "inputs"]
