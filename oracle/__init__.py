"""fp64 CPU oracle for exact non-causal multi-head scaled-dot-product attention.

TEST INFRASTRUCTURE ONLY. Only the test suite, the package entry point's smoke
check and the benchmark's CPU-baseline leg may import this package. The HIP
path never imports it, and it imports nothing from the HIP path.

Pinning: every function here is checked by the CPU tests against closed forms
(identical keys, a dominant key, N=1, all-ones V), invariants (permutation
equivariance, linearity in V, head independence, gradient identities), central
finite differences of the forward, an independent pure-Python evaluation of
the definition, and a library routine (PyTorch's CPU scaled-dot-product
attention with autograd) on small inputs. The paper itself prints no attention
values, so no pin comes from printed numbers.
"""
from .attention import (  # noqa: F401
    decode_bf16,
    fp32_scale,
    forward,
    forward_backward,
    forward_backward_rows,
    query_rows,
    row_statistics,
    key_rows,
)
from .segments import merge, segment_backward  # noqa: F401
from . import ulysses  # noqa: F401
from . import aggregation  # noqa: F401
from . import naive  # noqa: F401
