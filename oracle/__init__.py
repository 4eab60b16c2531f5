"""CPU oracle of the paged-KV hot path (append, prefix-reuse prefill
attention, paged decode attention), in float64.

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check of the
package entry file, and by the CPU-baseline leg of bench.py.  The product
path (the HIP library and its Python binding) never imports it, and this
package never imports the product path.

Modules:
  formats  bfloat16 and fp8 E4M3FN encode/decode from their definitions
  paged    append, gather, dense softmax attention, LSE merge (NumPy fp64)
  brute    pure-Python loops for tiny inputs, used to pin `paged`
  ttl      the TTL control plane (Eq. 2, cold start, eta, Alg. 1) in plain Python
"""
from . import brute, formats, paged, ttl  # noqa: F401
