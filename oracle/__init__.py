"""Float64 CPU oracle of the RoleSub hot path.

TEST INFRASTRUCTURE. Only the test suite, the smoke check and the benchmark's
CPU-baseline leg may import this package. The product path (librolesub and
its Python binding) never imports, calls or links anything here, and this
package imports nothing from the product.
"""
from .rolesub_oracle import *  # noqa: F401,F403
