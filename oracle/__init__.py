"""fp64 CPU oracle of the Llama-style decoder block (forward and backward).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the CPU
baseline leg of the benchmark.  The library's product path never imports or
calls anything here, and this package imports nothing from the product
package.  Every function is a plain float64 numpy definition; see block.py.
"""
from . import block  # noqa: F401
