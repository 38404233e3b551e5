"""CPU oracle for the int4-weight linear-projection path (test infrastructure).

Only the tests, the smoke check of the entry module and the ``cpu_baseline``
leg of the bench may import anything from this package; the product library
never does, and this package imports nothing from the product.
"""
from .qlinear_oracle import *  # noqa: F401,F403
from .qlinear_oracle import __all__  # noqa: F401
