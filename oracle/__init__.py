"""CPU oracle of the fused N-model training step -- test infrastructure only.

Only tests, the smoke check and the benchmark's CPU-baseline leg import this
package; the library's compute path never does.
"""
from .oracle import *  # noqa: F401,F403
