"""CPU fp64 oracle for the group-masked linear layer (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg use this
package.  The GPU library never imports, links or calls it, and it shares no
code with the GPU library.
"""
from .groupmask_oracle import *  # noqa: F401,F403
