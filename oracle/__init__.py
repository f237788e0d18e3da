"""CPU oracle for the parallelised StackLSTM step (test infrastructure only).

Only ``tests/``, the smoke check and the benchmark's CPU-baseline leg use this
package. The product path (``paper_1904_03409_amd``) never imports it.
"""
from .oracle import build, run, alg1, round_bf16, max_threads, OracleError  # noqa: F401
