"""MI355X-native parallelised StackLSTM step (Ding & Koehn, 2019).

The compute path lives in the HIP library built from ``csrc/`` and is reached
through ``paper_1904_03409_amd.stacklstm`` (a thin ctypes binding).
``paper_1904_03409_amd.workloads`` draws the seeded synthetic inputs.
"""
__all__ = ["workloads", "stacklstm"]
