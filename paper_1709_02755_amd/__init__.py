"""MI355X-native Simple Recurrent Unit (SRU) layer: HIP kernels behind a C ABI.

The compute lives in ``libsru.so`` (built from ``csrc/``); ``sru`` is the thin
ctypes binding.  Importing this package loads nothing; ``sru.lib()`` loads the
library on first use and fails loudly if it is missing.
"""

__all__ = ["sru", "workloads"]
