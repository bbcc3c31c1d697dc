"""MI355X-native KV-shared attention (KV-Pipe, arxiv 2608.15943).

The compute lives in the HIP library ``lib/libkvpipe.so`` behind the C ABI of
``include/kvpipe.h``; this package only marshals arguments (``binding``) and
builds the library (``build``).  Importing the package does not load the
library; ``binding.lib()`` does, and raises if it has not been built.
"""
from . import binding  # noqa: F401

__all__ = ["binding"]
