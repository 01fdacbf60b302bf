"""MI355X-native fused Indexer-TopK (LiteTopK) library.

The compute path is the HIP library ``liblitetopk.so`` (C ABI in
``include/litetopk.h``); ``litetopk`` is its Python binding and ``workloads``
draws seeded synthetic inputs. Importing the package does not load the
library; ``litetopk.load()`` does, and fails loudly if it is not built.
"""
__all__ = ["litetopk", "workloads"]
