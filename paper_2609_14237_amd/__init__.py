"""MI355X-native operator-level-disaggregated (ODS) decode hot path.

The HIP library (libods.so) exports the C ABI of include/ods.h; ``binding``
mirrors it with ctypes and ``runtime`` packs PyTorch device tensors into its
structs. Submodules are imported lazily so that building does not require a
built library.
"""
__all__ = ["binding", "runtime", "build"]
