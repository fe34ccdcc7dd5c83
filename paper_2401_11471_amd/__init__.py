"""Row-centric CNN training (LR-CNN, arXiv 2401.11471) for AMD MI355X.

The product is the HIP library ``liblrcnn.so`` with the C ABI of
``include/lrcnn.h``; ``lrcnn`` is its ctypes binding (same names) and
``device`` arranges torch device tensors for it.
"""
