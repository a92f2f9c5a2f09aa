"""MI355X-native hot path of DIGEST (arXiv 2206.00057): one graph partition's
GCN layer forward/backward with stale halo rows, plus push/pull, as a C-ABI
HIP library (``csrc/``) with a thin ctypes binding (``digest``)."""
__version__ = "0.1.0"
