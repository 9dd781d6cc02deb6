"""MI355X-native implementation of one node's per-layer gradient
synchronisation in Poseidon (arXiv 1706.03292): sufficient-factor
reconstruction fused with SGD for fully-connected layers, parameter-server
aggregation with momentum SGD for all other layers, and the per-layer hybrid
communication choice between them.

The compute lives in ``libposeidon.so`` (hand-written HIP for gfx950 behind a
C ABI, declared in ``include/poseidon.h``); ``api`` is a thin ctypes binding
that only marshals PyTorch device tensors and streams into that ABI.
"""
