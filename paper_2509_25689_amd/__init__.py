"""MI355X-native forward pass of a pruned, mixed-precision, block-quantized
Mixture-of-Experts layer (arXiv 2509.25689's compressed DeepSeek MoE block).

``paper_2509_25689_amd.moeq`` is the Python binding of the HIP library
(``libmoeq.so``, C interface in ``include/moeq.h``); ``build`` compiles it."""
