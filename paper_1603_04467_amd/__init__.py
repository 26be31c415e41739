"""MI355X-native dense-layer training step (TensorFlow white paper, 2015).

Submodules: ``tfdense`` (binding of the libtfdense C ABI), ``step`` (the
training step as a sequence of library calls), ``workloads`` (seeded
synthetic inputs), ``build`` (hipcc build of the library).
"""
