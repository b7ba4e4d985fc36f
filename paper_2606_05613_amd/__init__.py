"""MI355X-native bucket-level gradient-conflict resolution.

The HIP library (libbkmoo.so, C ABI in include/bkmoo.h) is the product; the
`bkmoo` submodule is its Python binding.  Build with
`python -m paper_2606_05613_amd.build`.
"""
