"""MI355X (gfx950) hot path of SAECache's semantic-aware prefix-cache eviction.

libsae.so (HIP) implements the C ABI of include/sae.h; `api` is its Python
binding with the same names, `pool` holds device-buffer helpers.  Importing
the package does not load the library; the first call does, and fails loudly
when it is not built.
"""
