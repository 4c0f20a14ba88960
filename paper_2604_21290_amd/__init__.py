"""MI355X-native GraphLeap hot path: dilated kNN graph build, max-relative
graph convolution and the one-block lookahead schedule, as HIP kernels for
gfx950 behind a C ABI (libgraphleap.so).

Importing the package loads nothing; the library is opened on first use by
`paper_2604_21290_amd.api` and raises if it has not been built.
"""
__all__ = ["api", "inputs"]
