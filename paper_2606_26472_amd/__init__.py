"""EpiKV eviction step on AMD Instinct MI355X (gfx950).

The hot path (score -> rolling z-score -> top-K select -> paged compaction)
is a set of hand-written HIP kernels behind the C ABI in include/epikv.h,
built into libepikv.so.  `epikv` is its Python binding.
"""
__all__ = ["epikv"]
