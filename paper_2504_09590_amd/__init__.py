"""MI355X-native bidirectional paged attention for mixed RT/BE serving batches.

The compute lives in libbros_attn.so (hand-written HIP for gfx950 behind a C ABI,
declared in include/bros_attn.h). `paper_2504_09590_amd.bros` is the thin ctypes
binding; `paper_2504_09590_amd.workload` draws seeded synthetic batches.
Submodules are imported on demand so that the input generator can be used
without loading the GPU library.
"""
__all__ = ["bros", "workload"]
