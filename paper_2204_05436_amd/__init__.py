"""MI355X-native hot path of the Hotline heterogeneous recommendation-training
pipeline (arXiv 2204.05436): hot-set profiling, popularity classification and
mu-batch partition, hot-slot remap, cold-row gather, and EmbeddingBag forward /
coalesced sparse-SGD backward, each a HIP kernel for gfx950 behind the C ABI in
include/hotline.h.  The HIP library is loaded lazily by `hotline`."""
