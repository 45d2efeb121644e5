"""MI355X-native NOBLE-CosNet linear layer (arXiv 2603.06492).

The compute path is libnoble.so: hand-written HIP kernels for gfx950 behind
the C ABI in include/noble.h.  ``paper_2603_06492_amd.noble`` is its Python
binding (argument marshalling only); ``paper_2603_06492_amd.inputs`` holds the
seeded synthetic input recipe.
"""
