"""MI355X-native paged translate-gather-pack for a decoupled VLM training pool.

The product is ``libflowpool.so`` (HIP kernels for gfx950 behind a C ABI,
declared in include/flowpool.h) and its thin ctypes binding
``paper_2606_23087_amd.flowpool``. Importing this package loads nothing;
``paper_2606_23087_amd.flowpool`` loads the library and fails loudly if it
has not been built.
"""
