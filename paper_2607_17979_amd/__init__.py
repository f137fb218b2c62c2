"""MI355X (gfx950) Gated DeltaNet decode and varlen prefill: a C-ABI HIP library
and a thin ctypes binding.  ``paper_2607_17979_amd.gdn`` holds the binding;
``workloads`` the seeded synthetic inputs.  Importing the package does not load
the native library; the first call into ``gdn`` does, and fails loudly if it has
not been built."""
