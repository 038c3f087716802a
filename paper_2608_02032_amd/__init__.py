"""DART hot path on AMD Instinct MI355X (gfx950): chunked SSD scan that keeps
the chunk state memories, state-memory attention with the gated residual, and
the single-token decode step, as hand-written HIP kernels behind a C ABI
(``include/dart.h``).  The Python functions here only marshal arguments."""
