"""Oracle: a plain, slow, obviously correct CPU implementation of the batched
Whisper-shaped ASR step and of the duration-aware waiting queue.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports it: only the
tests, the package's smoke check and the benchmark's CPU-baseline leg may.
It shares no code with the HIP library (no kernels, headers, tables or
helpers); the only thing both sides consume is the seeded input generators.

Floating point is float64 throughout (the paper fixes no precision).  Each
function names the passage of the paper, or the Whisper architecture the
paper serves, that it follows.
"""
