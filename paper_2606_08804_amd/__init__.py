"""MI355X-native Q-Delta: chunkwise-parallel layer forward/backward and the
single-token recurrent update, as hand-written HIP kernels for gfx950 behind a
C ABI (``libqdelta.so``).  The Python layer here only marshals arguments."""
