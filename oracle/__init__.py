"""Q-Delta CPU oracle.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call,
link or execute this package: only the test suite, the smoke check and the
benchmark's CPU-baseline leg use it.  It shares no code with the HIP kernels.

Modules
-------
recurrent  the plain fp64 token-by-token recurrence of the paper's final
           update rule (Sec. 3.3, Eq. (qdelta_decay)) and its exact gradient
           by back-propagation through time, in C (``qdref.c``), threaded over
           independent (sequence, head) units.
chunk      an fp64 numpy rendering of the chunkwise form (Sec. 3.3
           "Chunkwise parallel form", App. D.1 WY representation and App. D.2
           UT transform) for any chunk size, with its backward.  It checks the
           algebra that the GPU path follows; it is not the parity reference.
exact      rational-arithmetic brute force on tiny inputs: the dense
           transition-matrix product and the value-decomposition closed form
           of Sec. 3.1 (Eqs. (general_recurrence), (state_decomp),
           (b_recursion)).
deltanet   the DeltaNet and GatedDeltaNet rules of Sec. 2.1 written out
           separately, for the lambda = 0 reduction check.
"""
