"""CPU fp64 oracle for Higher-order Linear Attention (HLA).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import, call, link or run anything in this
package.  The GPU product path never routes through it and shares no code with
it: the two meet only on seeded inputs produced by a generator module that
holds none of the method's arithmetic.

Modules
  hla2      second-order HLA (Sec. 3 and Sec. 4 of the paper): the plain
            definition, the serial online recurrence, the chunked associative
            scan and the masked semidirect product.
  hla3      third-order HLA (Sec. 7): the triple sum over the index set of
            Thm. 3, the streaming kernel (Alg. 3), the corrected-state
            recurrence, the operator (x)_3 and the chunk-parallel scan (Alg. 4).
  hla2_decay  second-order HLA with exponential decay (decay section and the
            decay-aware concatenation of Sec. 4).
  hla2_backward  gradients of the masked second-order HLA (the reverse scan
            of Sec. 4.2 written out), pinned against torch autograd.
  ahla      asymmetric second-order HLA (Sec. 6): the double sum, the
            streaming recurrence, (+)_AHLA and the chunked scan.
  hla2_ref.c, hla2_decay_ref.c, hla3_ref.c, ahla_ref.c  the serial
            recurrences in plain C (fp64), used to
            time the oracle on host cores and to check large cases quickly.
  native    ctypes loader for the compiled C oracle.
"""
