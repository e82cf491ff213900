"""CPU oracle for the SAMD quantized-convolution path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg may import, call, link or run anything in this package.
The GPU library (``paper_1809_10572_amd``) never imports it, and the two share no
code: only the seeded input generators in ``samd_workloads`` serve both.

* ``reference`` - the plain definition of every result (``ref.c``, int64): the
  packed storage format, valid-mode 1-D convolution, the DNN 2-D convolution
  (cross-correlation with batch, stride and zero padding), ReLU + requantisation.
  This is what GPU parity is measured against.
* ``samd_model`` - the paper's SAMD routines themselves (lane masks, lane-wise add,
  subtract and multiply, vector scale, convolution by long multiplication, signed
  sign-extension and the underflow fix-up), on Python integers, with the readings
  of the paper's ambiguous passages.  It checks the method, not the GPU.
"""
