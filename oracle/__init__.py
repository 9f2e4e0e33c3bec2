"""Float64 CPU oracle for the FDC/FDP layer hot path (Goh, Chen and Lim, arXiv 2106.12736).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code, tables or
helpers with the HIP library; both sides receive the same seeded inputs.

The oracle is plain, slow and written to be checked by eye against the paper:

* ``dft``   -- the 2-D real DFT and its inverse written out as matrix products
               of explicit DFT matrices (section 2.4.1.1, Eq. 4), plus their
               adjoints under the real inner product.
* ``fdc``   -- Channel Independent Convolution (Eq. 5, Algorithm 1), the RFFT
               shift and the frequency-domain pooling crop (section 2.4.2),
               convolution-artifact handling (section 2.4.1.3), the Full FDC
               layer (Algorithm 2, with the convolution-over-volume sum of Eq. 2
               done per frequency bin) and the backward pass of each, composed
               step by step in reverse.
* ``conv``  -- brute-force spatial convolutions (Eq. 1, Eq. 2 and the circular
               convolution the convolution theorem refers to), used to pin the
               oracle against a computation that involves no transform at all.
* ``classifier`` -- the FDCNN head of section 2.5.1 (ReLU, a fully connected
               layer, softmax cross-entropy) and the Adam step of section 3.1.

Every function works in float64 (complex128 for spectra).  Pins: see the
``-m "not gpu"`` tests in ``tests/test_oracle_*.py``.  No oracle function is
"parity unpinned".
"""

from . import classifier, conv, dft, fdc  # noqa: F401
