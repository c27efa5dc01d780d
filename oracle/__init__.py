"""CPU oracle for Winograd convolution with CRT-built transforms (Barabasz & Gregg,
"Winograd Convolution for DNNs: Beyond linear polynomials", arXiv 1905.05233).

TEST INFRASTRUCTURE ONLY.  This package is the independent, slow, obviously
correct reference that the GPU library is checked against.  Only the test suite,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  The product path (``paper_1905_05233_amd`` and its native library)
never imports, links or calls anything here, and nothing here imports the
product package: the two share no code, tables or constants.

Modules
-------
polynomials  exact polynomial arithmetic over Q (Python ``fractions``), the
             remainder map R_m[.], vec(.), and the extended Euclidean algorithm
             (Section 2.1, eq. (1)).
plan         Algorithm 1 (G^W, A^W) and Algorithm 2 (B^W) in exact rationals,
             with the inner Toom-Cook sub-algorithm for degree-d moduli
             (Section 2.2), the multiplication ratio (Section 2.3, Table 1) and
             the exact identities the construction must satisfy.
fp           IEEE rounding emulation: exact rational -> fp32 RNE, fp32 -> fp16
             and fp32 -> bf16 RNE (Section 3.2 simulates fp16/bf16 by casting).
conv         direct convolution (exact rational and fp64), 2D Winograd by the
             matrix-exchange form of eq. (2) in exact rationals, and the
             same-algorithm, same-dtype rounding-emulated Winograd; rel-L2.

Parity status: every function here is pinned by a ``-m "not gpu"`` test
against values the paper prints, published Toom-Cook matrices, closed-form
identities, library routines or brute force, except the random-data error
magnitudes of Fig. 3, whose values are not in the paper text ("parity
unpinned" for magnitudes; only their direction is checked).
"""
