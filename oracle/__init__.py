"""CPU oracle for the fused multi-shell Leech-lattice dequantize + matvec.

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow, obviously
correct reference that the GPU path is checked against.  Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  The product (``paper_2609_02652_amd`` and its HIP library) never
imports, calls or links anything here, and this package imports nothing from
the product: the two share no code, tables or helpers.  The seeded input
generator (``paper_2609_02652_amd.synth``) feeds both sides and holds none of
the decode or matvec arithmetic.

What it computes (paper §2.1 "What a Λ24 index is", §2.2 "Unfolding at load
time", §2.4 "Verification"):

* ``lattice``: the extended binary Golay code, Λ24 membership in the √8
  scaling, the shells of the ball Λ24(12), its 301 classes (magnitude
  multisets) and their sizes, the per-class level values.
* ``decode``: decoded fields (class id, gain bit, sign mask, per-coordinate
  magnitude level) -> integer lattice coordinates -> f64 weights, and the f64
  matvec ``y64 = W x`` with the two tolerance normalisations.

Everything is f64 or exact integer arithmetic.  Every function names the
passage of the paper it follows; readings of points the paper leaves open are
listed in the module docstrings and in the repository's design notes.

Pins (tests/test_oracle_*.py, run with ``-m "not gpu"``) tie this code to facts
fixed outside it: the Golay weight enumerator, the theta series of Λ24 computed
from σ11 and Ramanujan's τ, the counts the paper prints (301 classes,
N = 111,043,117,458,000 points, 47 index bits, kissing number 196,560,
N(13) = 280,974,212,784,720), brute-force enumerations of small classes, and
brute-force matvecs on tiny matrices.
"""
