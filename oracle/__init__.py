"""CPU oracle for FT-CNN checksum-protected convolution (arXiv 2003.12203).

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The HIP library
never calls it, links it or falls back to it.

* ``oracle.core``: the C loops (direct convolution of eq. (1), input checksum
  sums) built from ``ftcnn_oracle.c`` with gcc, everything in float64;
* ``oracle.workflow``: checksums, detection and the correction chain of
  Sec. 3-4 in float64 numpy, following the paper's definitions and order.

Pins (tests/test_oracle_*.py): brute-force seven-loop convolution on tiny
shapes, torch's float64 CPU conv2d as an independent library evaluation,
closed forms (one-hot inputs, constant inputs, per-image constants),
integer-exact inputs, the distributive property of Sec. 3.1, the location
identities of Sec. 3.6 and the protection-ability table of Sec. 4.1.  The
tolerance constants kappa and eta are readings of this implementation, not
values from the paper: parity unpinned for their exact values.
"""
from . import core, workflow  # noqa: F401
from .workflow import (Checksums, Fault, Policy, Report, protect, store, verify,  # noqa: F401
                       correct, encode, coc_checksums, row_checksums, col_checksums)
