"""fp64 CPU oracle for the read-sparse readout and store-sparse commit.

TEST INFRASTRUCTURE ONLY.  This package is the slow, plain definition of what
the HIP path computes; it is imported only by the tests, by the smoke check
and by the benchmark's CPU-baseline leg.  The product path never calls it and
shares no code with it (neither imports the other).  Inputs come from the
seeded generator in ``workloads``; every floating-point step runs in float64
on values widened exactly from their stored bfloat16/float32 bits.

Modules:
  geometry  down-sampling, bounding boxes, Chebyshev dilation, tracker state
            (Sec. 3.1, Eqs. 1, 2 and 5; Algorithm 1)
  select    token energy and the read keep-set (Sec. 3.1, Eq. 4)
  readout   the sparse memory readout with scatter (Sec. 3.1, Eq. 6)
  rope      rotary positions on the gathered subset (Sec. 3.1, Eq. 7)
  bank      write compaction and the ring memory bank (Sec. 3.2, Eq. 8)
  write     the paper's fixed write keep-set K_w (Sec. 3.2, Eq. 8)
  post      closure of the decoded masks and the palette argmax (Sec. 3.3)
  stack     the L-layer memory-attention stack on the kept queries (Sec. 3.1,
            "Sparse memory attention"; the layer is a reading, see its doc)

Parity unpinned: absolute readout and stack values at the workload sizes (the paper
prints no tensors and its weights are not available); every other function is
pinned by the tests in tests/test_oracle_*.py.  The axial rotary table is a
reading (the paper gives only its shape); its stated form is pinned, its
choice is not.
"""
from .geometry import Track, bbox, down_s, down_s_box, fill_box, dilate, prior_object  # noqa: F401
from .select import energy, topk_keep, select_queries  # noqa: F401
from .rope import axial_table, table_from_pairs, rotate, rotate_heads  # noqa: F401
from .readout import (project_bank, rotate_keys, attention_weights, readout, readout_dense,  # noqa: F401
                      readout_dense_projected, attend)
from .write import write_keepset  # noqa: F401
from .post import close_square, palette, close_masks  # noqa: F401
from .bank import compact, RingBank, FrameListBank, RS3_OK, RS3_E_INVALID, RS3_E_CAPACITY  # noqa: F401
