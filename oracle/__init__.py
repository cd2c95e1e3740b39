"""Reference oracle for Top-p block-sparse video attention (test infrastructure).

This package is a plain, slow, fp64 CPU implementation of what the GPU path
computes. It exists only to check the GPU path: it may be imported by the
test-suite, by the smoke check and by the CPU-baseline leg of the benchmark,
and by nothing else. It shares no code, tables or helpers with the HIP
library; the two are written independently from the paper's definitions.

Passages followed (FVAttn, "Adaptive Sparse Attention with Runtime Load
Balancing for Video Generation"):

* video-aware block organisation and pooled block similarities -- §3.1
  (routing frontend paragraph), as 3D boxes or as runs of a Hilbert curve
  (the block reordering of the same paragraph);
* block mask M_{h,i,j} over (query block, key block) pairs -- §2.1;
* Top-p: keep key blocks in decreasing score order until their summed
  softmax mass is at least p (m_p = min{r : c_r >= p}) -- §2.1;
* Top-k safety floor -- §2.1 and §3.1;
* realised per-head workload L_h = mean_i sum_j M_{h,i,j} -- §2.2, Eq. 1;
* block-sparse attention over the retained blocks only -- §2.1, §3.1;
* the quantised-V variant (E4M3 codec, per-channel power-of-two scales,
  bound on the rounding of P) -- §3.4 (GPU-side V quantisation), in
  fp8.py, imported on its own;
* slack-aware sparse augmentation (per-rank slack, trigger, budget, extra
  blocks in the routing order) -- §3.3, in sasa.py, imported on its own.

Parity status of each function is stated in its docstring. One part is
"parity unpinned": whether these masks equal the masks of the paper's own
implementation. The paper prints no mask statistics, score scale, block size
or floor value, so the masks are exact to the reading written down here, not
checkable against the paper's numbers.
"""

from .tiling import TileGeometry, tile_geometry
from .curve import curve_bits, hilbert_index, curve_order, curve_geometry
from .route import (
    pool_blocks,
    block_scores,
    block_softmax,
    topp_select,
    route_ref,
    head_workload,
)
from .attention import attn_ref_rows, attn_ref_head

__all__ = [
    "TileGeometry",
    "tile_geometry",
    "curve_bits",
    "hilbert_index",
    "curve_order",
    "curve_geometry",
    "pool_blocks",
    "block_scores",
    "block_softmax",
    "topp_select",
    "route_ref",
    "head_workload",
    "attn_ref_rows",
    "attn_ref_head",
]
