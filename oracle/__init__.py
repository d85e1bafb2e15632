"""CPU oracle for Hilbert-guided block-sparse local attention (arXiv 2511.05832).

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or
execute anything in this package: only the tests, the smoke check and the
bench's CPU-baseline leg do. It shares no code with the HIP library and does not
import it.

It is the plain, slow, obviously-correct definition of what the hot path
computes, in float64 with NumPy:

  hilbert    Hilbert order of a 2^k x 2^k grid by recursive quadrant
             construction, and its inverse (Sec. 3.1-3.2).
  masks      element-wise attention masks: Hilbert window / slide /
             neighbourhood / shifted window on sequence positions, and the
             row-major window / slide / neighbourhood baselines (Sec. 3.1-3.3,
             Fig. 3).
  blockmask  tile classification full / partial / empty, by brute force from
             the element mask, and the per-row tile lists and per-column lists
             (Sec. 3.1).
  attention  dense element-wise-masked softmax attention and its log-sum-exp
             (Sec. 3.1, Eq. 1 context; the block-sparse kernel computes exactly
             this result faster), and its gradients with respect to q, k, v
             (the backward pass the paper times beside the forward).
  layer      the Hilbert-neighbourhood-style layer: QKV projection, Hilbert
             slide attention, output projection, computed in row-major order
             (Sec. 3.3, Sec. 4.2 "input processing").
  permute    gather into / scatter out of Hilbert order (Sec. 4.2, "reshape").

Every function is pinned by the CPU tests against values the paper prints
(sparsity columns of Tables 1-3 and 6-11, the worked example of Fig. 3),
closed forms, library routines on special cases, and brute force on tiny inputs.
"""
from . import hilbert, masks, blockmask, attention, layer, permute  # noqa: F401
