"""CPU oracle for the SLiM compressed linear layer and SLoPe's double-pruned backward.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package. The HIP product path
never calls it and shares no code with it.

Everything here is plain NumPy in float64 (pure Python in ``brute``), written from
the thesis' definitions:

* 2:4 magnitude mask along the reduction dimension (SLoPe, "Double-pruned Backward
  Pass"; background section "Sparse Tensor Core Acceleration").
* Group-wise symmetric AbsMax int4 quantisation of the kept weights (SLiM, section
  "Quantization" under the preliminaries and eq. symmetric_quantization, group size
  128 as in the SLiM experimental setup and "Low-rank adapter quantization").
* The compressed layer Y = X Wc^T + (X L) R (SLiM, sparse plus low-rank; SLoPe
  eq. sparse_plus_low_rank).
* SLoPe's double-pruned input gradient dX = dY W^{R,C} (eq. sparse_backward_input)
  and Lemma sparsity_ratio.
* The steps of SLoPe's training step after the input gradient (``slope_train``): the
  half-precision value packs of W^R and W^{R,C}, the masked and compressed weight
  gradient (eq. sparse_backward_weight), the same-pattern sparse add and the pack update
  (Alg. "Accelerated Sparse Pretraining Algorithm for a Linear Layer"; appendix
  "Implementation details").
* SLiM-Quant's histogram-based mean-squared-error scale search (``slim_quant``; SLiM,
  eq. error_summation and Alg. quantization) and the forward pack with its per-tensor scale.
* SLiM-LoRA's saliency-based adapters (``slim_lora``; SLiM, eq. lora_svd and Alg. lora).
* PATCH's hybrid dense / 2:4 tile weight and its product (``patch_hybrid``; PATCH, "Efficient
  deployment of PATCH").

Parity status per function is stated in ``slim_oracle``'s module docstring.
"""
from . import slim_oracle  # noqa: F401
from . import slope_train  # noqa: F401
from . import slim_quant  # noqa: F401
from . import slim_lora  # noqa: F401
from . import patch_hybrid  # noqa: F401
