"""Oracle for 1xN pruning and the 1xN-pruned convolution.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package.  It shares no code with the HIP
library and the HIP library never imports it.

Everything is computed in fp64 by the plain C in ``oracle.c`` (Lin et al.,
"1xN Pattern for Pruning Convolutional Neural Networks", arXiv 2105.14713):

* ``filter_perm``      - Sec. 3.3, filter rearrangement by decreasing l1 norm.
* ``block_scores``     - Sec. 3.2, Eq. 4/5: l1 norm of every 1xN block.
* ``select``           - Eq. 1 and the solution of Eq. 5: per-layer top-(1-p).
* ``masked_weight``    - Eq. 6: Omega-bar = Omega-tilde masked by T.
* ``pack``             - Sec. 3.4, Fig. 3: BSR arrays (P, I, D).
* ``conv2d`` / ``conv2d_at`` - Eq. 7: direct convolution with Omega-bar.
* ``decode``           - Eq. 8: block-wise decode over (P, I, D).
* ``conv2d_bwd_data`` / ``conv2d_bwd_weight`` - the backward of Eq. 7 for
                         fine-tuning with the pattern fixed (Sec. 4.1): the
                         adjoint through Omega-bar, and the weight gradient on
                         the kept blocks only.
* ``epilogue``         - per-channel scale/bias and ReLU/ReLU6 after a conv
                         (folded batch norm of the Sec. 4.1 networks).
* ``prune``            - the offline steps chained: perm, T, t, Omega-bar, BSR.

Every function takes and returns numpy arrays; weights and activations are
float64 (fp32 and bf16 values widen exactly).
"""
from .oracle import (apply_perm, block_scores, conv2d, conv2d_at, conv2d_bwd_data, conv2d_bwd_weight,
                     decode, epilogue, filter_norms,
                     filter_perm,
                     kept_count, masked_weight, num_threads, pack, prune, select,
                     set_num_threads)

__all__ = ["apply_perm", "block_scores", "conv2d", "conv2d_at", "conv2d_bwd_data", "conv2d_bwd_weight",
           "decode", "epilogue", "filter_norms",
           "filter_perm",
           "kept_count", "masked_weight", "num_threads", "pack", "prune", "select",
           "set_num_threads"]
