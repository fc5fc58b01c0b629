"""MI355X-native Ball Sparse Attention (BSA) layer hot path.

The HIP kernels and the C ABI live in ``csrc/`` and build into ``libbsa.so``
(``python -m paper_2506_12541_amd.build``); ``bsa`` is the torch binding.
"""
from .bsa import (BSA_BF16, BSA_F32, BSA_POOL_MEAN, BSA_POOL_MLP, Params, Saved, backward,  # noqa: F401
                  build_ball_tree, forward, permute, sizes, unpermute)
