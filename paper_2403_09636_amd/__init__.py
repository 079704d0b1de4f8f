"""MI355X (gfx950) Dynamic Memory Compression decode path.

The work happens in libdmc.so (HIP kernels behind the C ABI of
include/dmc.h); ``binding`` marshals torch tensors into it.
"""
from .binding import (DMCCache, DMCError, CacheConfig, make_config,  # noqa: F401
                      workspace_bytes, LIB_PATH, EXPORTS, DMCTrainer, TrainConfig,
                      make_train_config)
