"""MI355X-native batch-1 self-speculative decoding with learned
(exit layer, draft length) control.  The compute path is liblede.so
(hand-written gfx950 HIP kernels behind the C ABI in include/lede.h);
``lede`` is its ctypes binding."""
from .lede import (Dqn, Engine, LedeError, load, make_config, op_linear, op_read_groups, op_read_probe,  # noqa: F401
                   op_sample, op_sample_noalloc)
