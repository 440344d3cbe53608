"""MI355X (gfx950) implementation of one pipeline stage's training step under a one-step gradient
delay: decoder-block forward/backward and the delayed AdamW / Error-Feedback update, as HIP kernels
behind the C ABI of include/asyncstage.h."""
from . import binding  # noqa: F401  (raises ImportError when the library is not built)
