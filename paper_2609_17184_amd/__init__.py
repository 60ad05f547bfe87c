"""MI355X (gfx950) LoopSpec: pipelined self-speculative decoding of Looped
Transformers as hand-written HIP kernels behind a C ABI (include/loopspec.h).

`binding.Decoder` is the Python entry point; `build.build()` compiles the
library in-tree."""
from .binding import Decoder, LoopSpecError, load_library, worst_case_branches  # noqa: F401
