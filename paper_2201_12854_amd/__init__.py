"""Monte-Carlo Attention (MCA) forward pass for AMD Instinct MI355X (gfx950).

The compute path is the HIP library libmca.so (C ABI in include/mca.h); this
package only marshals arguments to it (``binding``) and builds it
(``build_lib``). ``workloads`` draws seeded synthetic BERT-shaped layers.
"""
from .binding import (ForwardResult, MCAError, Profiler, attention_forward, load_library,  # noqa: F401
                      prepare_weights, status_string, workspace_size, make_desc)
