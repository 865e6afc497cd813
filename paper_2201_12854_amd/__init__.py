"""Monte-Carlo Attention (MCA) forward pass for AMD Instinct MI355X (gfx950).

The compute path is the HIP library libmca.so (C ABI in include/mca.h); this
package only marshals arguments to it (``binding``) and builds it
(``build_lib``). ``workloads`` draws seeded synthetic BERT-shaped layers.
"""
from .binding import (ForwardPlan, ForwardResult, MCAError, Profiler, attention_forward,  # noqa: F401
                      load_library,
                      prepare_weights, prepared_size, rownorm, status_string, workspace_size, make_desc)
