"""Seeded synthetic inputs for the prefix-cached prefill path.

This package holds *no* arithmetic of the method (no hashing, no policy, no
attention): only the workload shapes, seeded token ids, seeded request streams
and seeded bf16 Q/K/V tensors.  Both the oracle-side tests and the library-side
harness take their inputs from here.

The paper measures on QuALITY / WikiQA documents sampled by windowed Zipf and
on the Qwen-Bailian conversation trace (Sec. 4).  None of those are available;
the configurations below are synthetic stand-ins with the same kind of
structure (long shared document prefixes with skewed popularity, growing
multi-turn histories, one-off scan traffic).
"""

from .configs import CONFIGS, Config, get_config  # noqa: F401
from .streams import Request, Source, make_stream  # noqa: F401
