"""Seeded synthetic inputs for the PASK decode hot path.

This package only draws inputs: workload shapes, structural-tag streams,
policy tables (a seeded stand-in for the offline calibration of the paper's
Alg. 1) and bf16 tensors.  It holds none of the hot path's arithmetic
(lookup, compaction, quantisation, attention); both the CPU oracle's tests
and the HIP path consume what it produces.
"""

from .configs import CONFIGS, Config, get_config  # noqa: F401
from .tags import (  # noqa: F401
    DECODE_TAGS,
    PROMPT_TAGS,
    iid_tags,
    function_call_tags,
    schema_prompt_tags,
    tag_mix,
)
from .policy import PolicyTable, make_policy, pack_blob  # noqa: F401
from .tensors import bf16_normal, prompt_lengths  # noqa: F401
