"""CPU oracle for the group-rollout hot path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct reference for what the HIP library computes:
a random-init decoder's prefill and KV-cached decode in float64 (numpy), exact
Gumbel-max sampling driven by Philox4x64-10, forced-length retirement, and the
group-relative advantage.  Only the test suite, the smoke entry point and the
CPU-baseline leg of the benchmark may import it.  It shares no code with the
HIP path; both consume the seeded inputs built by the ``workload`` package.
"""
from .philox import philox4x64_10, gumbel_uniform_bits, uniforms_from_bits, gumbel_noise  # noqa: F401
from .model import OracleModel  # noqa: F401
from .sampling import sample_token  # noqa: F401
from .rollout import rollout, group_offsets  # noqa: F401
from .advantage import group_advantage  # noqa: F401
