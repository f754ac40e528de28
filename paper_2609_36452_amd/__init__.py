"""MI355X (gfx950) commit step of Reliable Parallel Decoding.

``binding`` wraps the C ABI of ``librpd.so`` (include/rpd.h); ``workload``
draws seeded synthetic inputs of the paper's model shapes."""
from .binding import (Params, RpdError, ScoreCommit, abi_version, gate_commit, last_error, lib,  # noqa: F401
                      score_commit, status_string, workspace_size)
