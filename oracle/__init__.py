"""fp64 CPU oracle (test infrastructure only; see tree_oracle's header).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The library never does.
"""
from .tree_oracle import (  # noqa: F401
    GLA, GDN, BF16, F32, MAX_NODES_LIMIT, SUPPORTED_D,
    OracleError, InvalidArg, BadTree, BadPath, Unsupported,
    check_problem, check_forest, check_paths, root_path, topology, step,
    verify, commit, prefix_state, accepted_paths, commit_layers,
)
from .conv_oracle import conv_gates, conv_state_commit  # noqa: F401,E402
from .budget_oracle import budget_select, path_scores  # noqa: F401,E402
