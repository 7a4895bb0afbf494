"""CPU oracle (test infrastructure only): see ``oracle.resonator_oracle``.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import
this package.  It shares no code with the HIP path.
"""
from .resonator_oracle import *  # noqa: F401,F403
from .epilogue_oracle import coupling_matrix, epilogue_fwd, epilogue_bwd  # noqa: F401
from .params_oracle import params_map, params_map_bwd, params_init, half_lives, energy_decay, spectrum  # noqa: F401
from .block_oracle import grouped_linear, grouped_linear_bwd, block_fwd, block_bwd  # noqa: F401
