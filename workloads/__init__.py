"""Seeded synthetic workloads shared by the oracle and the GPU path (inputs only)."""
from .configs import (Workload, LayerShape, WORKLOADS, WORKLOAD_ORDER, TAU_JUMP, GAMMA,
                      LOOKAHEAD, TAU_PAD, LLADA8B, TINY, act_eps_for, scaled)
