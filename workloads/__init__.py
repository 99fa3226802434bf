"""Seeded synthetic inputs for the Coop window search (no search arithmetic here)."""
from .pools import (CONFIGS, EVICTABLE, FREE, GRAIN, LONG_RUN_SETS, PINNED, PoolSpec, Pools,
                    from_lists, generate, long_run, make_config, real_costs)

__all__ = ["CONFIGS", "EVICTABLE", "FREE", "GRAIN", "LONG_RUN_SETS", "PINNED", "PoolSpec", "Pools",
           "from_lists", "generate", "long_run", "make_config", "real_costs"]
