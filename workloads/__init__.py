"""Seeded synthetic inputs for the Coop window search (no search arithmetic here)."""
from .pools import (CONFIGS, EVICTABLE, FREE, GRAIN, PINNED, PoolSpec, Pools, from_lists,
                    generate, make_config, real_costs)

__all__ = ["CONFIGS", "EVICTABLE", "FREE", "GRAIN", "PINNED", "PoolSpec", "Pools",
           "from_lists", "generate", "make_config", "real_costs"]
