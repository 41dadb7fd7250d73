"""Seeded synthetic planning instances (inputs only; no planner arithmetic)."""
from .gen import (CONFIG_NAMES, LAYER_FIELDS, ISLAND_FIELDS, load_instance, make_instance,
                  random_tiny, fixture_path, dumps, extended, node_cluster)

__all__ = ["CONFIG_NAMES", "LAYER_FIELDS", "ISLAND_FIELDS", "load_instance", "make_instance",
           "random_tiny", "fixture_path", "dumps", "extended", "node_cluster"]
