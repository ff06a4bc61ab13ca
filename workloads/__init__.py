"""Seeded synthetic computation graphs (inputs only; no search arithmetic)."""
from .gen import (WORKLOADS, chain_graph, fc_chain, inception, lstm_grid, random_costs,  # noqa: F401
                  random_graph, residual_cnn, transformer, workload)
