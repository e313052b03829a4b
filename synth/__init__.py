"""Seeded synthetic workloads for the LookME hot path (inputs only).

This package holds no part of the method's arithmetic: it draws random
tensors with the shapes and distributions of the paper's workloads and is the
one piece shared by the tests, the benchmark and the CPU oracle's callers.
"""

from .gen import (Workload, WORKLOADS, make_inputs, make_integer_inputs,  # noqa: F401
                  make_fusion, make_gate, make_layer, make_multiscale, make_propagation,
                  make_relevance, make_text, n_keep_for)
