"""Seeded synthetic inputs (tree topologies and operand arrays) shared by the tests,
the benchmark and the oracle harness. Holds no part of the recurrence's arithmetic."""
from . import configs, operands, trees  # noqa: F401
