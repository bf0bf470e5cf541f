"""Seeded synthetic workloads shared by the oracle and the GPU path: network descriptions
(structure only) and input / parameter generators.  Holds none of the method's arithmetic."""
from .nets import Net, Node, Segment, config, CONFIG_NAMES  # noqa: F401
from .gen import make_all, make_input, make_labels, init_params, segment_shapes  # noqa: F401
