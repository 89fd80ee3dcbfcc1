"""Seeded float64 parameters of a network, from the shared input generator.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py)."""
from workloads import synth


def net_params(net, dtype, index_offset=0, family=synth.NORMAL):
    """[(W as float64 OIHW, b as float64 or None)] per layer, holding exactly
    the quantised values the HIP run receives."""
    out = []
    for idx in range(len(net.layers)):
        (w64, _), b = synth.layer_params(net, idx, dtype, index_offset, family)
        out.append((w64, None if b is None else b[0]))
    return out
