"""The oracle's float64 output of each single-layer workload, computed once
per test process and shared by every parity test that runs that layer
(split path at each tile and placement, OaAConv, spatial convolution).

Every output channel of every image is compared: the direct
cross-correlation of the largest layer (16 x 256 x 56 x 56 -> 256, K = 5)
takes about a second on 16 host cores.
"""
import functools

import oracle
from workloads import make_config


@functools.lru_cache(maxsize=None)
def config_inputs(name):
    return make_config(name)


@functools.lru_cache(maxsize=None)
def config_reference(name):
    x, w, b = config_inputs(name)
    ref = oracle.direct_xcorr2d(x, w, b)
    ref.setflags(write=False)
    return ref
