import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")


_CACHE = {}


@pytest.fixture(scope="session")
def workload_inputs():
    """Memoised synth.make_inputs(name) so that big workloads are generated once."""
    import synth

    def get(name):
        if name not in _CACHE:
            _CACHE[name] = synth.make_inputs(synth.get_workload(name))
        return _CACHE[name]
    return get


_EST = {}


@pytest.fixture(scope="session")
def oracle_estimate(workload_inputs):
    """Memoised oracle estimator output (masks, parts) per workload name."""
    import oracle

    def get(name):
        if name not in _EST:
            d = workload_inputs(name)
            w = d["workload"]
            _EST[name] = oracle.estimate_masks(
                d["q"], d["k_pool"], d["page_table"], d["cached_len"], w.page_size,
                w.q_block, w.chunk_len, w.words,
                oracle.EstimatorParams(w.top_frac, w.sink_blocks, w.local_blocks),
                return_parts=True)
        return _EST[name]
    return get
