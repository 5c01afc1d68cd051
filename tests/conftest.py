import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:           # helper modules shared by tests (precision_case)
    sys.path.insert(0, HERE)

_ORACLE_POOL = None


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running case")


def pytest_collection_finish(session):
    """Fork the oracle's worker pool after collection and before the first test
    runs, i.e. before any test touches the GPU, when GPU tests are selected:
    the full-batch parity tests run the oracle over every sequence of the
    large workloads in parallel."""
    global _ORACLE_POOL
    if _ORACLE_POOL is None and any(item.get_closest_marker("gpu") for item in session.items):
        from oracle.pool import OraclePool
        _ORACLE_POOL = OraclePool()


def pytest_sessionfinish(session, exitstatus):
    global _ORACLE_POOL
    if _ORACLE_POOL is not None:
        _ORACLE_POOL.close()
        _ORACLE_POOL = None


@pytest.fixture(scope="session")
def oracle_pool():
    global _ORACLE_POOL
    if _ORACLE_POOL is None:        # CPU tests that ask for it directly
        from oracle.pool import OraclePool
        _ORACLE_POOL = OraclePool()
    return _ORACLE_POOL


class _StageBatches:
    """The five generated workloads and their oracle outputs, built once per
    session (the long-context batch alone is 10.7 GB of pools)."""

    def __init__(self, pool):
        self.pool = pool
        self.w = {}
        self.ref = {}

    def workload(self, k):
        if k not in self.w:
            from workloads import build_config
            print(f"[gpu case] build config {k}", flush=True)
            self.w[k] = build_config(k)
        return self.w[k]

    def reference(self, k):
        """Oracle (out, lse) of every sequence of config k."""
        if k not in self.ref:
            w = self.workload(k)
            print(f"[gpu case] oracle over all {w.batch} sequences of config {k} "
                  f"({self.pool.workers} workers)", flush=True)
            self.ref[k] = self.pool.decode_workload(w)
        return self.ref[k]

    def drop(self, k):
        self.w.pop(k, None)
        self.ref.pop(k, None)


@pytest.fixture(scope="session")
def stage_batches(oracle_pool):
    sb = _StageBatches(oracle_pool)
    yield sb
    sb.w.clear()
    sb.ref.clear()
