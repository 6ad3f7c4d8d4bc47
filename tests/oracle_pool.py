"""CPU worker processes for the oracle side of the GPU parity tests (test
infrastructure).

The pool is forked when pytest configures a run that may hold GPU tests,
before anything in the process has touched the GPU, so the workers are plain
NumPy processes (one BLAS thread each).  The step protocol hands them one
unit's oracle step at a time; without a pool the jobs run in the calling
process.
"""

import multiprocessing as mp
import os

_POOL = None
MAX_WORKERS = 14   # the GPU test host gives one GPU's job 16 CPUs; leave two to the driving process


def _init_worker():
    for var in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ[var] = "1"
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except ImportError:
        pass


def _warm(_):
    import tests.protocol_jobs  # noqa: F401  (NumPy and the oracle, imported once per worker)
    return os.getpid()


def start(n=None):
    """Forks the workers (call before the GPU is used)."""
    global _POOL
    if _POOL is None:
        n = n or max(1, min(MAX_WORKERS, (os.cpu_count() or 2) - 1))
        _POOL = mp.get_context("fork").Pool(n, initializer=_init_worker)
        _POOL.map_async(_warm, range(n), 1)
    return _POOL


def shutdown():
    global _POOL
    if _POOL is not None:
        _POOL.terminate()
        _POOL.join()
        _POOL = None


def run(fn, jobs, chunksize=4, timeout=900):
    """[fn(job) for job in jobs], in the workers when there are some; an
    exception raised by a job is raised here, and a pool that has not answered
    within ``timeout`` seconds raises TimeoutError instead of waiting on."""
    jobs = list(jobs)
    if _POOL is None or len(jobs) < 2:
        return [fn(j) for j in jobs]
    return _POOL.map_async(fn, jobs, chunksize).get(timeout)
