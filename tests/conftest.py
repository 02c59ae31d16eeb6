import ctypes
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def _host_setup():
    """The fp64 oracle works on large temporaries: keep freed heap memory for reuse instead
    of returning it to the OS after every array (first-touch page faults dominate otherwise),
    and cap the BLAS thread pool (spinning BLAS workers starve numpy's element-wise loops)."""
    try:
        libc = ctypes.CDLL("libc.so.6")
        libc.mallopt(-4, 0)            # M_MMAP_MAX: serve large blocks from the heap
        libc.mallopt(-1, 2 ** 31 - 1)  # M_TRIM_THRESHOLD: never trim the heap
    except OSError:
        pass
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(int(os.environ.get("ORACLE_BLAS_THREADS", "4")))
    except Exception:
        pass


_host_setup()


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")
