"""pytest plugin for the sanitizer run of the C ABI tests: points the binding
at the host-only sanitizer build named by the test that starts the run."""
import os


def pytest_configure(config):
    from paper_2608_23167_amd import _lib
    _lib.use_library(os.environ["SSM_HOSTSAN_LIB"])
