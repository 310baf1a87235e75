"""pytest plugin (``-p asan_libs``) that points the library binding and the
oracle at the sanitizer builds in $GT_SANITIZED_DIR; used by
paper_1909_10616_amd/sanitize_host.sh, never collected as a test."""
import os


def pytest_configure(config):
    d = os.environ["GT_SANITIZED_DIR"]
    from paper_1909_10616_amd import gemmtune
    gemmtune.LIB_PATH = os.path.join(d, "libgemmtune.so")
    import oracle
    oracle._LIB = os.path.join(d, "liboracle.so")
