"""pytest plugin of the sanitizer run: point the binding and the oracle at the
AddressSanitizer/UBSan builds named by ECHO_SANITIZED_LIB and
ORACLE_SANITIZED_LIB before any test loads a library.  Loaded with
``-p tests.sanitize.plugin`` by tests/test_sanitized_host.py only."""
from __future__ import annotations

import os


def pytest_configure(config):
    lib = os.environ.get("ECHO_SANITIZED_LIB")
    if lib:
        import paper_2412_12487_amd.echo as echo
        echo.LIB_PATH = lib
    olib = os.environ.get("ORACLE_SANITIZED_LIB")
    if olib:
        import oracle
        oracle._LIB = olib
