"""The oracle against its pins (CPU only)."""
import pytest

from tests import oracle_checks as C


@pytest.mark.parametrize("check", C.ALL_CHECKS, ids=lambda f: f.__name__)
def test_pin(check):
    check()
