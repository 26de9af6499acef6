"""The driver's smoke entry point, run as the round-end check runs it."""
import pytest

from gpu_util import require_gpu

pytestmark = pytest.mark.gpu


def test_smoke_entry_point():
    require_gpu()
    import __graft_entry__
    __graft_entry__.smoke()
