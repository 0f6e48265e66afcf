"""Host-side checks of the two-stream step wrapper (no GPU needed): the
package exports it, and a bad schedule name is rejected before any stream or
device is touched."""
import pytest

import paper_1905_07931_amd as L1


def test_step_api_is_exported():
    assert "l1_step" in L1.__all__ and "side_stream" in L1.__all__
    assert callable(L1.l1_step) and callable(L1.side_stream)


@pytest.mark.parametrize("bad", ["parallel", "", "Serial", None])
def test_unknown_schedule_rejected_before_any_device_work(bad):
    with pytest.raises(ValueError):
        L1.l1_step(None, None, None, 0.01, 1e-4, Y=None, dX=None, dW=None, csc=None, out=None,
                   schedule=bad)
