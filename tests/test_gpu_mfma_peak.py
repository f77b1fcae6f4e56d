"""The measured MFMA peak (dash_mfma_peak) that bench.py reports beside the
published one: a physically possible bf16 dense rate for MI355X."""
import pytest

from paper_2601_21824_amd import binding as dash

pytestmark = pytest.mark.gpu


def test_mfma_peak_is_physical():
    print("\n[mfma_peak]", flush=True)
    t = dash.dash_mfma_peak(2000)
    # 256 CUs x 4 SIMDs x 1024 bf16 FLOP per cycle at 2.4 GHz = 2517 TFLOP/s;
    # a chip that cannot reach half of it is not running the MFMA chains
    assert 1250.0 < t < 2600.0, t
