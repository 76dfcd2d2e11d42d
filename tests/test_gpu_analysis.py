"""The synthetic data-type comparison (App. F) runs end to end on the GPU kernels."""
import math

import pytest

from gpu_helpers import needs_gpu, say
from paper_2110_02861_amd import analysis

pytestmark = [pytest.mark.gpu, needs_gpu]


def test_data_type_comparison_small():
    say("analysis 1024 x 512, 8 steps")
    res = analysis.run(rows=1024, cols=512, steps=8, blocksize=2048, row_spread=256, outlier=10.0)
    assert set(res) == set(analysis.FAMILIES)
    for fam, v in res.items():
        for k, x in v.items():
            assert math.isfinite(x), (fam, k, x)
    # the dynamic map has the smallest absolute error of the first state and a
    # far smaller relative Adam error than the linear map (App. F)
    err = {k: v["absolute_quantization_error"] for k, v in res.items()}
    assert err["dynamic"] < err["linear"]
    assert res["dynamic"]["relative_adam_error"] < res["linear"]["relative_adam_error"]
    assert res["linear"]["r_quantized_to_zero"] > res["dynamic"]["r_quantized_to_zero"]
