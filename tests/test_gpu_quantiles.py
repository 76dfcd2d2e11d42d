"""GPU quantile estimator (App. G) vs the oracle's chunked estimate: bit-exact
(each chunk's sort is exact, and both sides sum the chunk quantiles in chunk
order in double)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import dev, host, needs_gpu, say
from paper_2110_02861_amd import bq, workloads

pytestmark = [pytest.mark.gpu, needs_gpu]


def _inputs():
    rng = workloads.host_rng(0, "c2", 20, 0)
    return {
        "one": np.array([0.75], np.float32),
        "short": rng.standard_normal(100).astype(np.float32),
        "one_chunk": rng.standard_normal(4096).astype(np.float32),
        "chunk_plus_one": rng.standard_normal(4097).astype(np.float32),
        "ragged": workloads.student_t_host(3 * 4096 + 123, seed=3),
        "abs_t": np.abs(workloads.student_t_host(200_000, seed=4)),
        "ties": np.round(rng.standard_normal(50_000) * 3).astype(np.float32),
        "zeros": np.zeros(9000, np.float32),
        "normal_1m": rng.standard_normal(1 << 20).astype(np.float32),
    }


@pytest.mark.parametrize("name", list(_inputs()))
def test_estimate_matches_oracle(name):
    x = _inputs()[name]
    say(f"quantile estimate {name} n={x.size}")
    q = bq.bq_estimate_quantile_codebook(dev(x))
    torch.cuda.synchronize()
    ref = oracle.chunked_quantile_codebook(x)
    np.testing.assert_array_equal(host(q).view(np.uint32), ref.view(np.uint32))


def test_estimate_feeds_the_quantizer():
    """The estimated map is a valid map for the block-wise kernels."""
    x = workloads.student_t_host(1 << 18, seed=5)
    x_d = dev(x)
    say("quantile estimate -> quantize")
    q_d = bq.bq_estimate_quantile_codebook(x_d)
    codes, absmax = bq.bq_quantize_blockwise(q_d, x_d, 2048)
    torch.cuda.synchronize()
    q = host(q_d)
    assert np.all(np.diff(q) > 0)
    c_ref, a_ref = oracle.quantize_blockwise(q, x, 2048)
    np.testing.assert_array_equal(host(codes), c_ref)
    np.testing.assert_array_equal(host(absmax), a_ref)
