"""Many equal keys and segments of many tiles, HIP path against the oracle.

Equal keys at the threshold (exact zeros, values of a narrower float type)
put most candidates on one histogram bin; a segment whose tiles number in the
thousands (a bracket miss on a large tensor, or every element a candidate)
takes its tile prefixes from group sums.  Both must give the oracle's result
bit for bit (Algorithm 1, Section 4: the k largest |acc|, ties to the lower
index).
"""
import numpy as np
import pytest

from paper_1704_05021_amd import gd, workloads as wl
from parity import check_case

pytestmark = pytest.mark.gpu

C3 = wl.workload("nmt_85k_per_tensor")


def _to_bf16_values(x: np.ndarray) -> np.ndarray:
    return (x.view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32)


@pytest.mark.parametrize("per_tensor", [True, False], ids=["per_tensor", "global"])
def test_sparse_first_step_needs_zeros(per_tensor):
    # 1,000 tokens touch about 470 rows of each 85,000 x 500 embedding: fewer
    # nonzeros (about 234k) than k (425k), so each embedding keeps all its
    # nonzeros and its first zeros by index
    g = wl.grad_nmt(C3.layout, C3.seed, 0, tokens=1000)
    off = C3.layout.offsets
    if per_tensor:
        nnz = int(np.count_nonzero(g[off[0]:off[1]]))
        assert nnz < gd.keep_count(off[1] - off[0], 0.99)
    check_case(g, np.zeros_like(g), off, 0.99, per_tensor, False, what=f"sparse step 0 per_tensor={per_tensor}")


@pytest.mark.parametrize("per_tensor,quant", [(True, False), (False, False), (False, gd.GD_QUANT_THRESHOLD)],
                         ids=["per_tensor", "global", "global_threshold_centres"])
def test_bf16_valued_gradient(per_tensor, quant):
    g = _to_bf16_values(C3.grad(0))
    check_case(g, np.zeros_like(g), C3.layout.offsets, 0.99, per_tensor, quant,
               what=f"bf16-valued per_tensor={per_tensor} quant={quant}")


def _few_values(n: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return (rng.integers(-8, 9, n) * 0.25).astype(np.float32)


@pytest.mark.parametrize("debug", [0, 1, 3], ids=["sampled", "fallback", "all_cands"])
@pytest.mark.parametrize("drop", [0.99, 0.7])
@pytest.mark.parametrize("per_tensor", [True, False], ids=["per_tensor", "global"])
def test_grouped_segments_with_ties(per_tensor, drop, debug):
    # 17 distinct values: the threshold is a value shared by several hundred
    # thousand elements, and the 5M-element tensor spans about 4,900 tiles
    # when every element is a candidate
    off = [0, 5_000_000, 5_000_100, 6_300_003]
    g = _few_values(off[-1], 11)
    r = np.zeros_like(g)
    r[::7] = np.float32(0.25)  # some residual, so acc is not g alone
    check_case(g, r, off, drop, per_tensor, False, debug_bracket=debug,
               what=f"few values per_tensor={per_tensor} drop={drop} debug={debug}")


@pytest.mark.parametrize("per_tensor", [True, False], ids=["per_tensor", "global"])
def test_fp16_valued_ties_spread_over_bins(per_tensor):
    # fp16 keeps 10 mantissa bits: candidates that share the threshold's first
    # 18 key bits fall in two digit-2 bins, so both the run and the
    # one-by-one counting take part
    rng = np.random.default_rng(12)
    off = [0, 3_000_000, 3_500_000, 6_000_000]
    g = rng.standard_normal(off[-1]).astype(np.float16).astype(np.float32)
    check_case(g, np.zeros_like(g), off, 0.99, per_tensor, False, what=f"fp16-valued per_tensor={per_tensor}")


def test_grouped_segment_with_quantised_centres():
    off = [0, 5_000_000, 5_000_100, 6_300_003]
    g = _few_values(off[-1], 13)
    check_case(g, np.zeros_like(g), off, 0.99, False, gd.GD_QUANT_SIGN_MEAN, debug_bracket=3,
               what="few values, every element a candidate, sign-mean centres")
