"""The allocation-free decode entry point against the workspace one, through the C ABI.

attention_decode_deferred_noalloc keeps the key-range partials in the library's own device
array; its output must equal attention_decode_deferred's bit for bit, on a first call and on a
second, smaller one that reuses the array (partials left over from the first must not leak in).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2502_17728_amd import inputs as I
from tests.parity import TOL, cuda, rowwise_rel_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ops():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2502_17728_amd import ops as _ops
    return _ops


def _both(ops, case):
    q, k, v = cuda(case["Q"]), cuda(case["K"]), cuda(case["V"])
    ref = ops.attention_decode_deferred(q, k, v, scale=case["scale"])
    out = torch.empty_like(q)
    got = ops.attention_decode_deferred_noalloc(q, k, v, scale=case["scale"], out=out)
    torch.cuda.synchronize()
    return got, ref


@pytest.mark.parametrize("d", [64, 128])
def test_noalloc_matches_workspace_entry_point_twice(ops, d):
    # first call: many splits per head (a few heads, a long cache, 16 query rows: the largest
    # partials); second call: fewer heads, rows and keys, so most of the array holds stale data
    big = I.make_decode_case(3, 16, 20000, d, seed=31 + d)
    small = I.make_decode_case(2, 3, 900, d, seed=32 + d)
    for case in (big, small):
        got, ref = _both(ops, case)
        assert torch.equal(got, ref)
        BH, Lq = case["Q"].shape[:2]
        exp = oracle.attention(case["Q"].reshape(-1, d), case["K"], case["V"], case["scale"],
                               head=np.repeat(np.arange(BH), Lq))
        assert rowwise_rel_err(got.cpu().reshape(-1, d), exp) <= TOL[torch.bfloat16]


def test_noalloc_grouped_query_and_single_pass(ops):
    # grouped-query (4 query heads per key/value head) with splits, then enough heads for one
    # pass without partials
    gqa = I.make_decode_case(8, 1, 3000, 128, seed=33, group=4)
    wide = I.make_decode_case(1100, 1, 200, 128, seed=34)
    for case in (gqa, wide):
        got, ref = _both(ops, case)
        assert torch.equal(got, ref)


def test_noalloc_largest_partials_fit(ops):
    # every request the workspace entry point accepts fits the fixed array
    from paper_2502_17728_amd import ops as o
    for d in (64, 128):
        for BH in (1, 2, 3, 7, 100, 255, 511, 1279):
            need = o.attention_decode_workspace_bytes(BH, 16, 1 << 20, d)
            assert 0 < need <= 12 << 20, (d, BH, need)
