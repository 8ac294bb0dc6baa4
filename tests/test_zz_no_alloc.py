"""arckv_prefill_attention_noalloc (the entry point for callers that cannot allocate) against
arckv_prefill_attention with a caller workspace, through the C ABI, on the GPU.

Both calls run the same planned batch; the outputs must be bitwise equal (the same kernels
reduce in the same order) and within the attention tolerance of the fp64 oracle.  Calls follow
each other on one device, so they share the static scratch: a later, smaller batch must not
pick up the partials an earlier one left there.
"""

from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import paper_2606_21238_amd as ak  # noqa: E402
from tests.gpu_helpers import bits, compare, print_case  # noqa: E402
from tests.test_gpu_parity import DEV, build_batch, oracle_out, run_attention  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ak.lib()


def run_noalloc(b, hq, hkv, d, num_cus):
    ap = ak.attention_plan(b["cu"], b["seq"], hq, hkv, d, num_cus)
    out = torch.full_like(b["q"], float("nan"))
    ak.prefill_attention_noalloc(b["kp"], b["vp"], b["q"], out, torch.from_numpy(b["bt"]).to(DEV),
                                 torch.from_numpy(b["cu"]).to(DEV), torch.from_numpy(b["seq"]).to(DEV),
                                 torch.from_numpy(ap.work).to(DEV), ap.n_work, ap.n_combine, ap.tile_cols,
                                 d ** -0.5, ap.ws_bytes)
    torch.cuda.synchronize()
    return bits(out), ap


# (reqs [(L, P)], hq, hkv, d, num_cus): every plan splits key ranges (so the scratch is used);
# each case is smaller than the one before it
CASES = [
    ([(9000, 8872), (4000, 3872)], 32, 8, 128, 256),                   # wide tiles, 32 MiB of partials
    ([(5000, 4990), (3000, 2990), (2100, 2068)], 32, 8, 128, 100000),  # narrow tiles
    ([(1040, 1024), (600, 500)], 32, 8, 128, 256),
    ([(L, L - 1) for L in (300, 4097, 2000, 65)], 40, 8, 128, 256),    # decode-like batch
]


def test_noalloc_matches_the_workspace_entry_point_call_after_call():
    for k, (reqs, hq, hkv, d, num_cus) in enumerate(CASES):
        print_case(f"noalloc case {k}: {reqs} hq={hq} hkv={hkv} d={d} num_cus={num_cus}")
        b = build_batch(reqs, hq, hkv, d, seed=700 + k)
        want, ap = run_attention(b, hq, hkv, d, num_cus)
        got, ap2 = run_noalloc(b, hq, hkv, d, num_cus)
        assert ap.n_combine > 0 and 0 < ap.ws_bytes <= ak.NOALLOC_MAX_WS_BYTES
        assert ap2.ws_bytes == ap.ws_bytes
        assert np.array_equal(got, want), f"case {k}: outputs differ"
        compare(got, oracle_out(b, hq, hkv, d), f"noalloc case {k}")


def test_noalloc_refuses_a_plan_larger_than_its_scratch():
    # checked on the host before any launch
    reqs, hq, hkv, d = [(1040, 1024)], 32, 8, 128
    b = build_batch(reqs, hq, hkv, d, seed=790)
    ap = ak.attention_plan(b["cu"], b["seq"], hq, hkv, d, 256)
    out = torch.empty_like(b["q"])
    with pytest.raises(ak.ArckvError) as e:
        ak.prefill_attention_noalloc(b["kp"], b["vp"], b["q"], out, torch.from_numpy(b["bt"]).to(DEV),
                                     torch.from_numpy(b["cu"]).to(DEV), torch.from_numpy(b["seq"]).to(DEV),
                                     torch.from_numpy(ap.work).to(DEV), ap.n_work, ap.n_combine, ap.tile_cols,
                                     d ** -0.5, ak.NOALLOC_MAX_WS_BYTES + 1)
    assert e.value.code == "ENOSPC"
