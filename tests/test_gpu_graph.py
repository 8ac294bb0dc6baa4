"""Graph capture of the attention path, on the GPU: arckv_prefill_attention_noalloc (the entry
point that allocates nothing, meant for code under capture) recorded into one HIP graph through
torch.cuda.graph and replayed several times, with eager work and synchronisations between the
replays.  Every replay must equal the eager result bitwise, and the oracle within the attention
tolerance.  The plans split key ranges, so the captured launch sequence is attention plus the
split combine, both reading the static scratch.
"""

from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import paper_2606_21238_amd as ak  # noqa: E402
from tests.gpu_helpers import bits, compare, print_case  # noqa: E402
from tests.test_gpu_parity import DEV, build_batch, oracle_out, run_attention  # noqa: E402


@pytest.mark.parametrize("reqs,hq,hkv,d", [
    ([(L, L - 1) for L in (300, 4097, 2000, 65, 1500, 777, 9000, 33)], 32, 8, 128),  # lists
    ([(1040, 1024), (600, 500), (3000, 2900)], 32, 8, 128),                           # wide tiles
])
def test_captured_attention_replays_equal_the_eager_call(reqs, hq, hkv, d):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print_case(f"graph capture: {reqs} hq={hq} hkv={hkv} d={d}")
    b = build_batch(reqs, hq, hkv, d, seed=810 + len(reqs))
    want, ap = run_attention(b, hq, hkv, d, 256)
    assert ap.n_combine > 0 and ap.ws_bytes <= ak.NOALLOC_MAX_WS_BYTES
    bt = torch.from_numpy(b["bt"]).to(DEV)
    cu = torch.from_numpy(b["cu"]).to(DEV)
    seq = torch.from_numpy(b["seq"]).to(DEV)
    work = torch.from_numpy(ap.work).to(DEV)
    out = torch.full_like(b["q"], float("nan"))

    def call():
        ak.prefill_attention_noalloc(b["kp"], b["vp"], b["q"], out, bt, cu, seq, work, ap.n_work,
                                     ap.n_combine, ap.tile_cols, d ** -0.5, ap.ws_bytes)

    # the first call on this device finds the static scratch's address: outside the capture
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    assert np.array_equal(bits(out), want)

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    torch.cuda.synchronize()
    for k in range(3):
        out.fill_(float("nan"))                  # eager work between replays
        junk = torch.randn(1 << 20, device=DEV).sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = bits(out)
        assert np.array_equal(got, want), f"replay {k} differs from the eager call"
        assert torch.isfinite(junk)
    compare(got, oracle_out(b, hq, hkv, d), "graph replay")
