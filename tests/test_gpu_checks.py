"""The device-checked build (lib/libarckv_checked.so, kernels compiled with
ARCKV_DEVICE_CHECKS) on the GPU: on valid inputs it records nothing and its results equal the
oracle's; out-of-range scatter slots, block-table entries and work items, which every build
clamps or skips without touching memory outside the pools, are recorded with their kind.
Nothing here makes a kernel fault: the indices are the ones the kernels' own bounds checks
already turn away."""

from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2606_21238_amd as ak  # noqa: E402
from paper_2606_21238_amd import _lib  # noqa: E402
from paper_2606_21238_amd.build import CHECKED_LIB  # noqa: E402
from tests.gpu_helpers import bits, compare, print_case  # noqa: E402
from tests.test_gpu_parity import build_batch, oracle_out, run_attention  # noqa: E402

DEV = "cuda"


@pytest.fixture()
def checked(monkeypatch):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ak.lib()                                      # the product build stays loaded as well
    chk = _lib.load(CHECKED_LIB)
    monkeypatch.setattr(_lib, "_lib", chk)        # the binding's calls go to the checked build
    ak.device_checks(reset=True)
    return chk


def test_valid_batch_records_nothing(checked):
    print_case("checked build: valid scatter + attention (two split regimes)")
    reqs, hq, hkv, d = [(1040, 1024), (300, 16), (77, 0)], 32, 8, 128
    b = build_batch(reqs, hq, hkv, d, seed=71)            # scatter through the checked build
    ref = oracle_out(b, hq, hkv, d)
    for num_cus in (256, 100000):
        got, _ = run_attention(b, hq, hkv, d, num_cus)
        compare(got, ref, f"checked build, num_cus={num_cus}")
    assert ak.device_checks() == (0, 0)


def test_out_of_range_slots_are_recorded_and_skipped(checked):
    print_case("checked build: scatter with 4 slots outside the pool")
    nb, hkv, d, n = 6, 2, 64, 40
    g = torch.Generator(device=DEV).manual_seed(5)
    k_new = (torch.randn((n, hkv, d), generator=g, device=DEV)).to(torch.bfloat16)
    v_new = (torch.randn((n, hkv, d), generator=g, device=DEV)).to(torch.bfloat16)
    slots = np.arange(n, dtype=np.int32) + 8
    bad = [3, 17, 18, 39]
    slots[bad] = [16 * nb, 16 * nb + 100, -2, 1 << 30]
    kp = torch.full((nb, hkv, 16, d), -1, dtype=torch.int16, device=DEV)
    vp = torch.full((nb, hkv, d, 16), -1, dtype=torch.int16, device=DEV)
    ak.kv_scatter(kp, vp, k_new, v_new, torch.from_numpy(slots).to(DEV))
    torch.cuda.synchronize()
    kind, count = ak.device_checks()
    assert kind == _lib.CHECK_SLOT and count >= len(bad)
    # the valid tokens landed, the rest of the pool is untouched
    kb, vb = bits(kp), bits(vp)
    kn, vn = bits(k_new), bits(v_new)
    good = [t for t in range(n) if t not in bad]
    for t in good:
        s = int(slots[t])
        assert (kb[s // 16, :, s % 16, :] == kn[t]).all()
        assert (vb[s // 16, :, :, s % 16] == vn[t]).all()
    written = {int(slots[t]) for t in good}
    for s in range(16 * nb):
        if s not in written:
            assert (kb[s // 16, :, s % 16, :] == 0xFFFF).all() and (vb[s // 16, :, :, s % 16] == 0xFFFF).all()
    assert ak.device_checks() == (0, 0)                   # cleared by the read before


def test_out_of_range_block_entries_are_recorded(checked):
    print_case("checked build: attention with one block-table entry outside the pool")
    reqs, hq, hkv, d = [(640, 600), (200, 0)], 8, 2, 128
    b = build_batch(reqs, hq, hkv, d, seed=73)
    ak.device_checks(reset=True)
    ref = oracle_out(b, hq, hkv, d)
    nphys = int(b["kp"].shape[0])
    bt = b["bt"].copy()
    bt[0, 5] = nphys + 5                                   # a block of request 0's range
    got, _ = run_attention(b, hq, hkv, d, table_override=bt)
    kind, count = ak.device_checks()
    assert kind == _lib.CHECK_BLOCK and count >= 1
    # request 1 does not read the entry: its rows still equal the oracle's
    r1 = slice(int(b["cu"][1]), int(b["cu"][2]))
    compare(got[r1], ref[r1], "request 1 beside a bad entry of request 0")


def test_malformed_work_items_are_recorded(checked):
    print_case("checked build: attention plan with a work item naming no request")
    reqs, hq, hkv, d = [(300, 200)], 8, 2, 64
    b = build_batch(reqs, hq, hkv, d, seed=79)
    ap = ak.attention_plan(b["cu"], b["seq"], hq, hkv, d)
    bogus = np.array([[5, 0, 0, 0, 64, -1, 0, 0]], dtype=np.int32)      # request 5 of a 1-request batch
    work = np.ascontiguousarray(np.concatenate([ap.work[: ap.n_work], bogus, ap.work[ap.n_work:]]), dtype=np.int32)
    out = torch.empty_like(b["q"])
    ws = torch.zeros(max(ap.ws_bytes, 1), dtype=torch.uint8, device=DEV)
    ak.prefill_attention(b["kp"], b["vp"], b["q"], out, torch.from_numpy(b["bt"]).to(DEV),
                         torch.from_numpy(b["cu"]).to(DEV), torch.from_numpy(b["seq"]).to(DEV),
                         torch.from_numpy(work).to(DEV), ap.n_work + 1, ap.n_combine, ap.tile_cols,
                         d ** -0.5, ws, ap.ws_bytes)
    torch.cuda.synchronize()
    kind, _ = ak.device_checks()
    assert kind == _lib.CHECK_WORK
    compare(bits(out), oracle_out(b, hq, hkv, d), "the valid items' output")


def test_malformed_list_entries_are_skipped_and_recorded(checked):
    print_case("checked build: narrow list plan with an entry naming no request")
    reqs, hq, hkv, d = [(300, 290), (500, 480), (2000, 1990)], 8, 2, 128    # <= 80 columns: lists
    b = build_batch(reqs, hq, hkv, d, seed=83)
    ap = ak.attention_plan(b["cu"], b["seq"], hq, hkv, d)
    assert ap.tile_cols == 128
    work = ap.work.copy()
    lists = work[: ap.n_work].reshape(-1, 8, 8)
    n_live = (lists[:, :, 0] >= 0).sum(axis=1)
    k = int(np.argmax(n_live < 8))
    assert n_live[k] < 8
    lst = lists[k]
    lst[1: n_live[k] + 1] = lst[: n_live[k]].copy()          # the bogus entry goes first:
    lst[0] = [7, 0, 0, 0, 64, -1, 0, 0]                       # the list's items follow it
    out = torch.empty_like(b["q"])
    ws = torch.zeros(max(ap.ws_bytes, 1), dtype=torch.uint8, device=DEV)
    ak.prefill_attention(b["kp"], b["vp"], b["q"], out, torch.from_numpy(b["bt"]).to(DEV),
                         torch.from_numpy(b["cu"]).to(DEV), torch.from_numpy(b["seq"]).to(DEV),
                         torch.from_numpy(np.ascontiguousarray(work)).to(DEV), ap.n_work, ap.n_combine,
                         ap.tile_cols, d ** -0.5, ws, ap.ws_bytes)
    torch.cuda.synchronize()
    kind, _ = ak.device_checks()
    assert kind == _lib.CHECK_WORK
    compare(bits(out), oracle_out(b, hq, hkv, d), "the list's valid items")
