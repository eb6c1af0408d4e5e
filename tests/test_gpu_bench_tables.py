"""Full-size GPU parity of every window table bench.py times, at the size and in the
launch configuration it is timed in (parity.BENCH_TABLE_TESTS lists them all; the
entries checked elsewhere name their test there).

Prefill: a stratified sample of at least 256 (row, head) pairs over all query heads
(workloads.stratified_rows: the first and last 64 positions, the first and last
position of workgroup position tiles, both sides of the seams between 32-row MFMA
blocks, positions whose first kept key of a pair sits at a 32- or 64-key edge, and
seeded random rows), recomputed one by one by the oracle.  Decode: every (batch,
head) row.  Tolerances: O max-abs 1e-2, O mean-abs 1e-3, LSE 1e-3."""
import pytest
import torch

from conftest import gpu_available
import oracle
import workloads as W
from parity import (bench_rows, bench_tables_of, compare, gpu_decode, gpu_prefill, note,
                    pack_kcache, pack_vcache, table_windows, to_f64)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]

DEV = "cuda"
PREFILL_TABLES = bench_tables_of("prefill")
DECODE_TABLES = bench_tables_of("decode")


@pytest.mark.parametrize("name", sorted(PREFILL_TABLES))
def test_prefill_bench_tables_sampled_rows(name):
    wl = W.WORKLOADS[name]
    note(f"generate {name}")
    inp = W.make_inputs(wl, device=DEV)
    kp, vp = pack_kcache(inp["k"]), pack_vcache(inp["v"])
    host = (inp["q"].cpu(), inp["k"].cpu(), inp["v"].cpu())
    del inp["k"], inp["v"]
    failures = []
    for tag in PREFILL_TABLES[name]:
        win, widths, atom = table_windows(wl, tag)
        rows = bench_rows(wl, widths)
        assert len(rows) >= 256 and set(rows[:, 1].tolist()) == set(range(wl.h_q))
        note(f"prefill {name} {tag}: {len(rows)} sampled rows")
        o, lse = gpu_prefill(inp["q"], None, None, wl.q_pos0, win, kp=kp, vp=vp)
        idx = torch.from_numpy(rows).to(DEV)
        og = to_f64(o[idx[:, 0], idx[:, 2], idx[:, 1]])
        lg = to_f64(lse[idx[:, 0], idx[:, 1], idx[:, 2]])
        if tag == "default":
            # determinism: a second launch is bit-identical
            o2, lse2 = gpu_prefill(inp["q"], None, None, wl.q_pos0, win, kp=kp, vp=vp)
            assert torch.equal(o, o2) and torch.equal(lse, lse2), f"{name}: not deterministic"
            del o2, lse2
        del o, lse
        o_ref, lse_ref, _ = oracle.attend(*host, wl.q_pos0, widths, rows=rows, atom=atom)
        try:
            mx, mean, ml = compare(og, lg, o_ref, lse_ref, f"{name} {tag}")
            print(f"[parity] {name} {tag}: O max {mx:.2e} mean {mean:.2e} LSE {ml:.2e}",
                  flush=True)
        except AssertionError as e:
            failures.append(str(e))
    assert not failures, failures


@pytest.mark.parametrize("name", sorted(DECODE_TABLES))
def test_decode_bench_tables_all_rows(name):
    wl = W.WORKLOADS[name]
    note(f"generate {name}")
    inp = W.make_inputs(wl, device=DEV)
    kp, vp = pack_kcache(inp["k"]), pack_vcache(inp["v"])
    host = (inp["q"].cpu(), inp["k"].cpu(), inp["v"].cpu())
    qd = inp["q"][:, 0].contiguous()
    del inp
    failures = []
    for tag in DECODE_TABLES[name]:
        win, widths, atom = table_windows(wl, tag)
        note(f"decode {name} {tag}")
        o, lse = gpu_decode(qd, None, None, wl.q_pos0, win, kp=kp, vp=vp)
        o_ref, lse_ref, _ = oracle.attend(*host, wl.q_pos0, widths, atom=atom)
        try:
            mx, mean, ml = compare(to_f64(o), to_f64(lse), o_ref[:, 0], lse_ref[:, :, 0],
                                   f"{name} {tag}")
            print(f"[parity] {name} {tag}: O max {mx:.2e} mean {mean:.2e} LSE {ml:.2e}",
                  flush=True)
        except AssertionError as e:
            failures.append(str(e))
    assert not failures, failures
