"""The byte/FLOP model used for roofline figures, pinned to the paper's
Table 1 (decode self-attention cost, Llama2-7B shapes, 2048 context tokens)
and to closed forms of the workload trees."""
import pytest

from oracle import OracleTree, tables
from paper_2402_15220_amd.roofline import call_model, table1_self_attention
from workloads import make_static


@pytest.mark.parametrize("b,flops,mops", [
    (1, 33.57e6, 33.85e6), (32, 1074.27e6, 1083.18e6), (64, 2148.53e6, 2166.36e6)])
def test_table1_self_attention_cost(b, flops, mops):
    f, m = table1_self_attention(b, 2048, 32, 128, 2)
    assert abs(f - flops) / flops < 0.002
    assert abs(m - mops) / mops < 0.01


@pytest.mark.parametrize("cfg,total,flops", [
    (2, 285_736_960, 805_306_368), (3, 336_068_608, 2_415_919_104), (4, 370_147_328, 2_415_919_104)])
def test_workload_bytes_closed_form(cfg, total, flops):
    wl = make_static(cfg)
    t = OracleTree(c=wl.c, with_kv=False)
    for s in wl.seqs:
        t.insert(s.seq_id, s.tokens(wl.segments))
    m = call_model(tables(t).as_dict(), wl.H, wl.d, 2)
    assert m["total"] == total
    assert m["flops"] == flops
    assert m["private_kv"] == 268_435_456
