"""GPU: the config-5 serving loop of bench.py (admission through cs_sched_admit / cs_sched_bind on
the decoder's current occupancy, swap-out to host memory and swap-in when a step's tokens do not
fit, destruction at the end of the last turn) run to completion on a small agentic trace whose
decoder pool is too small to hold every conversation at once: every conversation completes, some
are swapped out and back in, the pool is empty at the end, and the sampled outputs match the oracle.
"""
import argparse

import pytest

from synth.traces import MixedTrace, Shape, pages_for

pytestmark = pytest.mark.gpu


def _trace():
    return MixedTrace(seed=77, shape=Shape(n_layers=2, n_q_heads=8, n_kv_heads=2, head_dim=128), n_convs=10,
                      turns_lo=2, turns_hi=4, turn1_median=400, turn1_lo=64, turn1_hi=1500,
                      append_median=200, append_lo=16, append_hi=800, decode_median=12, decode_lo=1,
                      decode_hi=40)


@pytest.mark.parametrize("collocated", [False, True])
def test_small_trace_served_to_completion(collocated):
    import bench
    tr = _trace()
    finals = [c.final_len() for c in tr.conversations()]
    pool = int(1.4 * pages_for(max(finals)))      # holds the longest conversation, not all of them
    assert pool < sum(pages_for(f) for f in finals) // 2
    args = argparse.Namespace(mixed_steps=0, mixed_to_completion=True, mixed_max_s=300,
                              mixed_check_every=15)
    print(f"serving loop: {tr.n_convs} conversations, pool {pool} pages, collocated={collocated}", flush=True)
    res = bench.bench_mixed(args, collocated=collocated, trace_cfg=tr, pool_pages=pool)
    out = res["mixed_collocated" if collocated else "mixed_to_completion"]
    print(out, flush=True)
    assert out["completed"] == tr.n_convs and out["admitted"] == tr.n_convs
    if not collocated:
        assert not out["stopped_early"] and out["live_end"] == 0 and out["waiting_end"] == 0
        assert out["swapped_out"] > 0 and out["swapped_in"] == out["swapped_out"]
        assert out["occupancy_end"]["used_pages"] == 0
        assert out["parity_samples"] and out["parity_ok"]
    else:
        assert all(v["ok"] for v in out["spot_parity"].values())
