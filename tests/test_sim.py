"""CPU: the host simulator of conversation-level serving (paper_2606_01839_amd/sim.py).

* Three hand-derived scenarios pin its event logic: admission with a refusal and a retry, the
  prefiller's queue, tool time between turns, iterations that batch a late joiner, the binding of
  conversations to the least occupied decoder, and preemption when the KV pages run out.
* On the synthetic agentic trace, timed with the measured MI355X rates of this library's kernels,
  it shows the paper's two phases qualitatively (Section 3.1, Section 3.2 and its collocation
  experiment): turn-1 TTFT grows quadratically with the prompt, later turns' TTFT stays small and
  nearly flat, and the more KV a decoder has active, the more often its iterations are set by the
  decode rather than the collocated extend work.
"""
import math

import numpy as np
import pytest

from paper_2606_01839_amd.sim import ConvSpec, CostModel, Simulator
from synth.traces import MixedTrace

INF = math.inf
# 1 layer; prefill t(L) = 1e-6 L^2 s; every decode iteration 0.1 s, every extend part 0.05 s;
# transfers and copies instantaneous
TOY = CostModel(n_layers=1, prefill_curve=(0.0, 0.0, 1e-6), decode_fixed_s=0.1, decode_gbs=INF,
                extend_fixed_s=0.05, extend_tflops=INF, move_gbs=INF, link_gbs=INF, host_gbs=INF)


def test_hand_scenario_admission_tool_time_and_batching():
    """One decoder, max wait 2 s, tool time 0.3 s. Derived by hand:
    A (t=0, 1000 tokens, decodes [2, 1], append [100]): prefill [0, 1] -> TTFT 1.0; decodes in
      [1.0, 1.1], [1.1, 1.2]; tool until 1.5; its append runs alone in [1.5, 1.55] (extend part
      only) -> turn-2 TTFT 0.05; one decode [1.55, 1.65] -> done at 1.65.
    B (t=0.5, 2000 tokens, decodes [4]): waits 0.5 s for A's prefill: [1, 5] -> TTFT 4.5; decodes
      [5.0, 5.1], [5.1, 5.2], [5.2, 5.3], [5.3, 5.4] -> done at 5.4.
    C (t=1.2, 500 tokens, decodes [2]): expected wait 5 - 1.2 = 3.8 > 2 -> refused; retried when B's
      prefill ends at 5.0 (wait 0): prefill [5.0, 5.25] -> TTFT 4.05; joins at the next iteration
      boundary 5.3, so [5.3, 5.4] decodes B and C together, then [5.4, 5.5] -> done at 5.5.
    Nine iterations, one refusal, makespan 5.5 s."""
    trace = [ConvSpec(1000, [100], [2, 1], 0.0), ConvSpec(2000, [], [4], 0.5), ConvSpec(500, [], [2], 1.2)]
    sim = Simulator(trace, TOY, n_decoders=1, pages_per_decoder=10_000, max_wait_s=2.0, tool_s=0.3)
    r = sim.run()
    assert r["completed"] == 3 and r["refusals"] == 1 and r["swaps"] == 0
    assert [t for _, t in r["turn1_ttft"]] == pytest.approx([1.0, 4.5, 4.05])
    assert [t for _, _, t in r["later_ttft"]] == pytest.approx([0.05])
    assert r["later_ttft"][0][:2] == (1002, 100)            # context before the append: 1000 + 2
    assert r["finish"] == pytest.approx([1.65, 5.4, 5.5])
    assert r["iterations"] == 9 and r["makespan_s"] == pytest.approx(5.5)
    starts = [round(i.start, 6) for i in sim.iterations]
    assert starts == pytest.approx([1.0, 1.1, 1.5, 1.55, 5.0, 5.1, 5.2, 5.3, 5.4])
    assert [i.n_decode for i in sim.iterations] == [1, 1, 0, 1, 1, 1, 1, 2, 1]


def test_hand_scenario_binding_least_occupied():
    """Two decoders of 100 pages, no waiting limit. Prefills run back to back: A (800 tokens =
    50 pages) [0, 0.64], B (160 = 10 pages) [0.64, 0.6656], C (320 = 20 pages) [0.6656, 0.768].
    A binds to decoder 0 (both empty: the lower index); B finds 51/100 against 0/100 pages used and
    binds to decoder 1; B's single decode ends at 0.7656 and frees decoder 1, so C (at 0.768, 51
    against 0 pages used) binds to decoder 1 as well."""
    trace = [ConvSpec(800, [], [10], 0.0), ConvSpec(160, [], [1], 0.0), ConvSpec(320, [], [1], 0.0)]
    sim = Simulator(trace, TOY, n_decoders=2, pages_per_decoder=100, max_wait_s=100.0)
    r = sim.run()
    assert r["completed"] == 3
    assert [c.decoder for c in sim.convs] == [0, 1, 1]
    assert [t for _, t in r["turn1_ttft"]] == pytest.approx([0.64, 0.6656, 0.768])
    assert sim.used == [0, 0]                                # every page returned at the end


def test_hand_scenario_preemption_when_pages_run_out():
    """One decoder of 30 pages; A and B (160 tokens = 10 pages each) each decode 200 tokens, so
    together they would need 46 pages. When B's growth no longer fits, B (the later bound) is
    swapped out, A finishes alone (23 pages), and B comes back and finishes."""
    trace = [ConvSpec(160, [], [200], 0.0), ConvSpec(160, [], [200], 0.0)]
    sim = Simulator(trace, TOY, n_decoders=1, pages_per_decoder=30, max_wait_s=100.0)
    r = sim.run()
    assert r["completed"] == 2 and r["swaps"] >= 1
    a, b = sim.convs
    assert a.swaps == 0 and b.swaps >= 1 and a.finish < b.finish
    assert sim.used == [0]


def _trace(n, rate, seed=7):
    convs = MixedTrace().conversations()[:n]
    arr = np.cumsum(np.random.default_rng(seed).exponential(1.0 / rate, size=n))
    return [ConvSpec(c.turn1, c.appends, c.decodes, float(a)) for c, a in zip(convs, arr)]


def test_two_phases_on_the_agentic_trace():
    # light load: no queueing, so turn-1 TTFT is the prefill itself
    sim = Simulator(_trace(96, 0.05), CostModel(), n_decoders=2, pages_per_decoder=116_000,
                    max_wait_s=30.0, tool_s=2.0)
    r = sim.run()
    assert r["completed"] == 96 and r["swaps"] == 0
    L = np.array([x[0] for x in r["turn1_ttft"]], dtype=float)
    T = np.array([x[1] for x in r["turn1_ttft"]])
    c = np.polyfit(L, T, 2)
    r2 = 1 - ((T - np.polyval(c, L)) ** 2).sum() / ((T - T.mean()) ** 2).sum()
    assert r2 > 0.99 and c[0] > 0
    assert np.polyval(c, 65536) / np.polyval(c, 8192) > 30      # quadratic, not linear (8x)
    later = np.array([t for _, _, t in r["later_ttft"]])
    assert np.percentile(later, 95) < 0.25 * np.percentile(T, 95)
    # heavy load: the decode share of collocated iterations grows with the decoder's active KV
    sim = Simulator(_trace(256, 1.0), CostModel(), n_decoders=2, pages_per_decoder=116_000,
                    max_wait_s=30.0, tool_s=2.0)
    r = sim.run()
    assert r["completed"] == 256
    bins = [b for b in sim.decode_dominance([0, 131072, 262144, 524288, 1048576, 1 << 40]) if b[2] >= 50]
    shares = [b[3] for b in bins]
    assert len(shares) >= 3 and shares == sorted(shares) and shares[-1] > 0.6 and shares[0] < 0.2
