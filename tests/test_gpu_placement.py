"""GPU: conversation-level placement end to end on one MI355X (Section 4): admission against the
prefill latency curve, turn-1 prefill on a prefiller pool, the one-time transfer, binding to the
least occupied of three decoder pools, decoding there, and termination freeing the pages. The
binding decisions and every pool's occupancy must equal the oracle's simulation of the same
sequence (oracle/placement.py); attention outputs on the decoders must match the fp64 oracle.
"""
import numpy as np
import pytest
import torch

from oracle import placement as op
from oracle.attention import attend_last
from tests.helpers import assert_close, f64, kv_tokens, q_tokens

pytestmark = pytest.mark.gpu

SEED = 4242
HQ, HKV, D = 8, 2, 128


def test_placement_trace_matches_oracle():
    from paper_2606_01839_amd import KVPool, Scheduler
    rng = np.random.default_rng(SEED)
    caps = [96, 160, 128]                      # decoder pools of different capacity (pages)
    pre = KVPool(1, HQ, HKV, D, n_pages=256, max_convs=4, max_pages_per_conv=128, placement_seed=1)
    decs = [KVPool(1, HQ, HKV, D, n_pages=c, max_convs=16, max_pages_per_conv=128, placement_seed=10 + i)
            for i, c in enumerate(caps)]
    coef = (0.001, 2e-6, 1e-10)
    sched = Scheduler(coef, 0.004, decs)
    adm = op.Admission(coef, 0.004)
    used = [0] * len(decs)

    live = []          # (decoder index, handle, conv id, length)
    now, bound, refused = 0.0, [], 0
    for cid in range(14):
        now += float(rng.exponential(0.002))
        L = int(rng.integers(40, 700))
        got, want = sched.admit(L, now), adm.admit(L, now)
        assert got == want, (cid, got, want)
        if got is None:
            refused += 1
            continue
        # turn-1 prefill on the prefiller
        k, v = kv_tokens(SEED, cid, 1, 0, L, HKV, D)
        h = pre.conv_create()
        pre.kv_append(h, k.cuda(), v.cuda())
        q = q_tokens(SEED, cid, 0, 0, L, HQ, D)
        out = pre.attn_prefill_turn1([h], [L], 0, q.cuda())
        wire = pre.kv_pack(h)
        torch.cuda.synchronize()
        if cid % 4 == 0:
            assert_close(out, attend_last(f64(q), f64(k[0]), f64(v[0])), f"prefill conv {cid}")
        # bind and transfer
        d = sched.bind(L)
        free = [c - u for c, u in zip(caps, used)]
        assert d == op.bind(used, free, op.pages_for(L)), (cid, d, used)
        bound.append(d)
        if d < 0:
            pre.conv_destroy(h)
            continue
        hd = decs[d].kv_unpack(wire, L)
        pre.conv_destroy(h)
        used[d] += op.pages_for(L)
        live.append((d, hd, cid, L))
        # every third admission, the oldest live conversation ends (Section 4.2: occupancy drops)
        if cid % 3 == 2:
            d0, h0, _, L0 = live.pop(0)
            decs[d0].conv_destroy(h0)
            used[d0] -= op.pages_for(L0)
        for i, p in enumerate(decs):
            assert p.occupancy() == (used[i], caps[i] - used[i]), (cid, i)
    assert len(set(b for b in bound if b >= 0)) >= 2, bound     # load actually spread
    assert refused >= 1, "the saturation path was not exercised"

    # one decode step on every decoder for its live conversations, checked against the oracle
    for i, p in enumerate(decs):
        mine = [(h, cid, L) for d, h, cid, L in live if d == i]
        if not mine:
            continue
        qs = []
        for h, cid, L in mine:
            k, v = kv_tokens(SEED, cid, 1, L, 1, HKV, D)
            p.kv_append(h, k.cuda(), v.cuda())
            qs.append(q_tokens(SEED, cid, 0, L, 1, HQ, D))
        out = p.attn_decode_batch([h for h, _, _ in mine], 0, torch.cat(qs).cuda())
        torch.cuda.synchronize()
        for j, (h, cid, L) in enumerate(mine):
            k, v = kv_tokens(SEED, cid, 1, 0, L + 1, HKV, D)
            assert_close(out[j:j + 1], attend_last(f64(qs[j]), f64(k[0]), f64(v[0])), f"decode conv {cid}")
    sched.close()
    pre.close()
    for p in decs:
        p.close()
