"""GPU: the mixed agentic step (extend chunks + single-token decodes batched across
conversations, every layer) against the fp64 oracle, on a scaled-down agentic trace with the
Llama-3-8B attention shape (32q/8kv heads, d 128) and two layers."""
import numpy as np
import pytest
import torch

from oracle.attention import attend_last
from synth import values as sv
from synth.traces import KIND_K, KIND_Q, KIND_V
from tests.helpers import assert_close

pytestmark = pytest.mark.gpu

SEED = 5151
HQ, HKV, D, NL = 32, 8, 128, 2


def _kv(conv, layer, start, n, device="cpu"):
    per = HKV * D
    k = sv.bf16_tensor(sv.mix_key(SEED, conv, KIND_K, layer), (n, HKV, D), start=start * per, device=device)
    v = sv.bf16_tensor(sv.mix_key(SEED, conv, KIND_V, layer), (n, HKV, D), start=start * per, device=device)
    return k, v


def _q(conv, layer, start, n, device="cpu"):
    return sv.bf16_tensor(sv.mix_key(SEED, conv, KIND_Q, layer), (n, HQ, D), start=start * HQ * D,
                          device=device)


def test_mixed_steps_match_oracle():
    from paper_2606_01839_amd import KVPool
    pool = KVPool(NL, HQ, HKV, D, n_pages=800, max_convs=8, max_pages_per_conv=256, placement_seed=9)
    # five conversations with different turn-1 contexts (filled by append, untimed here)
    lens0 = [700, 1, 64, 1500, 333]
    convs = []
    for c, L in enumerate(lens0):
        h = pool.conv_create()
        k = torch.stack([_kv(c, l, 0, L)[0] for l in range(NL)]).cuda()
        v = torch.stack([_kv(c, l, 0, L)[1] for l in range(NL)]).cuda()
        pool.kv_append(h, k, v)
        convs.append(h)
    lens = list(lens0)
    # three steps with different extend/decode splits (ragged chunks)
    plans = [([0, 3], [40, 129], [1, 2, 4]), ([1], [64], [0, 2, 3, 4]), ([2, 4, 0], [1, 17, 200], [1, 3])]
    for ext, ext_n, dec in plans:
        new = [(c, n) for c, n in zip(ext, ext_n)] + [(c, 1) for c in dec]
        ks = [torch.stack([_kv(c, l, lens[c], n)[0] for l in range(NL)]) for c, n in new]
        vs = [torch.stack([_kv(c, l, lens[c], n)[1] for l in range(NL)]) for c, n in new]
        k = torch.cat(ks, 1).contiguous().cuda()
        v = torch.cat(vs, 1).contiguous().cuda()
        qe = torch.stack([torch.cat([_q(c, l, lens[c], n) for c, n in zip(ext, ext_n)]) for l in range(NL)])
        qd = torch.stack([torch.cat([_q(c, l, lens[c], 1) for c in dec]) for l in range(NL)])
        oe, od = pool.mixed_step([convs[c] for c in ext], ext_n, [convs[c] for c in dec], k, v,
                                 qe.contiguous().cuda(), qd.contiguous().cuda())
        torch.cuda.synchronize()
        for c, n in new:
            lens[c] += n
        for layer in range(NL):
            row = 0
            for c, n in zip(ext, ext_n):
                kk, vv = _kv(c, layer, 0, lens[c])
                ref = attend_last(sv.bf16_to_f64(qe[layer, row:row + n]), sv.bf16_to_f64(kk), sv.bf16_to_f64(vv))
                assert_close(oe[layer, row:row + n], ref, f"extend conv {c} layer {layer}")
                row += n
            for i, c in enumerate(dec):
                kk, vv = _kv(c, layer, 0, lens[c])
                ref = attend_last(sv.bf16_to_f64(qd[layer, i:i + 1]), sv.bf16_to_f64(kk), sv.bf16_to_f64(vv))
                assert_close(od[layer, i:i + 1], ref, f"decode conv {c} layer {layer}")
    for c, h in enumerate(convs):
        assert pool.conv_len(h) == lens[c]
    pool.close()


def test_mixed_step_rejects_overlap_without_changes():
    from paper_2606_01839_amd import KVPool, ConserveError, CS_EINVAL
    pool = KVPool(NL, HQ, HKV, D, n_pages=64, max_convs=4, max_pages_per_conv=64, placement_seed=1)
    a = pool.conv_create()
    k, v = _kv(0, 0, 0, 10, "cuda")
    pool.kv_append(a, torch.stack([k, k]), torch.stack([v, v]))
    kk = torch.zeros(NL, 6, HKV, D, dtype=torch.bfloat16, device="cuda")
    qe = torch.zeros(NL, 5, HQ, D, dtype=torch.bfloat16, device="cuda")
    qd = torch.zeros(NL, 1, HQ, D, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ConserveError) as e:
        pool.mixed_step([a], [5], [a], kk, kk, qe, qd)      # same conversation twice
    assert e.value.code == CS_EINVAL
    assert pool.conv_len(a) == 10 and pool.occupancy()[0] == 1
    pool.close()
