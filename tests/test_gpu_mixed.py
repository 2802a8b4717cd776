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


def _kv(conv, layer, start, n, device="cpu", hkv=HKV, d=D):
    per = hkv * d
    k = sv.bf16_tensor(sv.mix_key(SEED, conv, KIND_K, layer), (n, hkv, d), start=start * per, device=device)
    v = sv.bf16_tensor(sv.mix_key(SEED, conv, KIND_V, layer), (n, hkv, d), start=start * per, device=device)
    return k, v


def _q(conv, layer, start, n, device="cpu", hq=HQ, d=D):
    return sv.bf16_tensor(sv.mix_key(SEED, conv, KIND_Q, layer), (n, hq, d), start=start * hq * d,
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


@pytest.mark.parametrize("shape", [(HQ, HKV, D), (4, 2, 64)], ids=["32q8kv_d128", "4q2kv_d64"])
@pytest.mark.parametrize("layer_ordered", [False, True])
@pytest.mark.parametrize("n_layers", [1, 3, 4])
def test_mixed_step_bitwise_equals_per_layer_calls(n_layers, layer_ordered, shape):
    """The mixed step gives bit for bit the outputs of the separate calls (kv_append_batch, then
    attn_extend and attn_decode_batch layer by layer, on a second pool with the same placement),
    both with all layers overlapped (one launch per layer that merges layer l-1 and splits layer l,
    alternating two partial buffers) and in layer order (at d 64 the fork/join form). Decode-only
    and extend-only steps included; the last layer's decode outputs are checked against the oracle."""
    from paper_2606_01839_amd import KVPool
    hq, hkv, d = shape
    mk = lambda: KVPool(n_layers, hq, hkv, d, n_pages=900, max_convs=8, max_pages_per_conv=256,
                        placement_seed=77)
    pa, pb = mk(), mk()
    lens0 = [1200, 5, 417, 2049, 96, 800]
    ha, hb, lens = [], [], list(lens0)

    def kv_rows(items):
        ks = [torch.stack([_kv(c, l, s, n, hkv=hkv, d=d)[0] for l in range(n_layers)]) for c, s, n in items]
        vs = [torch.stack([_kv(c, l, s, n, hkv=hkv, d=d)[1] for l in range(n_layers)]) for c, s, n in items]
        return torch.cat(ks, 1).contiguous().cuda(), torch.cat(vs, 1).contiguous().cuda()

    for c, L in enumerate(lens0):
        k, v = kv_rows([(c, 0, L)])
        for pool, hs in ((pa, ha), (pb, hb)):
            h = pool.conv_create()
            pool.kv_append(h, k, v)
            hs.append(h)
    plans = [([0, 4], [300, 33], [1, 2, 3, 5]), ([], [], [0, 1, 2, 3, 4, 5]), ([1, 3], [64, 2], [])]
    for ext, ext_n, dec in plans:
        items = [(c, lens[c], n) for c, n in zip(ext, ext_n)] + [(c, lens[c], 1) for c in dec]
        k, v = kv_rows(items)
        qe = (torch.stack([torch.cat([_q(c, l, lens[c], n, hq=hq, d=d) for c, n in zip(ext, ext_n)])
                           for l in range(n_layers)]).contiguous().cuda() if ext else None)
        qd = (torch.stack([torch.cat([_q(c, l, lens[c], 1, hq=hq, d=d) for c in dec])
                           for l in range(n_layers)]).contiguous().cuda() if dec else None)
        oe, od = pa.mixed_step([ha[c] for c in ext], ext_n, [ha[c] for c in dec], k, v, qe, qd,
                              layer_ordered=layer_ordered)
        pb.kv_append_batch([hb[c] for c, _, _ in items], [n for _, _, n in items], k, v)
        for layer in range(n_layers):
            if ext:
                ref_e = pb.attn_extend([hb[c] for c in ext], ext_n, layer, qe[layer])
                assert torch.equal(oe[layer], ref_e), f"extend layer {layer} of plan {ext}/{dec}"
            if dec:
                ref_d = pb.attn_decode_batch([hb[c] for c in dec], layer, qd[layer])
                assert torch.equal(od[layer], ref_d), f"decode layer {layer} of plan {ext}/{dec}"
        torch.cuda.synchronize()
        for c, s, n in items:
            lens[c] = s + n
        if dec:
            layer = n_layers - 1
            for i, c in enumerate(dec):
                kk, vv = _kv(c, layer, 0, lens[c], hkv=hkv, d=d)
                ref = attend_last(sv.bf16_to_f64(qd[layer, i:i + 1]), sv.bf16_to_f64(kk), sv.bf16_to_f64(vv))
                assert_close(od[layer, i:i + 1], ref, f"decode conv {c} layer {layer}")
    for c in range(len(lens0)):
        assert pa.conv_len(ha[c]) == pb.conv_len(hb[c]) == lens[c]
    assert pa.occupancy() == pb.occupancy()
    pa.close()
    pb.close()


def test_single_item_decode_direct_output_equals_merge_path():
    """A decode batch whose conversations are one work item each (at most 8 splits of 128 keys)
    has the split kernel write the output directly; add one long conversation (two items, same
    128-key splits) and the whole batch goes through partial records and the merge kernel. The
    short conversations' outputs must be the same bits both ways, and match the oracle."""
    from paper_2606_01839_amd import KVPool
    lens = [1, 17, 300, 777, 1000]
    long_len = 1500
    mk = lambda: KVPool(1, HQ, HKV, D, n_pages=512, max_convs=8, max_pages_per_conv=128, placement_seed=5)
    pa, pb = mk(), mk()
    ha, hb = [], []
    for c, L in enumerate(lens + [long_len]):
        k, v = _kv(c, 0, 0, L, "cuda")
        for pool, hs in ((pa, ha), (pb, hb)):
            if pool is pa and c == len(lens):
                continue
            h = pool.conv_create()
            pool.kv_append(h, k[None], v[None])
            hs.append(h)
    q = torch.cat([_q(c, 0, L - 1, 1) for c, L in enumerate(lens + [long_len])]).contiguous().cuda()
    direct = pa.attn_decode_batch(ha, 0, q[:len(lens)])
    merged = pb.attn_decode_batch(hb, 0, q)
    torch.cuda.synchronize()
    assert torch.equal(direct, merged[:len(lens)])
    for c, L in enumerate(lens):
        kk, vv = _kv(c, 0, 0, L)
        ref = attend_last(sv.bf16_to_f64(q[c:c + 1]), sv.bf16_to_f64(kk), sv.bf16_to_f64(vv))
        assert_close(direct[c:c + 1], ref, f"decode conv {c}")
    pa.close()
    pb.close()


@pytest.mark.parametrize("layer_ordered", [False, True])
def test_mixed_step_single_item_decode_all_layers(layer_ordered):
    """Short conversations only (one decode work item each): every layer's decode output comes
    straight from its split launch, in both orders, with and without extend chunks in the step.
    Outputs equal the per-layer calls bit for bit and match the oracle."""
    from paper_2606_01839_amd import KVPool
    nl = 3
    mk = lambda: KVPool(nl, HQ, HKV, D, n_pages=256, max_convs=8, max_pages_per_conv=64, placement_seed=21)
    pa, pb = mk(), mk()
    lens = [3, 40, 250, 600]
    ha, hb = [], []
    for c, L in enumerate(lens):
        k = torch.stack([_kv(c, l, 0, L)[0] for l in range(nl)]).cuda()
        v = torch.stack([_kv(c, l, 0, L)[1] for l in range(nl)]).cuda()
        for pool, hs in ((pa, ha), (pb, hb)):
            h = pool.conv_create()
            pool.kv_append(h, k, v)
            hs.append(h)
    for ext, ext_n, dec in (([], [], [0, 1, 2, 3]), ([3], [20], [0, 1, 2])):
        items = [(c, lens[c], n) for c, n in zip(ext, ext_n)] + [(c, lens[c], 1) for c in dec]
        k = torch.cat([torch.stack([_kv(c, l, s, n)[0] for l in range(nl)]) for c, s, n in items], 1)
        v = torch.cat([torch.stack([_kv(c, l, s, n)[1] for l in range(nl)]) for c, s, n in items], 1)
        k, v = k.contiguous().cuda(), v.contiguous().cuda()
        qe = (torch.stack([torch.cat([_q(c, l, lens[c], n) for c, n in zip(ext, ext_n)]) for l in range(nl)])
              .contiguous().cuda() if ext else None)
        qd = torch.stack([torch.cat([_q(c, l, lens[c], 1) for c in dec]) for l in range(nl)]).contiguous().cuda()
        oe, od = pa.mixed_step([ha[c] for c in ext], ext_n, [ha[c] for c in dec], k, v, qe, qd,
                               layer_ordered=layer_ordered)
        pb.kv_append_batch([hb[c] for c, _, _ in items], [n for _, _, n in items], k, v)
        for layer in range(nl):
            assert torch.equal(od[layer], pb.attn_decode_batch([hb[c] for c in dec], layer, qd[layer]))
            if ext:
                assert torch.equal(oe[layer], pb.attn_extend([hb[c] for c in ext], ext_n, layer, qe[layer]))
        torch.cuda.synchronize()
        for c, s, n in items:
            lens[c] = s + n
        for i, c in enumerate(dec):
            for layer in (0, nl - 1):
                kk, vv = _kv(c, layer, 0, lens[c])
                ref = attend_last(sv.bf16_to_f64(qd[layer, i:i + 1]), sv.bf16_to_f64(kk), sv.bf16_to_f64(vv))
                assert_close(od[layer, i:i + 1], ref, f"decode conv {c} layer {layer}")
    pa.close()
    pb.close()
