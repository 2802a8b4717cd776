"""GPU parity on the hard cases of softmax attention (the scaled dot-product attention of the
served model, Section 2.1), for turn-1 prefill, extend, decode on the direct single-item path and
decode on the split + merge path, at head_dim 64 and 128 and GQA groups 1, 2, 4 and 8.

Inputs come from ``synth.edge`` (see there): a sharply peaked softmax (Q = 4 K[j*]), scores that
climb ~10 log2 units per 64-key tile, a sawtooth of such climbs, and Q = 0 (uniform weights,
closed form: the running mean of V). For ``peak`` and ``rise`` the test first asserts, from the
scores of its own inputs, that some 64-key tile raises a row's maximum by more than 8 log2 units
over every earlier tile -- the condition under which both prefill kernels rescale O and the
denominator after their first tile (and the decode split rescales its running state).

Every output element is checked against the fp64 oracle within the bound that follows from the
kernels' arithmetic (tests.helpers.arith_bound: bf16-rounded weights summed into the denominator,
fp32 scores and accumulation, bf16 output) -- which holds at any |O| -- and, at unit-scale V, also
within the fixed tolerance of max-abs 1e-2 and rel-L2 3e-3. With V scaled by 64, outputs reach
|O| >> 4, where half a bf16 ulp alone exceeds 1e-2; there only the arithmetic bound applies.
"""
import numpy as np
import pytest
import torch

from oracle.attention import attend_rows, kv_head_of
from synth.edge import PROFILES, edge_inputs
from tests.helpers import assert_close, assert_within_arith_bound, f64, tile_jumps

pytestmark = pytest.mark.gpu

SHAPES = [(64, 1), (64, 2), (64, 4), (64, 8), (128, 1), (128, 2), (128, 4), (128, 8)]   # (d, G)
HKV = 2
# mode -> [(length, query rows)] per conversation
MODES = {
    "prefill": [(1, 1), (70, 70), (330, 330)],
    "extend": [(670, 70), (64, 47), (300, 1)],
    "decode_direct": [(1, 1), (333, 1), (1024, 1)],          # each conversation one work item
    "decode_merge": [(1100, 1), (2900, 1), (65, 1)],          # items of 1024 keys: merged
}


def _case(profile, d, G, mode, v_scale=1.0, seed=0):
    from paper_2606_01839_amd import KVPool
    hq = G * HKV
    convs_spec = MODES[mode]
    pages = sum((L + 15) // 16 for L, _ in convs_spec) + 4
    pool = KVPool(1, hq, HKV, d, n_pages=pages, max_convs=8, max_pages_per_conv=256,
                  placement_seed=17 + seed, device="cuda")
    convs, data = [], []
    for i, (L, n) in enumerate(convs_spec):
        k, v, q = edge_inputs(profile, L, n, hq, HKV, d, lambda h: kv_head_of(h, hq, HKV),
                              seed=1000 * seed + 31 * i + d + G, v_scale=v_scale)
        c = pool.conv_create()
        pool.kv_append(c, k[None].contiguous().cuda(), v[None].contiguous().cuda())
        convs.append(c)
        data.append((k, v, q))
    q_all = torch.cat([q for _, _, q in data]).cuda()
    if mode == "prefill":
        out = pool.attn_prefill_turn1(convs, [n for _, n in convs_spec], 0, q_all)
    elif mode == "extend":
        out = pool.attn_extend(convs, [n for _, n in convs_spec], 0, q_all)
    else:
        out = pool.attn_decode_batch(convs, 0, q_all)
    torch.cuda.synchronize()
    out = out.cpu()
    pool.close()
    return convs_spec, data, out


def _check(profile, d, G, mode, v_scale=1.0):
    print(f"edge case: profile={profile} d={d} G={G} mode={mode} v_scale={v_scale}", flush=True)
    spec, data, out = _case(profile, d, G, mode, v_scale)
    row, jumps, worst = 0, [], 0.0
    for i, ((L, n), (k, v, q)) in enumerate(zip(spec, data)):
        qf, kf, vf = f64(q), f64(k), f64(v)
        pos = np.arange(L - n, L)
        ref = attend_rows(qf, pos, kf, vf)
        got = out[row:row + n]
        what = f"{profile} d{d} G{G} {mode} conv {i} (L {L}, rows {n}, V x{v_scale})"
        worst = max(worst, assert_within_arith_bound(got, qf, pos, kf, vf, ref, what))
        if v_scale == 1.0:
            assert_close(got, ref, what)
        if profile == "zero":   # closed form: every row is the running mean of its visible V
            for j in (0, n - 1):
                for h in range(G * HKV):
                    m = vf[: pos[j] + 1, kv_head_of(h, G * HKV, HKV)].mean(0)
                    np.testing.assert_allclose(ref[j, h], m, atol=1e-12)
        if L > 64:
            jumps.append(float(tile_jumps(qf, pos, kf).max()))
        row += n
    if profile == "rise" or (profile == "peak" and mode in ("prefill", "extend")):
        assert max(jumps) > 8, f"no tile raised the running max by > 8 log2 units: {jumps}"
    return worst


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("d,G", SHAPES)
@pytest.mark.parametrize("profile", PROFILES)
def test_edge_profiles(profile, d, G, mode):
    _check(profile, d, G, mode)


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("profile", ["peak", "rise", "zero"])
def test_edge_large_outputs(profile, d, mode):
    """V x 64: outputs far above 4 in magnitude, checked within the arithmetic bound."""
    _check(profile, d, 4, mode, v_scale=64.0)


@pytest.mark.parametrize("layer_ordered", [False, True])
def test_edge_mixed_step(layer_ordered):
    """cs_mixed_step (the fused extend + decode launches) on rising scores, two layers."""
    from paper_2606_01839_amd import KVPool
    d, G, nl = 128, 4, 2
    hq = G * HKV
    print(f"edge mixed step layer_ordered={layer_ordered}", flush=True)
    # two extending conversations (prefix, chunk) and two decoding ones (prefix)
    ext, dec = [(900, 130), (40, 60)], [1500, 200]
    lens = [P + n for P, n in ext] + [P + 1 for P in dec]
    pool = KVPool(nl, hq, HKV, d, n_pages=sum((L + 15) // 16 for L in lens) + 4, max_convs=8,
                  max_pages_per_conv=256, placement_seed=5, device="cuda")
    data = []   # per conversation, per layer: (k, v, q) over the whole final length
    for i, L in enumerate(lens):
        n_q = ext[i][1] if i < len(ext) else 1
        data.append([edge_inputs("rise", L, n_q, hq, HKV, d, lambda h: kv_head_of(h, hq, HKV),
                                 seed=500 + 10 * i + layer) for layer in range(nl)])
    convs = []
    for i, L in enumerate(lens):
        P = ext[i][0] if i < len(ext) else dec[i - len(ext)]
        c = pool.conv_create()
        k = torch.stack([data[i][l][0][:P] for l in range(nl)]).contiguous().cuda()
        v = torch.stack([data[i][l][1][:P] for l in range(nl)]).contiguous().cuda()
        pool.kv_append(c, k, v)
        convs.append(c)
    new_k, new_v, q_ext, q_dec = [], [], [], []
    for l in range(nl):
        ks, vs = [], []
        for i, (P, n) in enumerate(ext):
            ks.append(data[i][l][0][P:P + n])
            vs.append(data[i][l][1][P:P + n])
        for j, P in enumerate(dec):
            ks.append(data[len(ext) + j][l][0][P:P + 1])
            vs.append(data[len(ext) + j][l][1][P:P + 1])
        new_k.append(torch.cat(ks))
        new_v.append(torch.cat(vs))
        q_ext.append(torch.cat([data[i][l][2] for i in range(len(ext))]))
        q_dec.append(torch.cat([data[len(ext) + j][l][2] for j in range(len(dec))]))
    cu = lambda xs: torch.stack(xs).contiguous().cuda()
    oe, od = pool.mixed_step(convs[:len(ext)], [n for _, n in ext], convs[len(ext):], cu(new_k), cu(new_v),
                             q_ext=cu(q_ext), q_dec=cu(q_dec), layer_ordered=layer_ordered)
    torch.cuda.synchronize()
    oe, od = oe.cpu(), od.cpu()
    pool.close()
    for l in range(nl):
        row = 0
        for i, (P, n) in enumerate(ext):
            k, v, q = (f64(t) for t in data[i][l])
            pos = np.arange(P, P + n)
            ref = attend_rows(q, pos, k, v)
            assert_within_arith_bound(oe[l, row:row + n], q, pos, k, v, ref, f"mixed ext {i} layer {l}")
            assert_close(oe[l, row:row + n], ref, f"mixed ext {i} layer {l}")
            row += n
        for j, P in enumerate(dec):
            k, v, q = (f64(t) for t in data[len(ext) + j][l])
            ref = attend_rows(q, [P], k, v)
            assert_within_arith_bound(od[l, j:j + 1], q, [P], k, v, ref, f"mixed dec {j} layer {l}")
            assert_close(od[l, j:j + 1], ref, f"mixed dec {j} layer {l}")
