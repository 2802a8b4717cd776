"""GPU: the tiny two-conversation agentic trace end to end, every call against the oracle.

Flow (Section 4): turn-1 prefill on the prefiller pool -> pack -> unpack into the decoder pool
(the one-time transfer) -> turn-1 decodes on the decoder -> turns 2..3 append 32 tokens, extend,
then decode 16 tokens one at a time. Decodes are batched across both conversations.
"""
import numpy as np
import pytest
import torch

from oracle import kvwire
from oracle.attention import attend_last
from synth import values as sv
from synth.traces import TinyTrace
from tests.helpers import assert_close, f64, kv_tokens, q_tokens

pytestmark = pytest.mark.gpu


def test_tiny_trace_end_to_end():
    from paper_2606_01839_amd import KVPool
    tr = TinyTrace()
    sh = tr.shape
    seed = tr.seed
    mk = lambda s: KVPool(sh.n_layers, sh.n_q_heads, sh.n_kv_heads, sh.head_dim, n_pages=64,
                          max_convs=4, max_pages_per_conv=32, placement_seed=s, device="cuda")
    pre, dec = mk(1), mk(2)
    cids = range(tr.n_convs)
    ref = {c: kvwire.ConversationKV(sh.n_layers, sh.n_kv_heads, sh.head_dim) for c in cids}

    def kv(c, start, n):
        k, v = kv_tokens(seed, c, sh.n_layers, start, n, sh.n_kv_heads, sh.head_dim)
        ref[c].append(sv.bf16_bits(k).reshape(k.shape), sv.bf16_bits(v).reshape(v.shape))
        return k, v

    def f64_bits(b):
        return sv.bf16_bits_to_f64(b)

    # turn 1: prefill on the prefiller
    hp = {}
    for c in cids:
        hp[c] = pre.conv_create()
        k, v = kv(c, 0, tr.turn1)
        pre.kv_append(hp[c], k.cuda(), v.cuda())
    q = [q_tokens(seed, c, 0, 0, tr.turn1, sh.n_q_heads, sh.head_dim) for c in cids]
    out = pre.attn_prefill_turn1([hp[c] for c in cids], [tr.turn1] * tr.n_convs, 0, torch.cat(q).cuda())
    torch.cuda.synchronize()
    for c in cids:
        r = attend_last(f64(q[c]), f64_bits(ref[c].k[0]), f64_bits(ref[c].v[0]))
        assert_close(out[c * tr.turn1:(c + 1) * tr.turn1], r, f"turn-1 prefill conv {c}")

    # the one-time transfer
    hd = {}
    for c in cids:
        wire = pre.kv_pack(hp[c])
        hd[c] = dec.kv_unpack(wire, tr.turn1)
        torch.cuda.synchronize()
        assert np.array_equal(wire.cpu().numpy().view(np.uint16), kvwire.serialize(ref[c].k, ref[c].v))
        pre.conv_destroy(hp[c])
    assert pre.occupancy()[0] == 0

    def decode_steps(n):
        for _ in range(n):
            lens = {c: ref[c].length for c in cids}
            ks, vs = zip(*[kv(c, lens[c], 1) for c in cids])
            dec.kv_append_batch([hd[c] for c in cids], [1] * tr.n_convs, torch.cat(ks, 1).cuda(),
                                torch.cat(vs, 1).cuda())
            qd = torch.cat([q_tokens(seed, c, 0, lens[c], 1, sh.n_q_heads, sh.head_dim) for c in cids])
            o = dec.attn_decode_batch([hd[c] for c in cids], 0, qd.cuda())
            torch.cuda.synchronize()
            for c in cids:
                r = attend_last(f64(qd[c:c + 1]), f64_bits(ref[c].k[0]), f64_bits(ref[c].v[0]))
                assert_close(o[c:c + 1], r, f"decode conv {c} at {lens[c]}")

    if tr.turn1_decode:
        decode_steps(tr.decodes)
    for _turn in range(2, tr.turns + 1):
        lens = {c: ref[c].length for c in cids}
        ks, vs = zip(*[kv(c, lens[c], tr.append) for c in cids])
        dec.kv_append_batch([hd[c] for c in cids], [tr.append] * tr.n_convs, torch.cat(ks, 1).cuda(),
                            torch.cat(vs, 1).cuda())
        qe = [q_tokens(seed, c, 0, lens[c], tr.append, sh.n_q_heads, sh.head_dim) for c in cids]
        o = dec.attn_extend([hd[c] for c in cids], [tr.append] * tr.n_convs, 0, torch.cat(qe).cuda())
        torch.cuda.synchronize()
        for c in cids:
            r = attend_last(f64(qe[c]), f64_bits(ref[c].k[0]), f64_bits(ref[c].v[0]))
            assert_close(o[c * tr.append:(c + 1) * tr.append], r, f"extend conv {c} turn {_turn}")
        decode_steps(tr.decodes)

    for c in cids:
        assert dec.conv_len(hd[c]) == tr.final_len() == ref[c].length
        assert len(dec.conv_pages(hd[c])) == (tr.final_len() + 15) // 16
        w = dec.kv_pack(hd[c])
        torch.cuda.synchronize()
        assert np.array_equal(w.cpu().numpy().view(np.uint16), kvwire.serialize(ref[c].k, ref[c].v))
    for c in cids:
        dec.conv_destroy(hd[c])
    assert dec.occupancy() == (0, 64)
    pre.close()
    dec.close()
