"""GPU: KV append, page tables, pack and unpack are bit-exact against the oracle's concatenation and
wire format (Section 4: the turn-1 KV is transferred exactly once; later turns only append)."""
import numpy as np
import pytest
import torch

from oracle import kvwire
from synth import values as sv
from tests.helpers import kv_tokens

pytestmark = pytest.mark.gpu

SEED = 4242


def _pool(n_layers=2, hq=4, hkv=2, d=64, n_pages=96, seed=1, max_convs=8, max_pages=64):
    from paper_2606_01839_amd import KVPool
    return KVPool(n_layers, hq, hkv, d, n_pages=n_pages, max_convs=max_convs,
                  max_pages_per_conv=max_pages, placement_seed=seed, device="cuda")


def _bits(t):
    return sv.bf16_bits(t)


def _gather_pool(pool, conv, n_layers, hkv, d):
    """Read a conversation's K/V back out of the pool through its page list (host-side numpy)."""
    pages = pool.conv_pages(conv)
    L = pool.conv_len(conv)
    blocks = pool.kv_view().cpu().numpy().view(np.uint16)  # [layer][page][head][2*16*d]
    k = np.zeros((n_layers, L, hkv, d), dtype=np.uint16)
    v = np.zeros_like(k)
    for lp, pg in enumerate(pages):
        t0, t1 = 16 * lp, min(L, 16 * lp + 16)
        b = blocks[:, pg]                                 # [layer][head][2*16*d]
        # K part: d/32 sub-blocks of 32 dims, each [16 tokens][32 dims]
        kb = b[..., : 16 * d].reshape(n_layers, hkv, d // 32, 16, 32).transpose(0, 1, 3, 2, 4)
        kb = kb.reshape(n_layers, hkv, 16, d)
        vb = b[..., 16 * d:].reshape(n_layers, hkv, d, 16)
        k[:, t0:t1] = kb[:, :, : t1 - t0].transpose(0, 2, 1, 3)
        v[:, t0:t1] = vb[:, :, :, : t1 - t0].transpose(0, 3, 1, 2)
        # tail slots of the last page are zero
        assert (kb[:, :, t1 - t0:] == 0).all() and (vb[:, :, :, t1 - t0:] == 0).all()
    return k, v


@pytest.mark.parametrize("d", [64, 128])
def test_append_pages_and_pack_bit_exact(d):
    hq, hkv, nl = (4, 2, 2) if d == 64 else (32, 8, 1)
    pool = _pool(nl, hq, hkv, d)
    conv = pool.conv_create()
    ref = kvwire.ConversationKV(nl, hkv, d)
    pos = 0
    for n in [1, 15, 16, 17, 1, 1, 31, 64, 3, 0, 100]:   # ragged appends across page boundaries
        k, v = kv_tokens(SEED, 0, nl, pos, n, hkv, d)
        pool.kv_append(conv, k.cuda(), v.cuda())
        ref.append(_bits(k).reshape(k.shape), _bits(v).reshape(v.shape))
        pos += n
        assert pool.conv_len(conv) == pos
        pages = pool.conv_pages(conv)
        assert len(pages) == (pos + 15) // 16 and len(set(pages.tolist())) == len(pages)
        assert pool.occupancy()[0] == len(pages)
    torch.cuda.synchronize()
    gk, gv = _gather_pool(pool, conv, nl, hkv, d)
    assert np.array_equal(gk, ref.k) and np.array_equal(gv, ref.v)
    wire = pool.kv_pack(conv)
    torch.cuda.synchronize()
    want = kvwire.serialize(ref.k, ref.v)
    assert wire.numel() == want.size * 2
    assert np.array_equal(wire.cpu().numpy().view(np.uint16), want)
    pool.close()


def test_unpack_round_trip_into_other_placement():
    nl, hq, hkv, d = 2, 4, 2, 64
    src = _pool(nl, hq, hkv, d, seed=11)
    dst = _pool(nl, hq, hkv, d, seed=99)
    keep = dst.conv_create()                                 # occupy some pages first
    k0, v0 = kv_tokens(SEED, 9, nl, 0, 40, hkv, d)
    dst.kv_append(keep, k0.cuda(), v0.cuda())
    for L in [1, 16, 37, 250]:
        c = src.conv_create()
        k, v = kv_tokens(SEED, L, nl, 0, L, hkv, d)
        src.kv_append(c, k.cuda(), v.cuda())
        w1 = src.kv_pack(c)
        c2 = dst.kv_unpack(w1, L)
        w2 = dst.kv_pack(c2)
        torch.cuda.synchronize()
        assert dst.conv_len(c2) == L
        assert torch.equal(w1, w2)
        gk, gv = _gather_pool(dst, c2, nl, hkv, d)
        assert np.array_equal(gk, _bits(k).reshape(k.shape)) and np.array_equal(gv, _bits(v).reshape(v.shape))
        # appending after an unpack continues the conversation (turn 2 on the decoder)
        k2, v2 = kv_tokens(SEED, L, nl, L, 5, hkv, d)
        dst.kv_append(c2, k2.cuda(), v2.cuda())
        torch.cuda.synchronize()
        gk, _ = _gather_pool(dst, c2, nl, hkv, d)
        assert np.array_equal(gk[:, L:], _bits(k2).reshape(k2.shape))
        dst.conv_destroy(c2)
        src.conv_destroy(c)
    gk, gv = _gather_pool(dst, keep, nl, hkv, d)
    assert np.array_equal(gk, _bits(k0).reshape(k0.shape))
    src.close()
    dst.close()


def test_batched_append_matches_single_appends():
    nl, hq, hkv, d = 1, 32, 8, 128
    a = _pool(nl, hq, hkv, d, n_pages=200, seed=5)
    convs = [a.conv_create() for _ in range(5)]
    lens = [0, 3, 16, 21, 40]
    for c, L in zip(convs, lens):
        if L:
            k, v = kv_tokens(SEED, c, nl, 0, L, hkv, d)
            a.kv_append(c, k.cuda(), v.cuda())
    n_new = [7, 1, 0, 30, 16]
    ks, vs = [], []
    for c, L, n in zip(convs, lens, n_new):
        k, v = kv_tokens(SEED, c, nl, L, n, hkv, d)
        ks.append(k)
        vs.append(v)
    a.kv_append_batch(convs, n_new, torch.cat(ks, 1).cuda(), torch.cat(vs, 1).cuda())
    torch.cuda.synchronize()
    for c, L, n in zip(convs, lens, n_new):
        k, v = kv_tokens(SEED, c, nl, 0, L + n, hkv, d)
        gk, gv = _gather_pool(a, c, nl, hkv, d)
        assert np.array_equal(gk, _bits(k).reshape(k.shape)) and np.array_equal(gv, _bits(v).reshape(v.shape))
    a.close()


def test_pool_exhaustion_changes_nothing():
    from paper_2606_01839_amd import ConserveError, CS_ENOMEM
    nl, hq, hkv, d = 1, 4, 2, 64
    p = _pool(nl, hq, hkv, d, n_pages=4)
    c = p.conv_create()
    k, v = kv_tokens(SEED, 0, nl, 0, 60, hkv, d)
    p.kv_append(c, k.cuda(), v.cuda())
    k2, v2 = kv_tokens(SEED, 0, nl, 60, 5, hkv, d)
    with pytest.raises(ConserveError) as e:
        p.kv_append(c, k2.cuda(), v2.cuda())
    assert e.value.code == CS_ENOMEM
    assert p.conv_len(c) == 60 and p.occupancy() == (4, 0)
    p.conv_destroy(c)
    assert p.occupancy() == (0, 4)
    p.close()
