"""GPU parity of turn-1 prefill, extend and batched decode against the fp64 oracle.

Sizes span several 64-query / 64-key tiles, page boundaries, ragged tails and the degenerate cases
(L = 1, q_len = 1, q_len = L, empty batch). Tolerance per call: max-abs 1e-2, rel-L2 3e-3.
"""
import numpy as np
import pytest
import torch

from oracle.attention import attend_last
from tests.helpers import assert_close, f64, kv_tokens, q_tokens, errors

pytestmark = pytest.mark.gpu

SEED = 777


def _pool(hq, hkv, d, n_pages, seed=3, max_convs=64, max_pages=4096, n_layers=1):
    from paper_2606_01839_amd import KVPool
    return KVPool(n_layers, hq, hkv, d, n_pages=n_pages, max_convs=max_convs,
                  max_pages_per_conv=max_pages, placement_seed=seed, device="cuda")


def _fill(pool, conv, cid, L, hkv, d, scales=(None, None)):
    k, v = kv_tokens(SEED, cid, 1, 0, L, hkv, d, k_scale=scales[0], v_scale=scales[1])
    if L:
        pool.kv_append(conv, k.cuda(), v.cuda())
    return k, v


def _extend_case(hq, hkv, d, prefixes, chunks, pool_seed=3, scales=(None, None)):
    pages = sum((p + c + 15) // 16 for p, c in zip(prefixes, chunks)) + 8
    pool = _pool(hq, hkv, d, pages, seed=pool_seed)
    convs, kvs, qs = [], [], []
    for i, (P, n) in enumerate(zip(prefixes, chunks)):
        c = pool.conv_create()
        k, v = _fill(pool, c, i, P + n, hkv, d, scales)
        convs.append(c)
        kvs.append((k, v))
        qs.append(q_tokens(SEED, i, 0, P, n, hq, d))
    q = torch.cat(qs).cuda()
    if all(P == 0 for P in prefixes):
        out = pool.attn_prefill_turn1(convs, chunks, 0, q)
    else:
        out = pool.attn_extend(convs, chunks, 0, q)
    torch.cuda.synchronize()
    row = 0
    for i, n in enumerate(chunks):
        ref = attend_last(f64(qs[i]), f64(kvs[i][0][0]), f64(kvs[i][1][0]))
        assert_close(out[row:row + n], ref, f"conv {i} prefix {prefixes[i]} chunk {n}")
        row += n
    pool.close()
    return out


@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (4, 2, 64), (16, 8, 128), (64, 8, 128), (8, 8, 128),
                                      (8, 1, 64), (4, 4, 64)])
def test_prefill_turn1_ragged(hq, hkv, d):
    _extend_case(hq, hkv, d, [0, 0, 0, 0, 0], [1, 17, 64, 130, 333])


@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (16, 8, 128), (64, 8, 128), (4, 2, 64)])
def test_extend_against_prefix(hq, hkv, d):
    _extend_case(hq, hkv, d, [1, 15, 64, 100, 1000, 2047], [1, 64, 65, 127, 200, 77])


def test_extend_with_head_scales():
    sk = np.array([0.5, 0.9, 1.3, 2.0, 1.0, 0.7, 1.7, 1.1], dtype=np.float32)
    sv_ = np.array([2.0, 0.6, 1.0, 1.5, 0.5, 1.9, 0.8, 1.2], dtype=np.float32)
    _extend_case(32, 8, 128, [300, 900], [256, 96], scales=(sk, sv_))


def _decode_case(hq, hkv, d, lens, pool_seed=3, scales=(None, None)):
    pages = sum((L + 15) // 16 for L in lens) + 8
    pool = _pool(hq, hkv, d, pages, seed=pool_seed)
    convs, kvs = [], []
    for i, L in enumerate(lens):
        c = pool.conv_create()
        kvs.append(_fill(pool, c, i, L, hkv, d, scales))
        convs.append(c)
    q = torch.cat([q_tokens(SEED, i, 0, L - 1, 1, hq, d) for i, L in enumerate(lens)]).cuda()
    out = pool.attn_decode_batch(convs, 0, q)
    torch.cuda.synchronize()
    for i, L in enumerate(lens):
        ref = attend_last(f64(q[i:i + 1].cpu()), f64(kvs[i][0][0]), f64(kvs[i][1][0]))
        assert_close(out[i:i + 1], ref, f"decode conv {i} L {L}")
    res = out.clone()
    pool.close()
    return res, q


@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (4, 2, 64), (8, 8, 64), (16, 8, 128), (64, 8, 128),
                                      (8, 8, 128)])
def test_decode_ragged(hq, hkv, d):
    _decode_case(hq, hkv, d, [1, 2, 15, 16, 17, 31, 32, 33, 100, 511, 512, 513, 1024, 1025, 3000])


def test_full_pool_and_full_page_table_rows():
    """Maximum sizes of a pool: every page allocated and every conversation at max_pages_per_conv
    (its page-table row full); decode, extend of the last 100 tokens and turn-1 prefill of a whole
    row all match the oracle, and one more token is refused without changing anything."""
    from paper_2606_01839_amd import KVPool, ConserveError, CS_ERANGE, CS_ENOMEM
    hq, hkv, d, rows, n = 32, 8, 128, 64, 4
    L = rows * 16
    pool = KVPool(1, hq, hkv, d, n_pages=n * rows, max_convs=n, max_pages_per_conv=rows,
                  placement_seed=11, device="cuda")
    convs, kvs = [], []
    for i in range(n):
        c = pool.conv_create()
        kvs.append(_fill(pool, c, i, L, hkv, d))
        convs.append(c)
    assert pool.occupancy() == (n * rows, 0)
    q = torch.cat([q_tokens(SEED, i, 0, L - 1, 1, hq, d) for i in range(n)]).cuda()
    out = pool.attn_decode_batch(convs, 0, q)
    qe = torch.cat([q_tokens(SEED, i, 0, L - 100, 100, hq, d) for i in range(n)]).cuda()
    oe = pool.attn_extend(convs, [100] * n, 0, qe)
    q1 = q_tokens(SEED, 0, 0, 0, L, hq, d)
    o1 = pool.attn_prefill_turn1([convs[0]], [L], 0, q1.cuda())
    torch.cuda.synchronize()
    assert_close(o1, attend_last(f64(q1), f64(kvs[0][0][0]), f64(kvs[0][1][0])), "prefill of a full row")
    for i in range(n):
        k, v = kvs[i]
        assert_close(out[i:i + 1], attend_last(f64(q[i:i + 1].cpu()), f64(k[0]), f64(v[0])), f"decode {i}")
        assert_close(oe[100 * i:100 * i + 100], attend_last(f64(qe[100 * i:100 * i + 100].cpu()), f64(k[0]),
                                                            f64(v[0])), f"extend {i}")
    one = torch.zeros(1, 1, hkv, d, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ConserveError) as e:
        pool.kv_append(convs[0], one, one)
    assert e.value.code in (CS_ERANGE, CS_ENOMEM)
    assert pool.conv_len(convs[0]) == L and pool.occupancy() == (n * rows, 0)
    pool.close()


def test_decode_long_contexts_few_convs():
    sk = np.linspace(0.5, 2.0, 8).astype(np.float32)
    _decode_case(32, 8, 128, [9000, 20000], scales=(sk, sk[::-1].copy()))


def test_decode_bitwise_deterministic_and_placement_invariant():
    lens = [5, 700, 1500, 2600]
    a, _ = _decode_case(32, 8, 128, lens, pool_seed=1)
    b, _ = _decode_case(32, 8, 128, lens, pool_seed=1)
    c, _ = _decode_case(32, 8, 128, lens, pool_seed=12345)
    assert torch.equal(a, b), "decode is not bitwise deterministic"
    assert torch.equal(a, c), "decode depends on physical page placement"


def test_decode_bitwise_independent_of_batch_order():
    """Work items are launched in an order that depends on the whole batch (full items first, then
    the others by decreasing key count); a conversation's output must not: the same conversations
    decoded in reversed and shuffled batch order give bitwise the same rows."""
    hq, hkv, d = 32, 8, 128
    lens = [5, 700, 1500, 2600, 1024, 1025, 3000, 2048]
    pool = _pool(hq, hkv, d, sum((L + 15) // 16 for L in lens) + 8, seed=5)
    convs = []
    for i, L in enumerate(lens):
        c = pool.conv_create()
        _fill(pool, c, i, L, hkv, d)
        convs.append(c)
    q = torch.cat([q_tokens(SEED, i, 0, L - 1, 1, hq, d) for i, L in enumerate(lens)]).cuda()
    base = pool.attn_decode_batch(convs, 0, q)
    for perm in (list(reversed(range(len(lens)))), [3, 0, 6, 1, 7, 2, 5, 4]):
        out = pool.attn_decode_batch([convs[j] for j in perm], 0, q[perm].contiguous())
        torch.cuda.synchronize()
        assert torch.equal(out, base[perm]), perm
    pool.close()


def test_extend_bitwise_placement_invariant():
    a = _extend_case(32, 8, 128, [0, 500], [200, 150], pool_seed=1)
    b = _extend_case(32, 8, 128, [0, 500], [200, 150], pool_seed=777)
    assert torch.equal(a, b)


def test_decode_matches_extend_of_one_and_last_prefill_row():
    hq, hkv, d = 32, 8, 128
    L = 777
    pool = _pool(hq, hkv, d, 80)
    c = pool.conv_create()
    _fill(pool, c, 0, L, hkv, d)
    qall = q_tokens(SEED, 0, 0, 0, L, hq, d).cuda()
    full = pool.attn_prefill_turn1([c], [L], 0, qall)
    ext = pool.attn_extend([c], [1], 0, qall[-1:].contiguous())
    dec = pool.attn_decode_batch([c], 0, qall[-1:].contiguous())
    torch.cuda.synchronize()
    for x, y in [(full[-1:], ext), (ext, dec), (full[-1:], dec)]:
        m, r = errors(x, f64(y))
        assert m <= 1e-2 and r <= 3e-3
    pool.close()


def test_chunked_extend_matches_one_shot_prefill():
    hq, hkv, d = 32, 8, 128
    L = 640
    cuts = [0, 100, 101, 333, 640]
    pool = _pool(hq, hkv, d, 100)
    one = pool.conv_create()
    k, v = kv_tokens(SEED, 0, 1, 0, L, hkv, d)
    pool.kv_append(one, k.cuda(), v.cuda())
    q = q_tokens(SEED, 0, 0, 0, L, hq, d).cuda()
    full = pool.attn_prefill_turn1([one], [L], 0, q)
    ch = pool.conv_create()
    parts = []
    for a, b in zip(cuts[:-1], cuts[1:]):
        pool.kv_append(ch, k[:, a:b].contiguous().cuda(), v[:, a:b].contiguous().cuda())
        parts.append(pool.attn_extend([ch], [b - a], 0, q[a:b].contiguous()))
    torch.cuda.synchronize()
    m, r = errors(torch.cat(parts), f64(full))
    assert m <= 1e-2 and r <= 3e-3
    pool.close()


@pytest.mark.parametrize("hq,hkv", [(32, 8), (16, 8)])
def test_aligned_chunked_prefill_is_bitwise_one_shot(hq, hkv):
    """Chunked turn-1 prefill (the prefiller's chunked prefill, Section 5.1) with chunks that are
    multiples of the query tile (64 queries at 32q/8kv, 128 at 16q/8kv): every query tile sweeps
    the same key tiles in the same order as in the one-shot prefill, so the outputs agree bit for
    bit (and both match the oracle)."""
    d = 128
    lens, chunk = [700, 300], 256
    pool = _pool(hq, hkv, d, 2 * sum((L + 15) // 16 for L in lens) + 8)
    one = [pool.conv_create() for _ in lens]
    kv = [kv_tokens(SEED, b, 1, 0, L, hkv, d) for b, L in enumerate(lens)]
    for c, (k, v) in zip(one, kv):
        pool.kv_append(c, k.cuda(), v.cuda())
    qs = [q_tokens(SEED, b, 0, 0, L, hq, d).cuda() for b, L in enumerate(lens)]
    full = pool.attn_prefill_turn1(one, lens, 0, torch.cat(qs))
    ch = [pool.conv_create() for _ in lens]
    got = [[] for _ in lens]
    for s0 in range(0, max(lens), chunk):
        act = [b for b, L in enumerate(lens) if L > s0]
        n = [min(chunk, lens[b] - s0) for b in act]
        k = torch.cat([kv[b][0][:, s0:s0 + nb] for b, nb in zip(act, n)], dim=1).contiguous().cuda()
        v = torch.cat([kv[b][1][:, s0:s0 + nb] for b, nb in zip(act, n)], dim=1).contiguous().cuda()
        pool.kv_append_batch([ch[b] for b in act], n, k, v)
        out = pool.attn_extend([ch[b] for b in act], n, 0,
                               torch.cat([qs[b][s0:s0 + nb] for b, nb in zip(act, n)]))
        r = 0
        for b, nb in zip(act, n):
            got[b].append(out[r:r + nb])
            r += nb
    torch.cuda.synchronize()
    assert torch.equal(torch.cat([torch.cat(g) for g in got]), full)
    for b, L in enumerate(lens):
        k, v = kv[b]
        row0 = sum(lens[:b])
        assert_close(full[row0:row0 + L], attend_last(f64(qs[b]), f64(k[0]), f64(v[0])), f"conv {b}")
    pool.close()


def test_nan_poisoned_pool_does_not_leak():
    """Every page starts as NaN; appends zero their pages' tails, so nothing past a conversation's
    end (or in never-used pages) can reach the outputs."""
    hq, hkv, d = 32, 8, 128
    lens = [1, 17, 300]
    pool = _pool(hq, hkv, d, 40)
    pool.kv.view(torch.int16).fill_(0x7FC0)  # bf16 quiet NaN everywhere
    convs, kvs = [], []
    for i, L in enumerate(lens):
        c = pool.conv_create()
        kvs.append(_fill(pool, c, i, L, hkv, d))
        convs.append(c)
    q = torch.cat([q_tokens(SEED, i, 0, L - 1, 1, hq, d) for i, L in enumerate(lens)]).cuda()
    out = pool.attn_decode_batch(convs, 0, q)
    qp = torch.cat([q_tokens(SEED, i, 0, 0, L, hq, d) for i, L in enumerate(lens)]).cuda()
    outp = pool.attn_prefill_turn1(convs, lens, 0, qp)
    torch.cuda.synchronize()
    row = 0
    for i, L in enumerate(lens):
        ref = attend_last(f64(q[i:i + 1].cpu()), f64(kvs[i][0][0]), f64(kvs[i][1][0]))
        assert_close(out[i:i + 1], ref, f"poisoned decode {i}")
        refp = attend_last(f64(qp[row:row + L].cpu()), f64(kvs[i][0][0]), f64(kvs[i][1][0]))
        assert_close(outp[row:row + L], refp, f"poisoned prefill {i}")
        row += L
    pool.close()


def test_empty_batches_are_noops():
    pool = _pool(32, 8, 128, 8)
    c = pool.conv_create()
    _fill(pool, c, 0, 20, 8, 128)
    q0 = torch.empty(0, 32, 128, dtype=torch.bfloat16, device="cuda")
    assert pool.attn_decode_batch([], 0, q0).shape == (0, 32, 128)
    assert pool.attn_extend([c], [0], 0, q0).shape == (0, 32, 128)
    pool.close()
